"""Oracle: query/key channel balancer (Section 3.2, Eq. 2-4).

Test infrastructure only.  Eq. 2 sets, per layer, head and channel, the
balancer to the square root of (max |q| / max |k|) over the prefill prompt.
Eq. 3 multiplies keys by it before quantization and Eq. 4 divides queries by
it.  Readings where the paper is silent:
  * the balancer is per (sequence, KV head, channel); under grouped-query
    attention the query maximum runs over every query head of the group;
  * if either maximum is 0 the balancer is 1;
  * arithmetic is fp32: one correctly rounded divide and one correctly rounded
    square root, stored as fp32;
  * values are not balanced; the balanced key is the single fp32 product
    k * b, and the balanced query the single fp32 quotient q / b.
"""
from __future__ import annotations

import numpy as np


def balancer(q_prefill, k_prefill) -> np.ndarray:
    """q_prefill fp16 [..., G, T, D], k_prefill fp16 [..., T, D] -> b fp32 [..., D]."""
    q = np.abs(np.asarray(q_prefill, dtype=np.float16).astype(np.float32))
    k = np.abs(np.asarray(k_prefill, dtype=np.float16).astype(np.float32))
    qm = q.max(axis=(-3, -2))
    km = k.max(axis=-2)
    with np.errstate(divide="ignore", invalid="ignore"):
        b = np.sqrt(qm / km)
    return np.where((qm == 0) | (km == 0), np.float32(1), b).astype(np.float32)


def balance_keys(k16, b) -> np.ndarray:
    """Eq. 3 argument: k * b in fp32 (b broadcast over tokens)."""
    k = np.asarray(k16, dtype=np.float16).astype(np.float32)
    return k * np.asarray(b, dtype=np.float32)


def balance_query(q16, b) -> np.ndarray:
    """Eq. 4: q / b in fp32."""
    q = np.asarray(q16, dtype=np.float16).astype(np.float32)
    return q / np.asarray(b, dtype=np.float32)
