"""Oracle: decode-step attention over the mixed-precision cache (Section 3.4, Fig. 3).

Test infrastructure only.  During generation the current query attends to
every cached token; MiKV keeps K and V at reduced precision while the query
and the attention map stay floating point.  Since attention after RoPE is
permutation invariant, the order in which tokens are visited does not change
the result, so the oracle visits them in position order.

Computation (fp64 from the fp32 operands):
  q_hat = q / b                (Eq. 4; fp32; b = 1 when not balanced)
  s_j   = (q_hat . k_j) * scale
  p     = softmax(s)
  o     = sum_j p_j v_j
with k_j, v_j the fp32 decoded keys and values (fp16 values widened, or
alpha * code + beta).  o and p are returned as fp32.
"""
from __future__ import annotations

import numpy as np


def attention(q16, keys, values, scale: float, b=None):
    """q16 fp16 [G, D]; keys, values fp32 [L, D]; b fp32 [D] or None.

    Returns (o fp32 [G, D], p fp32 [G, L]).
    """
    q = np.asarray(q16, dtype=np.float16).astype(np.float32)
    if b is not None:
        q = q / np.asarray(b, dtype=np.float32)
    k = np.asarray(keys, dtype=np.float32).astype(np.float64)
    v = np.asarray(values, dtype=np.float32).astype(np.float64)
    s = (q.astype(np.float64) @ k.T) * float(scale)
    s = s - s.max(axis=1, keepdims=True)
    e = np.exp(s)
    p = e / e.sum(axis=1, keepdims=True)
    o = p @ v
    return o.astype(np.float32), p.astype(np.float32)
