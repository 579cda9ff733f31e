"""Oracle: the MiKV cache and one decode step, position indexed.

Test infrastructure only.  The cache of each (sequence, KV head) is kept as
plain per-position arrays: a precision flag, the high-precision representation
(fp16 values, or INT8 codes with fp16 alpha/beta per group), the
low-precision representation (N-bit codes with fp16 alpha/beta per group) and
the importance score.  Only one representation of a token is meaningful at a
time, the one its flag names.

Step order (Fig. 3; H2O order -- attend, accumulate, then evict/demote):
  1. append the new token's key/value at high precision (keys balanced,
     Eq. 3), score 0;
  2. attention of the query over every cached token (Section 3.4);
  3. importance update with the step's probabilities;
  4. selection; every demoted token is re-quantized from its high-precision
     representation to the low precision (Section 3.1: tokens that eviction
     would drop are retained at low precision instead).  Keys in the cache are
     already balanced, so the balancer is not applied again.
Prefill stores the prompt's tokens after a first selection in which every
token outside the window is eligible, scored by the supplied initial scores.

``lo_bits = 0`` is the eviction baseline the paper compares against (H2O, a
retained cache of 0 bits, Section 4 / Table 1): a token outside the
importance cache is dropped, and attention runs over the importance cache
alone (its probabilities are 0 at evicted positions).
"""
from __future__ import annotations

import numpy as np

from .attention import attention
from .balance import balance_keys
from .policy import accumulate, select
from .quant import dequantize, f16_bits, f16_value, quantize


class OracleCache:
    """Position-indexed MiKV cache for ``n_heads`` independent (sequence, KV
    head) pairs, each serving ``group_size`` query heads."""

    def __init__(self, n_heads: int, group_size: int, max_len: int, hi_bits: int, lo_bits: int,
                 group: int, head_dim: int = 128):
        assert hi_bits in (16, 8, 4) and lo_bits in (0, 2, 3, 4, 8)
        self.n_heads, self.G, self.max_len = n_heads, group_size, max_len
        self.hi_bits, self.lo_bits, self.group, self.d = hi_bits, lo_bits, group, head_dim
        ng = head_dim // group
        shape, pshape = (n_heads, max_len, head_dim), (n_heads, max_len, ng)
        self.is_hi = np.zeros((n_heads, max_len), dtype=bool)
        self.acc = np.zeros((n_heads, max_len), dtype=np.float32)
        # high-precision representation: fp16 bits, or INT8 codes + params
        self.hk = np.zeros(shape, dtype=np.uint16 if hi_bits == 16 else np.uint8)
        self.hv = np.zeros_like(self.hk)
        self.hk_a, self.hk_b = np.zeros(pshape, np.uint16), np.zeros(pshape, np.uint16)
        self.hv_a, self.hv_b = np.zeros(pshape, np.uint16), np.zeros(pshape, np.uint16)
        # low-precision representation (unpacked codes)
        self.lk = np.zeros(shape, dtype=np.uint8)
        self.lv = np.zeros(shape, dtype=np.uint8)
        self.lk_a, self.lk_b = np.zeros(pshape, np.uint16), np.zeros(pshape, np.uint16)
        self.lv_a, self.lv_b = np.zeros(pshape, np.uint16), np.zeros(pshape, np.uint16)
        self.length = 0

    # -- representations ---------------------------------------------------
    def _store_hi(self, h, pos, kx, vx):
        if self.hi_bits == 16:
            self.hk[h, pos] = f16_bits(kx)
            self.hv[h, pos] = f16_bits(vx)
        else:
            n = self.hi_bits  # INT8, or INT4 (Table 3's INT4 importance cache)
            self.hk[h, pos], self.hk_a[h, pos], self.hk_b[h, pos] = quantize(kx, n, self.group)
            self.hv[h, pos], self.hv_a[h, pos], self.hv_b[h, pos] = quantize(vx, n, self.group)

    def _store_lo(self, h, pos, kx, vx):
        n = self.lo_bits
        if n == 0:  # evicted: nothing is kept
            return
        self.lk[h, pos], self.lk_a[h, pos], self.lk_b[h, pos] = quantize(kx, n, self.group)
        self.lv[h, pos], self.lv_a[h, pos], self.lv_b[h, pos] = quantize(vx, n, self.group)

    def _hi_values(self, h, pos):
        if self.hi_bits == 16:
            return f16_value(self.hk[h, pos]), f16_value(self.hv[h, pos])
        g = self.group
        return (dequantize(self.hk[h, pos], self.hk_a[h, pos], self.hk_b[h, pos], g),
                dequantize(self.hv[h, pos], self.hv_a[h, pos], self.hv_b[h, pos], g))

    def _lo_values(self, h, pos):
        g = self.group
        return (dequantize(self.lk[h, pos], self.lk_a[h, pos], self.lk_b[h, pos], g),
                dequantize(self.lv[h, pos], self.lv_a[h, pos], self.lv_b[h, pos], g))

    def values(self, h):
        """Decoded fp32 keys and values [L, D] of head ``h`` in position order."""
        L = self.length
        pos = np.arange(L)
        hi = self.is_hi[h, :L]
        k = np.empty((L, self.d), np.float32)
        v = np.empty((L, self.d), np.float32)
        k[hi], v[hi] = self._hi_values(h, pos[hi])
        if self.lo_bits:
            k[~hi], v[~hi] = self._lo_values(h, pos[~hi])
        else:  # evicted positions hold nothing
            k[~hi], v[~hi] = 0.0, 0.0
        return k, v

    # -- phases -------------------------------------------------------------
    def prefill(self, k16, v16, scores, k_heavy: int, window: int, balance=None):
        """k16, v16 fp16 [H, T, D]; scores fp32 [H, T]; balance fp32 [H, D] or None."""
        H, T, _ = np.shape(k16)
        assert H == self.n_heads and T <= self.max_len
        for h in range(H):
            hi = select(scores[h], None, T, k_heavy, window, initial=True)
            kx = balance_keys(k16[h], balance[h]) if balance is not None else \
                np.asarray(k16[h], np.float16).astype(np.float32)
            vx = np.asarray(v16[h], np.float16).astype(np.float32)
            pos = np.arange(T)
            self._store_hi(h, pos[hi], kx[hi], vx[hi])
            self._store_lo(h, pos[~hi], kx[~hi], vx[~hi])
            self.is_hi[h, :T] = hi
            self.acc[h, :T] = np.asarray(scores[h], np.float32)
        self.length = T

    def append(self, k16, v16, balance=None):
        """One new token per head: k16, v16 fp16 [H, D]."""
        pos = self.length
        assert pos < self.max_len
        for h in range(self.n_heads):
            kx = balance_keys(k16[h], balance[h]) if balance is not None else \
                np.asarray(k16[h], np.float16).astype(np.float32)
            vx = np.asarray(v16[h], np.float16).astype(np.float32)
            self._store_hi(h, pos, kx, vx)
            self.is_hi[h, pos] = True
            self.acc[h, pos] = 0.0
        self.length = pos + 1

    def attend(self, q16, scale: float, balance=None):
        """q16 fp16 [H, G, D] -> (o fp32 [H, G, D], p fp32 [H, G, L])."""
        o = np.empty((self.n_heads, self.G, self.d), np.float32)
        p = np.empty((self.n_heads, self.G, self.length), np.float32)
        for h in range(self.n_heads):
            k, v = self.values(h)
            b = None if balance is None else balance[h]
            if self.lo_bits:
                o[h], p[h] = attention(q16[h], k, v, scale, b)
            else:  # eviction: only the importance cache is attended
                keep = self.is_hi[h, :self.length]
                p[h] = 0.0
                o[h], p[h][:, keep] = attention(q16[h], k[keep], v[keep], scale, b)
        return o, p

    def accumulate(self, probs):
        """probs fp32 [H, G, L] (the step's attention probabilities)."""
        L = self.length
        for h in range(self.n_heads):
            self.acc[h, :L] = accumulate(self.acc[h, :L], probs[h])

    def select(self, k_heavy: int, window: int):
        """Re-rank, demote and re-quantize.  Returns the demoted positions per head."""
        L = self.length
        demoted = []
        for h in range(self.n_heads):
            new_hi = select(self.acc[h], self.is_hi[h], L, k_heavy, window, initial=False)
            dem = np.nonzero(self.is_hi[h, :L] & ~new_hi)[0]
            if dem.size:
                kx, vx = self._hi_values(h, dem)
                self._store_lo(h, dem, kx, vx)
            self.is_hi[h, :L] = new_hi
            demoted.append(dem)
        return demoted

    def step(self, q16, k16, v16, scale: float, k_heavy: int, window: int, balance=None, probs=None):
        """One full decode step.  ``probs`` (optional) replaces the oracle's own
        probabilities in the importance update (lock-step comparison)."""
        self.append(k16, v16, balance)
        o, p = self.attend(q16, scale, balance)
        self.accumulate(p if probs is None else probs)
        self.select(k_heavy, window)
        return o, p
