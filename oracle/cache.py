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

``key_block = 64`` is the per-channel key quantization of Appendix C: the
retained cache's keys are quantized per channel over blocks of 64
consecutive positions (Eq. 1 with token and channel exchanged), values stay
per token.  Readings where the appendix is silent (it only simulates the
scheme, quantizing keys as they are, without reordering):
  * a block's parameters come from all 64 of its keys, whatever their
    precision, taken from the fp16 keys as given (prefill) or as the
    importance cache holds them (a block completed during decoding);
  * a block is quantized once, when its last position arrives; with a window
    of at least 64 positions all keys of a block that is not complete are in
    the importance cache, so a retained key always has its block's
    parameters;
  * a token's key codes are those of its block at the time it is demoted
    (the same codes as quantizing the whole block at once: a code depends
    only on the key and the block's parameters);
  * the importance cache is fp16, and no channel balancer is applied (the
    per-channel quantizer takes the balancer's place in Table 6).
"""
from __future__ import annotations

import numpy as np

from .attention import attention
from .balance import balance_keys
from .policy import accumulate, select
from .quant import dequantize, encode, f16_bits, f16_value, quantize, quantize_channels


class OracleCache:
    """Position-indexed MiKV cache for ``n_heads`` independent (sequence, KV
    head) pairs, each serving ``group_size`` query heads."""

    def __init__(self, n_heads: int, group_size: int, max_len: int, hi_bits: int, lo_bits: int,
                 group: int, head_dim: int = 128, key_block: int = 0):
        assert hi_bits in (16, 8, 4) and lo_bits in (0, 2, 3, 4, 8)
        assert key_block in (0, 64) and (key_block == 0 or (hi_bits == 16 and lo_bits in (2, 3, 4)))
        self.n_heads, self.G, self.max_len = n_heads, group_size, max_len
        self.hi_bits, self.lo_bits, self.group, self.d = hi_bits, lo_bits, group, head_dim
        self.key_block = key_block
        if key_block:
            # per-channel key parameters of each block of key_block positions
            nb = max_len // key_block
            self.kb_a = np.zeros((n_heads, nb, head_dim), np.uint16)
            self.kb_b = np.zeros((n_heads, nb, head_dim), np.uint16)
            self.kb_done = np.zeros((n_heads, nb), bool)
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
        if self.key_block:
            blk = np.asarray(pos) // self.key_block
            assert self.kb_done[h, blk].all(), "retained key of a block that is not complete"
            self.lk[h, pos] = encode(kx, self.kb_a[h, blk], self.kb_b[h, blk], n)
        else:
            self.lk[h, pos], self.lk_a[h, pos], self.lk_b[h, pos] = quantize(kx, n, self.group)
        self.lv[h, pos], self.lv_a[h, pos], self.lv_b[h, pos] = quantize(vx, n, self.group)

    def _close_block(self, h, blk, keys):
        """Per-channel parameters of key block ``blk`` from its keys fp32 [64, D]."""
        _, self.kb_a[h, blk], self.kb_b[h, blk] = quantize_channels(keys, self.lo_bits)
        self.kb_done[h, blk] = True

    def _hi_values(self, h, pos):
        if self.hi_bits == 16:
            return f16_value(self.hk[h, pos]), f16_value(self.hv[h, pos])
        g = self.group
        return (dequantize(self.hk[h, pos], self.hk_a[h, pos], self.hk_b[h, pos], g),
                dequantize(self.hv[h, pos], self.hv_a[h, pos], self.hv_b[h, pos], g))

    def _lo_values(self, h, pos):
        g = self.group
        if self.key_block:
            blk = np.asarray(pos) // self.key_block
            # alpha * code + beta per channel with the block's parameters
            k = f16_value(self.kb_a[h, blk]) * self.lk[h, pos].astype(np.float32) + f16_value(self.kb_b[h, blk])
        else:
            k = dequantize(self.lk[h, pos], self.lk_a[h, pos], self.lk_b[h, pos], g)
        return k, dequantize(self.lv[h, pos], self.lv_a[h, pos], self.lv_b[h, pos], g)

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
        assert not self.key_block or (balance is None and window >= self.key_block)
        for h in range(H):
            hi = select(scores[h], None, T, k_heavy, window, initial=True)
            kx = balance_keys(k16[h], balance[h]) if balance is not None else \
                np.asarray(k16[h], np.float16).astype(np.float32)
            vx = np.asarray(v16[h], np.float16).astype(np.float32)
            pos = np.arange(T)
            if self.key_block:  # every complete block of the prompt, from its keys as given
                kb = self.key_block
                for blk in range(T // kb):
                    self._close_block(h, blk, kx[blk * kb:(blk + 1) * kb])
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
            kb = self.key_block
            if kb and (pos + 1) % kb == 0:  # the token completes a block: quantize it per channel
                blk = pos // kb
                span = np.arange(blk * kb, pos + 1)
                assert self.is_hi[h, span].all(), "a block completes with keys outside the importance cache"
                self._close_block(h, blk, f16_value(self.hk[h, span]))
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
