"""Pins for the oracle's per-channel key quantization (Appendix C, Table 6).

Keys of the retained cache are quantized per channel over blocks of 64
consecutive positions -- Eq. 1 with token and channel exchanged -- and
values per token.  What pins it here, none of it the oracle's own output:

* Table 6's cache sizes (38 % INT3, 33 % INT2 with 20 % fp16 importance
  cache) from the storage format;
* hand-checkable per-channel blocks: a channel spanning [beta, beta + 3 alpha]
  gives codes 0 .. 3 and the stored fp16 alpha, beta; an outlier channel does
  not widen any other channel's scale (the point of Appendix C);
* lossless blocks: every channel of every 64-position block on its own grid
  beta_c + alpha_c * {0 .. 2^N - 1} (both ends taken), values lossless per
  token -- the whole decode (prefill, block completions during decoding,
  demotions) must then attend exactly like textbook attention over the
  original keys and values (torch fp64);
* lazy encoding: a token's key codes taken at demotion with its block's
  parameters equal quantizing the whole block at once;
* block boundaries: parameters of a block completed during decoding equal
  those a prefill of the same keys computes;
* planted mistakes, each of which must fail one of the above.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from tests.conftest import read_golden

SCALE = 1.0 / math.sqrt(128.0)
D = 128
KB = 64


@pytest.mark.parametrize("row", read_golden("table6_per_channel.txt"), ids=lambda r: r[0])
def test_table6_cache_sizes(row):
    """Table 6: 20 % fp16 importance cache; retained keys per channel over 64
    positions (N-bit codes + fp16 scale and zero per channel and block),
    retained values per token (g = 64)."""
    _, r, n, pct = row
    r, n = float(r), int(n)
    key = oracle.bits_per_element(n, KB)       # per channel, group of 64 tokens
    val = oracle.bits_per_element(n, 64)       # per token, group of 64 channels
    size = r * 16 / 16 + (1 - r) * (key + val) / 2 / 16
    assert math.floor(size * 100 + 0.5) == int(pct)


def test_quantize_channels_hand_example():
    """Two channels over a 4-token block: channel 0 spans [-1, 2] (alpha 1,
    beta -1, codes 0 1 2 3), channel 1 holds an outlier 100 that sets only
    its own scale (alpha = f16(103/3) = 34.34375, codes rint((x+3)/alpha))."""
    x = np.array([[-1, -3], [0, 1], [1, 100], [2, -2]], np.float32)
    codes, a, b = oracle.quantize_channels(x, 2)
    assert a.view(np.float16).tolist() == [1.0, 34.34375]
    assert b.view(np.float16).tolist() == [-1.0, -3.0]
    assert codes[:, 0].tolist() == [0, 1, 2, 3]
    assert codes[:, 1].tolist() == [0, 0, 3, 0]


def test_per_channel_isolates_an_outlier_channel():
    """Appendix C's motivation: with one outlier channel the per-token groups
    that contain it get a scale several times larger, while per-channel
    scales of the other channels do not change."""
    rng = np.random.default_rng(0)
    x = rng.standard_normal((KB, D)).astype(np.float32)
    y = x.copy()
    y[:, 5] *= 20
    _, a0, _ = oracle.quantize_channels(x, 2)
    _, a1, _ = oracle.quantize_channels(y, 2)
    others = np.arange(D) != 5
    np.testing.assert_array_equal(a0[others], a1[others])
    _, t0, _ = oracle.quantize(x, 2, 32)
    _, t1, _ = oracle.quantize(y, 2, 32)
    ratio = t1[:, 0].view(np.float16).astype(np.float64) / t0[:, 0].view(np.float16).astype(np.float64)
    assert np.median(ratio) > 2


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_lazy_encoding_equals_block_quantization(bits):
    """A code depends only on the key and its block's parameters: encoding
    each token with the block's stored parameters reproduces the block's
    codes, and both match brute-force nearest-level search."""
    rng = np.random.default_rng(bits)
    blk = (rng.standard_normal((KB, D)) * np.where(np.arange(D) % 17 == 0, 20, 1)).astype(np.float16)
    x = blk.astype(np.float32)
    codes, a, b = oracle.quantize_channels(x, bits)
    for t in range(KB):
        np.testing.assert_array_equal(oracle.encode(x[t], a, b, bits), codes[t])
    af, bf = a.view(np.float16).astype(np.float64), b.view(np.float16).astype(np.float64)
    grid = bf[None, :, None] + af[None, :, None] * np.arange(2 ** bits)[None, None, :]   # [1, D, levels]
    dist = np.abs(x.astype(np.float64)[:, :, None] - grid)
    best = dist.min(-1)
    chosen = np.take_along_axis(dist, codes[:, :, None].astype(np.int64), -1)[..., 0]
    np.testing.assert_array_equal(chosen, best)      # the code is a nearest level (ties: either)


# -- lossless blocks ----------------------------------------------------------------

def lossless_channel_keys(rng, n, levels, mult):
    """fp16 keys [n, 128]: in every block of 64 positions, channel c takes
    values (m_c + mult * code) * 2^e_c, interior codes except at one random
    position with code 0 and another with levels - 1, so per-channel Eq. 1
    over the whole block reconstructs them exactly at any width whose grid
    holds the levels (mult = 85: 2, 4 and 8 bits), and over a subset of the
    block usually does not."""
    k = np.empty((n, D), np.float64)
    for b0 in range(0, n, KB):
        t = min(KB, n - b0)
        e = rng.integers(-9, -5, D)
        m = rng.integers(-600, 600, D)
        c = rng.integers(1, levels - 1, (t, D))
        if t >= 2:
            for col in range(D):
                i0, i1 = rng.choice(t, 2, replace=False)
                c[i0, col], c[i1, col] = 0, levels - 1
        k[b0:b0 + t] = (m + mult * c) * 2.0 ** e
    k16 = k.astype(np.float16)
    assert (k16.astype(np.float64) == k).all()
    return k16


def lossless_token_values(rng, n, group, levels, mult):
    x = np.empty((n, D), np.float64)
    for r in range(n):
        for gi in range(D // group):
            e = int(rng.integers(-9, -5))
            m = int(rng.integers(-600, 600))
            c = rng.integers(0, levels, group)
            i0, i1 = rng.choice(group, 2, replace=False)
            c[i0], c[i1] = 0, levels - 1
            x[r, gi * group:(gi + 1) * group] = (m + mult * c) * 2.0 ** e
    return x.astype(np.float16)


def sdpa(q16, K16, V16):
    q = torch.from_numpy(np.asarray(q16, np.float16).astype(np.float64))
    K = torch.from_numpy(np.asarray(K16, np.float16).astype(np.float64))
    V = torch.from_numpy(np.asarray(V16, np.float16).astype(np.float64))
    o = torch.nn.functional.scaled_dot_product_attention(q[None, :, None, :], K[None, None].expand(1, len(q), -1, -1),
                                                         V[None, None].expand(1, len(q), -1, -1), scale=SCALE)
    return o[0, :, 0].numpy(), torch.softmax((q @ K.T) * SCALE, dim=-1).numpy()


def run_channel_lossless(cache_cls, lo_bits, group=32, G=1, H=2, T=250, steps=10, W=64, seed=0):
    """Prefill of T tokens, then decode steps that complete a block (position
    255) and demote tokens; o and p checked against torch every step.
    Returns the demotions seen and the cache."""
    rng = np.random.default_rng(seed)
    levels, mult = (8, int(rng.integers(3, 40)) | 1) if lo_bits == 3 else (4, 85)
    n = T + steps
    K = np.stack([lossless_channel_keys(rng, n, levels, mult) for _ in range(H)])
    V = np.stack([lossless_token_values(rng, n, group, levels, mult) for _ in range(H)])
    q = rng.standard_normal((steps, H, G, D)).astype(np.float16)
    sc = rng.random((H, T)).astype(np.float32)
    c = cache_cls(H, G, n, 16, lo_bits, group, key_block=KB)
    kh = lambda L: max(0, L // 2 - W)
    c.prefill(K[:, :T], V[:, :T], sc, kh(T), W)
    assert (~c.is_hi[:, :T]).any()
    demoted = 0
    for t in range(steps):
        L = T + t + 1
        before = c.is_hi[:, :L].copy()
        before[:, L - 1] = True
        o, p = c.step(q[t], K[:, T + t], V[:, T + t], SCALE, kh(L) - 3 * (t % 2), W)
        demoted += int((before & ~c.is_hi[:, :L]).sum())
        for h in range(H):
            o_ref, p_ref = sdpa(q[t, h], K[h, :L], V[h, :L])
            np.testing.assert_allclose(o[h], o_ref, rtol=1e-6, atol=1e-7, err_msg=f"step {t} head {h}: o")
            np.testing.assert_allclose(p[h], p_ref, rtol=1e-6, atol=1e-12, err_msg=f"step {t} head {h}: p")
    assert c.kb_done[:, (T + steps) // KB - 1].all()   # a block completed during decoding
    return demoted, c, K


@pytest.mark.parametrize("lo_bits,group", [(2, 32), (3, 32), (4, 64), (2, 128)])
def test_lossless_channel_blocks_equal_textbook_attention(lo_bits, group):
    demoted, c, K = run_channel_lossless(oracle.OracleCache, lo_bits, group)
    assert demoted > 0
    # retained keys decode to the original keys, demoted ones included
    for h in range(c.n_heads):
        lo = np.nonzero(~c.is_hi[h, :c.length])[0]
        k, _ = c._lo_values(h, lo)
        np.testing.assert_array_equal(k, K[h, lo].astype(np.float32))


def test_block_parameters_do_not_depend_on_when_the_block_completes():
    """A block completed by decode-step appends gets the parameters that a
    prefill of the same keys gives it; demoted keys are their block's codes."""
    rng = np.random.default_rng(4)
    H, T0, T1 = 2, 150, 300
    K = (rng.standard_normal((H, T1, D)) * np.where(np.arange(D) % 23 == 0, 15, 1)).astype(np.float16)
    V = rng.standard_normal((H, T1, D)).astype(np.float16)
    sc = rng.random((H, T1)).astype(np.float32)
    full = oracle.OracleCache(H, 1, T1, 16, 2, 32, key_block=KB)
    full.prefill(K, V, sc, 40, 64)
    part = oracle.OracleCache(H, 1, T1, 16, 2, 32, key_block=KB)
    part.prefill(K[:, :T0], V[:, :T0], sc[:, :T0], 20, 64)
    q = rng.standard_normal((H, 1, D)).astype(np.float16)
    for t in range(T0, T1):
        part.step(q, K[:, t], V[:, t], SCALE, max(0, (t + 1) // 5 - 64), 64)
    nb = T1 // KB
    assert part.kb_done[:, :nb].all() and full.kb_done[:, :nb].all()
    np.testing.assert_array_equal(part.kb_a[:, :nb], full.kb_a[:, :nb])
    np.testing.assert_array_equal(part.kb_b[:, :nb], full.kb_b[:, :nb])
    for h in range(H):
        for blk in range(nb):
            codes, a, b = oracle.quantize_channels(K[h, blk * KB:(blk + 1) * KB].astype(np.float32), 2)
            np.testing.assert_array_equal(a, full.kb_a[h, blk])
            lo = [j for j in range(blk * KB, (blk + 1) * KB) if not part.is_hi[h, j]]
            np.testing.assert_array_equal(part.lk[h, lo], codes[np.array(lo, int) - blk * KB])


# -- planted mistakes ---------------------------------------------------------------

class BlockFromRetainedOnly(oracle.OracleCache):
    """Mistake: a prompt block's parameters from its retained keys only."""

    def prefill(self, k16, v16, scores, k_heavy, window, balance=None):
        self._scores, self._kw = scores, (k_heavy, window)
        super().prefill(k16, v16, scores, k_heavy, window, balance)

    def _close_block(self, h, blk, keys):
        if self.length == 0:     # during prefill: keep the retained rows only
            hi = oracle.select(self._scores[h], None, len(self._scores[h]), *self._kw, initial=True)
            sub = ~hi[blk * 64:(blk + 1) * 64]
            if sub.sum() >= 2:
                keys = keys[sub]
        super()._close_block(h, blk, keys)


class KeysWithValueParams(oracle.OracleCache):
    """Mistake: retained keys decoded per token with the value's parameters."""

    def _lo_values(self, h, pos):
        g = self.group
        return (oracle.dequantize(self.lk[h, pos], self.lv_a[h, pos], self.lv_b[h, pos], g),
                oracle.dequantize(self.lv[h, pos], self.lv_a[h, pos], self.lv_b[h, pos], g))


class BlockNeverRefreshed(oracle.OracleCache):
    """Mistake: blocks completed during decoding keep the previous block's parameters."""

    def _close_block(self, h, blk, keys):
        if self.length > 0 and blk > 0:
            self.kb_a[h, blk], self.kb_b[h, blk] = self.kb_a[h, blk - 1], self.kb_b[h, blk - 1]
            self.kb_done[h, blk] = True
            return
        super()._close_block(h, blk, keys)


@pytest.mark.parametrize("cls", [BlockFromRetainedOnly, KeysWithValueParams, BlockNeverRefreshed])
def test_channel_pins_reject_planted_mistakes(cls):
    with pytest.raises(AssertionError):
        run_channel_lossless(cls, 2, 32, steps=40)
