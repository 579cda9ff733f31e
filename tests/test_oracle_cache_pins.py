"""Pins for the oracle's whole decode step over quantized and balanced caches.

The quantizer pins (test_oracle_quant.py) check Eq. 1 on its own, and the
attention pins check softmax attention on its own; these check what the
cache does with them: which scale and zero point decode which tokens, what
the balancer touches, what demotion re-quantizes.

Lossless inputs.  A group of values that lies exactly on the grid
beta + alpha * c (alpha, beta fp16, c = 0 .. 2^N - 1 with both ends taken) is
reconstructed exactly by Eq. 1 at N bits: the minimum is beta, the range over
2^N - 1 is alpha, and (x - beta) / alpha is the integer c.  With
alpha = 85 * 2^e the same values also lie on the 4-bit grid (step 17 * 2^e)
and the 8-bit grid (step 2^e), so every representation the cache can give a
token -- fp16, INT8 or INT4 importance cache, INT2 or INT4 retained cache,
demotion from one to the other -- decodes to the original values.  Attention
over such a cache must then be textbook attention over the original fp16
keys and values (torch's fp64 scaled_dot_product_attention and softmax),
whatever the precision map; a cache that decodes a value with the key's
scale, balances values or re-balances at demotion breaks that.

Balanced caches (Section 3.2, Eq. 3-4).  With a power-of-two balancer every
product k * b and quotient q / b is exact and Eq. 1 commutes with the
scaling, so a balanced cache must give bit-for-bit the attention of the
unbalanced one, store f16(k * b) (or Eq. 1 of k * b), and demote from the
stored balanced row without applying b again.

Each pin is also run against a copy of the oracle with a planted mistake
(a subclass overriding one method), which it must reject.
"""
import math

import numpy as np
import pytest
import torch

import oracle

SCALE = 1.0 / math.sqrt(128.0)
D = 128


# -- lossless inputs ------------------------------------------------------------

def lossless_rows(rng, n, group, levels, step_mult):
    """fp16 [n, 128] rows whose every group is exactly beta + alpha * c,
    alpha = step_mult * 2^e, c in [0, levels) with both 0 and levels - 1
    present, so Eq. 1 at log2(levels) bits reconstructs it exactly."""
    ng = D // group
    x = np.empty((n, D), np.float64)
    for r in range(n):
        for gi in range(ng):
            e = int(rng.integers(-9, -5))
            m = int(rng.integers(-600, 600))
            c = rng.integers(0, levels, group)
            i0, i1 = rng.choice(group, 2, replace=False)
            c[i0], c[i1] = 0, levels - 1
            x[r, gi * group:(gi + 1) * group] = (m + step_mult * c) * 2.0 ** e
    x16 = x.astype(np.float16)
    assert (x16.astype(np.float64) == x).all()          # fp16-exact by construction
    return x16


def sdpa_reference(q16, K16, V16):
    """torch fp64: o by scaled_dot_product_attention, p by softmax."""
    q = torch.from_numpy(np.asarray(q16, np.float16).astype(np.float64))     # [G, D]
    K = torch.from_numpy(np.asarray(K16, np.float16).astype(np.float64))     # [L, D]
    V = torch.from_numpy(np.asarray(V16, np.float16).astype(np.float64))
    o = torch.nn.functional.scaled_dot_product_attention(q[None, :, None, :], K[None, None].expand(1, len(q), -1, -1),
                                                         V[None, None].expand(1, len(q), -1, -1), scale=SCALE)
    p = torch.softmax((q @ K.T) * SCALE, dim=-1)
    return o[0, :, 0].numpy(), p.numpy()


def run_lossless(cache_cls, hi_bits, lo_bits, group, G=2, H=2, T=200, steps=5, W=16, seed=0):
    """Prefill + decode steps over lossless rows; every step's o and p must
    equal torch's attention over the original rows.  Returns the number of
    demotions seen (so the caller can require that demotion ran)."""
    rng = np.random.default_rng(seed)
    levels, mult = (8, int(rng.integers(3, 40)) | 1) if lo_bits == 3 else (4, 85)
    n = T + steps
    K = np.stack([lossless_rows(rng, n, group, levels, mult) for _ in range(H)])
    V = np.stack([lossless_rows(rng, n, group, levels, mult) for _ in range(H)])
    q = rng.standard_normal((steps, H, G, D)).astype(np.float16)
    sc = rng.random((H, T)).astype(np.float32)
    c = cache_cls(H, G, n, hi_bits, lo_bits, group)
    kh = lambda L: max(0, L // 4 - W)
    c.prefill(K[:, :T], V[:, :T], sc, kh(T), W)
    assert c.is_hi[:, :T].any() and (~c.is_hi[:, :T]).any()
    demoted = 0
    for t in range(steps):
        L = T + t + 1
        before = c.is_hi[:, :L].copy()
        before[:, L - 1] = True                                  # the appended token
        o, p = c.step(q[t], K[:, T + t], V[:, T + t], SCALE, kh(L) - 3 * (t % 2), W)   # shrinking budgets demote
        demoted += int((before & ~c.is_hi[:, :L]).sum())
        for h in range(H):
            o_ref, p_ref = sdpa_reference(q[t, h], K[h, :L], V[h, :L])
            np.testing.assert_allclose(o[h], o_ref, rtol=1e-6, atol=1e-7, err_msg=f"step {t} head {h}: o")
            np.testing.assert_allclose(p[h], p_ref, rtol=1e-6, atol=1e-12, err_msg=f"step {t} head {h}: p")
    return demoted


# (importance cache bits, retained cache bits, group)
LOSSLESS_CASES = [(16, 2, 32), (8, 2, 32), (4, 2, 32), (16, 4, 64), (8, 4, 64), (16, 3, 32), (16, 3, 64),
                  (8, 8, 128)]


@pytest.mark.parametrize("hi,lo,group", LOSSLESS_CASES)
def test_lossless_mixed_cache_equals_textbook_attention(hi, lo, group):
    """Section 3.4 / Eq. 1: over inputs Eq. 1 reconstructs exactly, the
    mixed-precision cache attends like an unquantized one."""
    assert run_lossless(oracle.OracleCache, hi, lo, group) > 0


def test_lossless_rows_really_are_lossless():
    """The generator's premise, checked with the quantizer's own pins'
    arithmetic left out: brute-force nearest-level search over the grid the
    stored fp16 scale and zero describe reproduces every value."""
    rng = np.random.default_rng(3)
    for bits, levels, mult in ((2, 4, 85), (4, 4, 85), (8, 4, 85), (3, 8, 13)):
        x = lossless_rows(rng, 6, 32, levels, mult).astype(np.float32)
        codes, a16, b16 = oracle.quantize(x, bits, 32)
        a = a16.view(np.float16).astype(np.float64)[..., None]
        b = b16.view(np.float16).astype(np.float64)[..., None]
        grid = b + a * np.arange(2 ** bits)            # [rows, groups, levels]
        xg = x.reshape(6, 4, 32).astype(np.float64)
        nearest = np.abs(xg[..., None] - grid[..., None, :]).min(-1)
        assert (nearest == 0).all()


# -- planted mistakes ---------------------------------------------------------------

class ValueWithKeyParams(oracle.OracleCache):
    """Mistake: retained values decoded with the key's scale and zero point."""

    def _lo_values(self, h, pos):
        g = self.group
        return (oracle.dequantize(self.lk[h, pos], self.lk_a[h, pos], self.lk_b[h, pos], g),
                oracle.dequantize(self.lv[h, pos], self.lk_a[h, pos], self.lk_b[h, pos], g))


class HiValueWithKeyParams(oracle.OracleCache):
    """Mistake: quantized importance-cache values decoded with the key's parameters."""

    def _hi_values(self, h, pos):
        if self.hi_bits == 16:
            return super()._hi_values(h, pos)
        g = self.group
        return (oracle.dequantize(self.hk[h, pos], self.hk_a[h, pos], self.hk_b[h, pos], g),
                oracle.dequantize(self.hv[h, pos], self.hk_a[h, pos], self.hk_b[h, pos], g))


class SwappedScaleZero(oracle.OracleCache):
    """Mistake: retained keys decoded as beta * code + alpha."""

    def _lo_values(self, h, pos):
        k, v = super()._lo_values(h, pos)
        g = self.group
        return oracle.dequantize(self.lk[h, pos], self.lk_b[h, pos], self.lk_a[h, pos], g), v


class DemoteFromOriginalBits(oracle.OracleCache):
    """Mistake: demotion re-quantizes the importance cache's raw codes as if
    they were values (skips the decode)."""

    def select(self, k_heavy, window):
        L = self.length
        out = []
        for h in range(self.n_heads):
            new_hi = oracle.select(self.acc[h], self.is_hi[h], L, k_heavy, window, initial=False)
            dem = np.nonzero(self.is_hi[h, :L] & ~new_hi)[0]
            if dem.size:
                raw = lambda a: a.astype(np.float32) if self.hi_bits != 16 else oracle.f16_value(a)
                self._store_lo(h, dem, raw(self.hk[h, dem]), raw(self.hv[h, dem]))
            self.is_hi[h, :L] = new_hi
            out.append(dem)
        return out


@pytest.mark.parametrize("cls,hi,lo,group", [
    (ValueWithKeyParams, 16, 2, 32),
    (HiValueWithKeyParams, 8, 2, 32),
    (SwappedScaleZero, 16, 4, 64),
    (DemoteFromOriginalBits, 8, 2, 32),
])
def test_lossless_pin_rejects_planted_mistakes(cls, hi, lo, group):
    with pytest.raises(AssertionError):
        run_lossless(cls, hi, lo, group)


# -- balanced caches (Eq. 3-4) -----------------------------------------------------

def run_balanced_pair(cache_cls, hi_bits, lo_bits, group, G=2, H=2, T=160, steps=5, W=16, seed=1, lossless=False):
    """The same prompt and steps through a cache balanced by b and an
    unbalanced one; o and p must agree bit for bit every step.  b is a power
    of two constant over each quantization group, so k * b is exact and
    Eq. 1 of k * b is Eq. 1 of k with alpha and beta times b (the fp16
    rounding of alpha commutes with the scale).
    Returns (balanced cache, unbalanced cache, b, keys)."""
    rng = np.random.default_rng(seed)
    n = T + steps
    if lossless:
        K = np.stack([lossless_rows(rng, n, group, 4, 85) for _ in range(H)])
        V = np.stack([lossless_rows(rng, n, group, 4, 85) for _ in range(H)])
    else:
        K = (rng.standard_normal((H, n, D)) * np.where(np.arange(D) % 37 == 0, 12, 1)).astype(np.float16)
        V = rng.standard_normal((H, n, D)).astype(np.float16)
    q = rng.standard_normal((steps, H, G, D)).astype(np.float16)
    # b >= 1: a product below 1 could fall into fp16's subnormal range and
    # round there (f16(k * b) != f16(k) * b)
    b = np.repeat(2.0 ** rng.integers(0, 4, (H, D // group)), group, axis=1).astype(np.float32)
    sc = rng.random((H, T)).astype(np.float32)
    kh = lambda L: max(0, L // 4 - W)
    cb = cache_cls(H, G, n, hi_bits, lo_bits, group)
    cu = oracle.OracleCache(H, G, n, hi_bits, lo_bits, group)
    cb.prefill(K[:, :T], V[:, :T], sc, kh(T), W, balance=b)
    cu.prefill(K[:, :T], V[:, :T], sc, kh(T), W)
    for t in range(steps):
        L = T + t + 1
        ob, pb = cb.step(q[t], K[:, T + t], V[:, T + t], SCALE, kh(L) - 2 * (t % 2), W, balance=b)
        ou, pu = cu.step(q[t], K[:, T + t], V[:, T + t], SCALE, kh(L) - 2 * (t % 2), W)
        np.testing.assert_array_equal(ob, ou, err_msg=f"step {t}: o, balanced vs unbalanced")
        np.testing.assert_array_equal(pb, pu, err_msg=f"step {t}: p, balanced vs unbalanced")
        np.testing.assert_array_equal(cb.is_hi, cu.is_hi)
    return cb, cu, b, K


@pytest.mark.parametrize("hi,lo,group", [(16, 2, 32), (8, 2, 32), (8, 4, 64), (4, 2, 32), (16, 3, 32)])
def test_power_of_two_balance_leaves_attention_unchanged(hi, lo, group):
    """Eq. 3-4 with a power-of-two balancer: identical o and p, every step,
    through prefill placement, appends, demotions and re-quantization."""
    run_balanced_pair(oracle.OracleCache, hi, lo, group)


@pytest.mark.parametrize("hi,lo,group", [(16, 2, 32), (8, 2, 32)])
def test_balanced_cache_stores_balanced_keys_and_demotes_without_rebalancing(hi, lo, group):
    """The balanced cache's stored key rows: fp16 pool f16(k * b) (widened
    k times b in fp32, rounded once); INT8 pool codes and parameters equal
    the unbalanced cache's codes with alpha, beta scaled by b (Eq. 1 commutes
    with a power-of-two scale); retained keys likewise -- so demotion
    decoded the stored (balanced) row and did not multiply by b again.
    Values are never balanced: identical to the unbalanced cache's."""
    cb, cu, b, K = run_balanced_pair(oracle.OracleCache, hi, lo, group, lossless=True)
    L = cb.length
    ng = D // group
    for h in range(cb.n_heads):
        hi_pos = np.nonzero(cb.is_hi[h, :L])[0]
        lo_pos = np.nonzero(~cb.is_hi[h, :L])[0]
        assert lo_pos.size > 0 and hi_pos.size > 0
        bh = b[h].astype(np.float64)
        bg = bh.reshape(ng, group)[:, 0]                          # b of each group
        f16 = lambda bits: bits.view(np.float16).astype(np.float64)
        if hi == 16:
            want = (K[h, hi_pos].astype(np.float64) * bh).astype(np.float16).view(np.uint16)
            np.testing.assert_array_equal(cb.hk[h, hi_pos], want)
        else:
            np.testing.assert_array_equal(cb.hk[h, hi_pos], cu.hk[h, hi_pos])
            np.testing.assert_array_equal(f16(cb.hk_a[h, hi_pos]), f16(cu.hk_a[h, hi_pos]) * bg)
            np.testing.assert_array_equal(f16(cb.hk_b[h, hi_pos]), f16(cu.hk_b[h, hi_pos]) * bg)
        np.testing.assert_array_equal(cb.hv[h, hi_pos], cu.hv[h, hi_pos])
        # retained keys: the unbalanced cache's codes, parameters times b --
        # and, the rows being lossless, decoded exactly to k * b; values are
        # the unbalanced cache's
        np.testing.assert_array_equal(cb.lk[h, lo_pos], cu.lk[h, lo_pos])
        np.testing.assert_array_equal(f16(cb.lk_a[h, lo_pos]), f16(cu.lk_a[h, lo_pos]) * bg)
        np.testing.assert_array_equal(f16(cb.lk_b[h, lo_pos]), f16(cu.lk_b[h, lo_pos]) * bg)
        kb, vb = cb._lo_values(h, lo_pos)
        np.testing.assert_array_equal(kb.astype(np.float64), K[h, lo_pos].astype(np.float64) * bh)
        ku, vu = cu._lo_values(h, lo_pos)
        np.testing.assert_array_equal(vb, vu)
        np.testing.assert_array_equal(cb.lv[h, lo_pos], cu.lv[h, lo_pos])


class RebalanceOnDemotion(oracle.OracleCache):
    """Mistake: demoted keys multiplied by the balancer a second time."""

    def prefill(self, k16, v16, scores, k_heavy, window, balance=None):
        self._b = balance
        super().prefill(k16, v16, scores, k_heavy, window, balance)

    def select(self, k_heavy, window):
        L = self.length
        out = []
        for h in range(self.n_heads):
            new_hi = oracle.select(self.acc[h], self.is_hi[h], L, k_heavy, window, initial=False)
            dem = np.nonzero(self.is_hi[h, :L] & ~new_hi)[0]
            if dem.size:
                kx, vx = self._hi_values(h, dem)
                self._store_lo(h, dem, kx * self._b[h], vx)
            self.is_hi[h, :L] = new_hi
            out.append(dem)
        return out


class BalancedValues(oracle.OracleCache):
    """Mistake: values multiplied by the balancer too."""

    def append(self, k16, v16, balance=None):
        if balance is not None:
            v16 = (np.asarray(v16, np.float16).astype(np.float32) * balance).astype(np.float16)
        super().append(k16, v16, balance)


class QueryNotBalanced(oracle.OracleCache):
    """Mistake: the query is not divided by the balancer (Eq. 4 dropped)."""

    def attend(self, q16, scale, balance=None):
        return super().attend(q16, scale, None)


@pytest.mark.parametrize("cls", [RebalanceOnDemotion, BalancedValues, QueryNotBalanced])
def test_balance_pin_rejects_planted_mistakes(cls):
    with pytest.raises(AssertionError):
        run_balanced_pair(cls, 16, 2, 32)
