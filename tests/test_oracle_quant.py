"""Pins for the oracle's Eq. 1 quantizer, its packing and fp16 rounding.

None of these compares the oracle with a re-typed copy of itself: the pins are
hand-worked values, a second library's fp16 rounding, brute force over all
quantization levels, error bounds and exact algebraic invariances.
"""
import math
import struct

import numpy as np
import pytest

import oracle
from tests.conftest import read_golden


def _f32(s):
    return np.float32(float(s))


@pytest.mark.parametrize("row", read_golden("quantizer_examples.txt"), ids=lambda r: r[0])
def test_hand_worked_examples(row):
    name, bits = row[0], int(row[1])
    x = np.array([_f32(v) for v in row[2:6]], dtype=np.float32)
    a16, b16 = int(row[6], 16), int(row[7], 16)
    codes = [int(v) for v in row[8:12]]
    xhat = np.array([_f32(v) for v in row[12:16]], dtype=np.float32)
    c, a, b = oracle.quantize(x, bits, 4)
    assert int(a[0]) == a16, name
    assert int(b[0]) == b16, name
    assert c.tolist() == codes, name
    np.testing.assert_array_equal(oracle.dequantize(c, a, b, 4), xhat)


@pytest.mark.parametrize("row", read_golden("packing_examples.txt"))
def test_packing_examples(row):
    bits = int(row[0])
    arrow = row.index("->")
    codes = np.array([int(v) for v in row[1:arrow]], dtype=np.uint8)
    expect = [int(v, 16) for v in row[arrow + 1:]]
    assert oracle.pack(codes, bits).tolist() == expect
    assert oracle.unpack(oracle.pack(codes, bits), bits).tolist() == codes.tolist()


def test_fp16_rounding_agrees_with_python_struct():
    """numpy's fp32->fp16 and CPython's binary16 packing are two independent
    round-to-nearest-even implementations; they must agree everywhere,
    including the subnormal range and exact ties."""
    rng = np.random.default_rng(5)
    vals = [0.0, -0.0, 65504.0, 65519.99, 65520.0, 6.103515625e-05, 5.960464477539063e-08,
            2.9802322387695312e-08, 8.940696716308594e-08, 1.0 + 2 ** -11, 1.0 + 3 * 2 ** -11]
    # exact ties between adjacent fp16 values, normal and subnormal
    h = np.arange(0, 0x7bff, 37, dtype=np.uint16)
    lo = h.view(np.float16).astype(np.float64)
    hi = (h + 1).view(np.float16).astype(np.float64)
    ties = ((lo + hi) / 2).astype(np.float32)
    rand = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 10, 20000))).astype(np.float32)
    xs = np.concatenate([np.array(vals, np.float32), ties, -ties, rand])
    ours = oracle.f16_bits(xs)
    for x, o in zip(xs.tolist(), ours.tolist()):
        ref = struct.unpack("<H", struct.pack("<e", x))[0] if abs(x) < 65520 else (0x7c00 | (0x8000 if x < 0 else 0))
        assert o == ref, (x, hex(o), hex(ref))


def _random_groups(rng, n, g, scale=1.0):
    x = rng.standard_normal((n, g)).astype(np.float32) * np.float32(scale)
    x[: n // 8] += np.float32(50.0)        # offset-dominated groups
    x[n // 8: n // 4] *= np.float32(1e-3)  # tiny ranges
    return x


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
@pytest.mark.parametrize("g", [32, 64])
def test_nearest_level_brute_force(bits, g):
    """Each code names the level alpha*c + beta nearest to x (up to fp32
    rounding of the division), unless clamped; found by trying every level."""
    rng = np.random.default_rng(bits * 100 + g)
    x = _random_groups(rng, 4000, g)
    c, a16, b16 = oracle.quantize(x, bits, g)
    a = oracle.f16_value(a16).astype(np.float64)
    b = oracle.f16_value(b16).astype(np.float64)
    levels = np.arange(2 ** bits, dtype=np.float64)
    xd = x.astype(np.float64)
    lv = a[:, :, None] * levels[None, None, :] + b[:, :, None]           # [n, 1, levels]
    dist = np.abs(xd[:, :, None] - lv)                                  # [n, g, levels]
    best = dist.min(axis=-1)
    chosen = np.take_along_axis(dist, c[:, :, None].astype(np.int64), axis=-1)[..., 0]
    slack = 4 * np.spacing(np.abs(xd).max(axis=1, keepdims=True)) + 1e-12
    assert np.all(chosen <= best + slack)
    assert c.max() <= 2 ** bits - 1


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_reconstruction_error_bound(bits):
    """|x - x_hat| <= alpha/2 + |beta16 - min| + |alpha16*(2^N-1) - range| + fp32 slack."""
    g = 32
    rng = np.random.default_rng(7 + bits)
    x = _random_groups(rng, 3000, g, scale=3.0)
    c, a16, b16 = oracle.quantize(x, bits, g)
    xh = oracle.dequantize(c, a16, b16, g).astype(np.float64)
    a = oracle.f16_value(a16).astype(np.float64)[:, 0]
    b = oracle.f16_value(b16).astype(np.float64)[:, 0]
    mn, mx = x.min(1).astype(np.float64), x.max(1).astype(np.float64)
    bound = a / 2 + np.abs(b - mn) + np.abs(a * (2 ** bits - 1) - (mx - mn)) + \
        8 * np.spacing(np.abs(x).max(1).astype(np.float32)).astype(np.float64)
    err = np.abs(xh - x.astype(np.float64)).max(axis=1)
    assert np.all(err <= bound)


def test_extremes_map_to_end_codes():
    """For groups whose min and max are exactly representable in fp16 and whose
    range divides exactly, min -> 0 and max -> 2^N - 1."""
    for bits in (2, 4, 8):
        top = 2 ** bits - 1
        x = np.linspace(-4.0, -4.0 + top * 0.25, 32).astype(np.float32)  # alpha = 0.25 exactly
        x[3] = np.float32(-4.0)
        x[7] = np.float32(-4.0 + top * 0.25)
        c, a, b = oracle.quantize(x, bits, 32)
        assert oracle.f16_value(a)[0] == np.float32(0.25)
        assert c.min() == 0 and c.max() == top
        assert c[3] == 0 and c[7] == top


def test_power_of_two_scaling_commutes():
    """Every step of Eq. 1 commutes exactly with scaling by 2^k (no fp16
    subnormals or overflow involved), so codes are unchanged and alpha, beta
    scale by 2^k."""
    rng = np.random.default_rng(11)
    x = rng.standard_normal((500, 64)).astype(np.float32)
    for k in (-3, 2, 5):
        s = np.float32(2.0 ** k)
        c0, a0, b0 = oracle.quantize(x, 2, 32)
        c1, a1, b1 = oracle.quantize(x * s, 2, 32)
        np.testing.assert_array_equal(c0, c1)
        np.testing.assert_array_equal(oracle.f16_value(a0) * s, oracle.f16_value(a1))
        np.testing.assert_array_equal(oracle.f16_value(b0) * s, oracle.f16_value(b1))


def test_int8_integer_groups_exact():
    """Integer groups spanning exactly 0..255 have alpha = 1, beta = 0 and
    reconstruct exactly at 8 bits."""
    rng = np.random.default_rng(3)
    x = rng.integers(0, 256, (200, 64)).astype(np.float32)
    x[:, 0], x[:, 1] = 0, 255
    c, a, b = oracle.quantize(x, 8, 64)
    np.testing.assert_array_equal(c.astype(np.float32), x)
    np.testing.assert_array_equal(oracle.dequantize(c, a, b, 64), x)


def test_groups_are_independent_and_contiguous():
    """Changing one group's values leaves the other groups' outputs unchanged."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal((10, 128)).astype(np.float32)
    y = x.copy()
    y[:, 32:64] *= np.float32(100)
    cx, ax, bx = oracle.quantize(x, 2, 32)
    cy, ay, by = oracle.quantize(y, 2, 32)
    keep = np.r_[0:32, 64:128]
    np.testing.assert_array_equal(cx[:, keep], cy[:, keep])
    np.testing.assert_array_equal(ax[:, [0, 2, 3]], ay[:, [0, 2, 3]])
    assert not np.array_equal(ax[:, 1], ay[:, 1])


@pytest.mark.parametrize("row", read_golden("cache_size_tables.txt"), ids=lambda r: r[0])
def test_cache_size_tables(row):
    """Table 2 / Table 3 cache sizes follow from the storage format at g = 64."""
    _, r, hi, lo, pct = row
    r, hi, lo = float(r), int(hi), int(lo)
    size = r * oracle.bits_per_element(hi, 64) / 16 + (1 - r) * oracle.bits_per_element(lo, 64) / 16
    assert math.floor(size * 100 + 0.5) == int(pct)


def test_memory_table_head_shapes():
    """Table 5's full-cache memory for batch 8, sequence 4K equals
    2 (K,V) x layers x KV heads x 128 x 4096 x 8 x 4 bytes with the model
    shapes our workloads use (Llama-2-7b 32 heads, 13b 40, Mistral 8 KV heads)."""
    def gb(layers, kv_heads):
        return 2 * layers * kv_heads * 128 * 4096 * 8 * 4 / 1e9
    assert round(gb(32, 32), 2) == 34.36
    assert round(gb(32, 8), 2) == 8.59
    assert round(gb(40, 40), 2) == 53.69
    assert round(gb(32, 32) * 0.25, 2) == 8.59 and round(gb(32, 32) * 0.2, 2) == 6.87


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_exact_quotient_ties_round_half_even(bits):
    """Eq. 1 on groups whose quotients (x - beta) / alpha are exact
    half-integers or one fp16 ulp from them: every code is the quotient taken
    in exact rational arithmetic, rounded half to even and clamped."""
    from fractions import Fraction
    from tests.quant_inputs import tie_rows
    rng = np.random.default_rng(100 + bits)
    x = tie_rows(rng, 24, bits, 32)
    c, a, b = oracle.quantize(x.astype(np.float32), bits, 32)
    al = a.view(np.float16).astype(np.float64)
    be = b.view(np.float16).astype(np.float64)
    top = (1 << bits) - 1
    ties = 0
    for r in range(x.shape[0]):
        for j in range(128):
            q = (Fraction(float(x[r, j])) - Fraction(be[r, j // 32])) / Fraction(al[r, j // 32])
            ties += q.denominator == 2
            assert int(c[r, j]) == min(max(round(q), 0), top), (r, j, q)
    assert ties > x.size // 3


def test_three_bit_packing_straddles_bytes():
    """3-bit codes packed least significant bits first across byte
    boundaries: the row's bit string read as one little-endian integer is
    sum_c code_c * 8**c (big-integer arithmetic, independent of the packer)."""
    rng = np.random.default_rng(7)
    codes = rng.integers(0, 8, size=(3, 128)).astype(np.uint8)
    packed = oracle.pack(codes, 3)
    assert packed.shape == (3, 48)
    for r in range(3):
        value = sum(int(c) << (3 * i) for i, c in enumerate(codes[r]))
        np.testing.assert_array_equal(packed[r], np.frombuffer(value.to_bytes(48, "little"), np.uint8))
    np.testing.assert_array_equal(oracle.unpack(packed, 3), codes)
    # the first eight codes 1..7, 0 give the 24-bit word 0x1F58D1
    first = np.array([[1, 2, 3, 4, 5, 6, 7, 0]], np.uint8)
    np.testing.assert_array_equal(oracle.pack(first, 3)[0], [0xD1, 0x58, 0x1F])
