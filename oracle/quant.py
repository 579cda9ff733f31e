"""Oracle: per-token grouped asymmetric N-bit quantizer (Section 3.1, Eq. 1).

Test infrastructure only.  Plain numpy; every operation below is one IEEE
fp32 operation (numpy float32 elementwise arithmetic is correctly rounded and
never contracted), so the reader can check each line against the paper.

Eq. 1 gives  x_hat = alpha * round((x - beta) / alpha) + beta  with
alpha = (max x - min x) / (2^N - 1) and beta = min x, taken per token and,
following Section 3.2, per group of channels inside one token and head.
Where the paper is silent the following readings are used:
  * "round" is round-half-to-even in fp32;
  * alpha and beta are stored as fp16 and the codes are computed from the
    stored (fp16-rounded) alpha and beta, so that decoding is self-consistent;
  * (x - beta) / alpha is a correctly rounded fp32 divide;
  * a group whose fp16 alpha is 0 (all values equal, or a range too small for
    fp16) gets all-zero codes and decodes to beta;
  * codes are clamped to [0, 2^N - 1] (needed because beta16 may exceed the
    true minimum after fp16 rounding);
  * groups are contiguous channel ranges [g*i, g*i + g) of one token and head;
  * packing is least-significant-bits first: channel c of an N-bit code lives
    in byte c*N/8, bits (c*N) mod 8 and up.
Fp16 rounding uses numpy's float32 -> float16 conversion (round to nearest
even), a library routine.
"""
from __future__ import annotations

import numpy as np


def f16_bits(x) -> np.ndarray:
    """fp32 -> fp16 (round to nearest even), returned as uint16 bit patterns."""
    return np.asarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)


def f16_value(bits) -> np.ndarray:
    """fp16 bit patterns -> exact fp32 values."""
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float32)


def quantize(x, bits: int, group: int):
    """Eq. 1 encode of the last axis of ``x`` (fp32) in groups of ``group``.

    Returns (codes uint8 [..., D], alpha16 uint16 [..., D/group],
    beta16 uint16 [..., D/group]).
    """
    x = np.asarray(x, dtype=np.float32)
    *lead, d = x.shape
    assert d % group == 0
    xg = x.reshape(*lead, d // group, group)
    mn = xg.min(axis=-1)
    mx = xg.max(axis=-1)
    top = np.float32(2 ** bits - 1)
    alpha32 = (mx - mn) / top                       # alpha of Eq. 1, fp32
    alpha16 = f16_bits(alpha32)                     # stored scale
    beta16 = f16_bits(mn)                           # stored zero point (= min)
    a = f16_value(alpha16)[..., None]
    b = f16_value(beta16)[..., None]
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.rint((xg - b) / a)                   # round((x - beta) / alpha)
    t = np.where(a == 0, np.float32(0), t)          # degenerate group
    codes = np.clip(t, np.float32(0), top).astype(np.uint8)
    return codes.reshape(*lead, d), alpha16, beta16


def encode(x, alpha16, beta16, bits: int) -> np.ndarray:
    """Eq. 1 codes of ``x`` (fp32, [..., D]) for given stored parameters
    alpha16, beta16 (uint16 fp16 bits broadcastable to x): the encode step of
    :func:`quantize` with the parameters supplied instead of derived."""
    x = np.asarray(x, dtype=np.float32)
    a = f16_value(alpha16)
    b = f16_value(beta16)
    top = np.float32(2 ** bits - 1)
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.rint((x - b) / a)                    # round((x - beta) / alpha)
    t = np.where(a == 0, np.float32(0), t)          # degenerate parameters
    return np.clip(t, np.float32(0), top).astype(np.uint8)


def quantize_channels(x_block, bits: int):
    """Eq. 1 per channel over a block of tokens (the per-channel key
    quantization of Appendix C): x_block fp32 [T, D] -> (codes uint8 [T, D],
    alpha16 uint16 [D], beta16 uint16 [D]), i.e. the per-token quantizer with
    the roles of token and channel exchanged (one group = one channel's T
    values)."""
    xt = np.asarray(x_block, dtype=np.float32).T             # [D, T]
    codes, a16, b16 = quantize(xt, bits, xt.shape[-1])
    return codes.T.copy(), a16[:, 0], b16[:, 0]


def dequantize(codes, alpha16, beta16, group: int) -> np.ndarray:
    """Eq. 1 decode: alpha * code + beta in fp32 (the product is exact for an
    fp16 alpha and a code below 256, so this has a single rounding)."""
    codes = np.asarray(codes)
    *lead, d = codes.shape
    c = codes.reshape(*lead, d // group, group).astype(np.float32)
    a = f16_value(alpha16)[..., None]
    b = f16_value(beta16)[..., None]
    return (a * c + b).reshape(*lead, d)


def pack(codes, bits: int) -> np.ndarray:
    """Pack N-bit codes along the last axis, least significant bits first:
    code c occupies bits [N c, N c + N) of the row's bit string, bit b of the
    string being bit b % 8 of byte b // 8 (so a 3-bit code may straddle two
    bytes)."""
    codes = np.asarray(codes, dtype=np.uint8)
    *lead, d = codes.shape
    assert (d * bits) % 8 == 0
    bitarr = np.zeros((*lead, d * bits), dtype=np.uint8)       # one entry per bit, LSB first
    for i in range(bits):
        bitarr[..., i::bits] = (codes >> i) & 1
    weights = (1 << np.arange(8)).astype(np.uint32)
    return (bitarr.reshape(*lead, d * bits // 8, 8).astype(np.uint32) * weights).sum(-1).astype(np.uint8)


def unpack(packed, bits: int) -> np.ndarray:
    """Inverse of :func:`pack`."""
    packed = np.asarray(packed, dtype=np.uint8)
    *lead, nb = packed.shape
    bitarr = ((packed[..., None] >> np.arange(8)) & 1).reshape(*lead, nb * 8)
    d = nb * 8 // bits
    out = np.zeros((*lead, d), dtype=np.uint32)
    for i in range(bits):
        out |= bitarr[..., i::bits][..., :d].astype(np.uint32) << i
    return out.astype(np.uint8)


def bits_per_element(bits: int, group: int) -> float:
    """Storage cost of one quantized element: the code plus its share of the
    fp16 scale and zero point of its group; fp16 storage costs 16 bits.  A
    per-channel group of ``group`` tokens costs the same share."""
    if bits == 16:
        return 16.0
    return bits + 32.0 / group
