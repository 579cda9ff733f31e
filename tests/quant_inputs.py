"""Seeded quantizer inputs shared by the oracle pins and the GPU parity tests."""
import numpy as np


def tie_rows(rng, n, bits, group):
    """Groups whose quotients (x - beta) / alpha of Eq. 1 lie exactly on
    half-integers (three in five) or one fp16 ulp beside them: beta = 0 and
    alpha = m 2^e with m odd, so 1 / alpha is inexact in fp32 and a quotient
    taken through the reciprocal can land on either side of the tie."""
    top = (1 << bits) - 1
    ng = 128 // group
    m = rng.choice([3, 5, 7] if bits == 8 else [3, 5, 7, 9, 11, 13, 15], (n, ng, 1))   # top m < 2^11
    alpha = m * 2.0 ** rng.integers(-6, 1, (n, ng, 1))
    kmax = np.minimum(top, (2047 // m - 1) // 2 + 1)           # (2k + 1) m < 2^11: exact in fp16
    t = (np.floor(rng.random((n, ng, group)) * kmax) + 0.5) * alpha
    t[..., 0] = 0.0
    t[..., 1] = top * alpha[..., 0]
    assert (t.astype(np.float16).astype(np.float64) == t).all()
    t = t.astype(np.float16)
    step = rng.choice([-1, 0, 0, 0, 1], t.shape)
    step[..., :2] = 0
    t = np.where(step > 0, np.nextafter(t, np.float16(np.inf)), np.where(step < 0, np.nextafter(t, np.float16(-np.inf)), t))
    return t.reshape(n, 128)
