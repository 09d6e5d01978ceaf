"""Constructed inputs of the activation codec whose codes are fixed by hand reasoning from the
codec's definition (q = clamp(floor(fma(x - m, s, u)), 0, 2^b - 1), u of flat index e from
Philox4x32-10, whose known answers pin the generator), shared by the oracle pins and the GPU
parity tests."""
from fractions import Fraction

import numpy as np

import oracle


def codec_uniform(seed, e):
    """u of flat index e: word e mod 4 of Philox4x32-10 at counter (e / 4 mod 2^32, e / 2^34, 0, 0),
    key (seed mod 2^32, seed / 2^32), top 24 bits times 2^-24."""
    out = oracle.philox4x32_10([(e // 4) & 0xFFFFFFFF, e >> 34, 0, 0], [seed & 0xFFFFFFFF, seed >> 32])
    return Fraction(int(out[e % 4]) >> 8, 1 << 24)


def flat_index_case(seed, n, F, G=64):
    """1 bit, every group holding a 0 (its first feature) and a 1 (its second), so m = 0, s = 1
    and the code is floor(fl(x + u)).  Every other feature is a probe: x = 1 - u_e (exact in fp32,
    u_e being a multiple of 2^-24) sums to exactly 1, code 1; one 2^-24 step lower sums to
    1 - 2^-24, code 0.  Returns (x, expected decoded values): a code read with r = 1, m = 0."""
    x = np.zeros((n, F), np.float32)
    want = np.zeros((n, F), np.float32)
    for i in range(n):
        for f in range(F):
            j = f % G
            if j == 0:
                continue
            if j == 1:
                x[i, f] = want[i, f] = 1.0
                continue
            e = i * F + f
            u = codec_uniform(seed, e)
            v = 1 - u if (e * 7 + i) % 3 else 1 - u - Fraction(1, 1 << 24)
            assert Fraction(float(np.float32(float(v)))) == v        # exact in fp32
            x[i, f] = float(v)
            want[i, f] = 1.0 if v + u == 1 else 0.0
    return x, want


def clamp_case(seed, tail=0):
    """8 bits, one group of 64 holding 0 and 255 (s = 1), the 255 at an element whose uniform is
    at least 1 - 2^-17: there 255 + u rounds to 256 in fp32 (the step between 128 and 256 is
    2^-16), and the code must still be 255.  Every other group is constant 0.  `tail` extra
    features make the row ragged.  Returns (x, e, expected decoded values)."""
    top = Fraction((1 << 24) - (1 << 7), 1 << 24)
    e = next(e for e in range(1 << 22) if codec_uniform(seed, e) >= top)
    assert float(np.float32(255.0) + np.float32(float(codec_uniform(seed, e)))) == 256.0
    F = (e // 64 + 1) * 64 + tail
    x = np.zeros((1, F), np.float32)
    x[0, e] = 255.0
    return x, e, x.copy()
