"""Pins for the oracle's MXFP4 quantizer (CPU only).

Checks: the E8M0 decode of every code against torch's float8_e8m0fnu, one
hand-worked block per branch of the scale rule (written out below; our
construction, not a printed example), exact power-of-two invariance, a
scalar brute-force quantizer written with exact rationals, zero and tiny
blocks, the element error bound, and the MXFP4 GEMM in exact integer
arithmetic on a tiny shape.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import formats, linalg, mxfp4


def test_e8m0_decode_matches_torch():
    codes = np.arange(256, dtype=np.uint8)
    ours = mxfp4.e8m0_decode(codes)
    ref = torch.from_numpy(codes.copy()).view(torch.float8_e8m0fnu).float().double().numpy()
    assert np.isnan(ours[255]) and np.isnan(ref[255])
    assert np.array_equal(ours[:255], ref[:255])
    # and the closed form 2**(c - 127), from exact Python integers
    for c in (0, 1, 126, 127, 128, 254):
        assert Fraction(ours[c]) == (Fraction(2) ** (c - 127))


def _one_block(vals):
    x = np.zeros((1, 32), np.float32)
    x[0, : len(vals)] = vals
    q, s = mxfp4.quantize(x)
    return q[0], int(s[0, 0])


def test_hand_worked_blocks():
    # block maximum 6: shared exponent floor(log2 6) - 2 = 0, scale 1; the
    # elements are the E2M1 ties (0.25 -> 0, 0.75 -> 1, 1.25 -> 1, 1.75 -> 2,
    # 2.5 -> 2, 3.5 -> 4, 5 -> 4)
    x = [0, .25, .5, .75, 1, 1.25, 1.5, 1.75, 2, 2.5, 3, 3.5, 4, 5, 6, -6]
    q, s = _one_block(x)
    assert s == 127
    assert list(q[:16]) == [0, 0, 1, 2, 2, 2, 3, 4, 4, 4, 5, 6, 6, 6, 7, 15]
    assert not q[16:].any()
    # maximum 7 (and 7.99): exponent 0, the maximum saturates to 6
    q, s = _one_block([7.0, -3.0, 0.3])
    assert s == 127 and list(q[:3]) == [7, 8 | 5, 1]
    q, s = _one_block([np.float32(7.99)])
    assert s == 127 and q[0] == 7
    # maximum 8: exponent 1, scale 2: 8 -> 4, 3 -> 1.5, 0.5 -> 0.25 -> 0
    q, s = _one_block([8.0, 3.0, 0.5, -1.0])
    assert s == 128 and list(q[:4]) == [6, 3, 0, 8 | 1]
    # maximum 0.75: exponent floor(log2 0.75) - 2 = -3, scale 1/8: 0.75 -> 6, 0.1 -> 0.8 -> 1
    q, s = _one_block([0.75, np.float32(0.1), -0.75])
    assert s == 124 and list(q[:3]) == [7, 2, 15]


def test_zero_and_tiny_blocks():
    q, s = _one_block([])
    assert s == 0 and not q.any()
    # a subnormal fp32 maximum (2**-130): the exponent clamps at -127, and the
    # scaled value 2**-3 rounds to zero
    q, s = _one_block([np.float32(2.0 ** -130)])
    assert s == 0 and not q.any()
    # 2**-125: exponent -127 exactly, scaled value 4 -> code 6
    q, s = _one_block([np.float32(2.0 ** -125)])
    assert s == 0 and q[0] == 6


def test_power_of_two_invariance():
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((16, 128)) * np.exp(rng.uniform(-8, 8, (16, 1)))).astype(np.float32)
    q0, s0 = mxfp4.quantize(x)
    for k in (-20, -1, 1, 7, 40):
        q1, s1 = mxfp4.quantize((x * np.float32(2.0 ** k)).astype(np.float32))
        assert np.array_equal(q0, q1)
        assert np.array_equal(s1.astype(np.int64), s0.astype(np.int64) + k)


def _brute_block(vals):
    """Scalar MXFP4 block quantizer in exact rationals."""
    a = max(abs(Fraction(float(v))) for v in vals)
    if a == 0:
        e = -127
    else:
        m, ex = math.frexp(float(a))
        e = max(-127, min(127, (ex - 1) - 2))
    X = Fraction(2) ** e
    cands = [(Fraction(float(formats.E2M1_MAGNITUDES[i])), i) for i in range(8)]
    codes = []
    for v in vals:
        y = Fraction(float(v)) / X
        ay = min(abs(y), Fraction(6))
        best = min(cands, key=lambda c: (abs(ay - c[0]), c[1] % 2))   # nearest, ties to the even index
        i = best[1]
        codes.append((8 if (y < 0 and i > 0) else 0) | i)
    return codes, e + 127


@pytest.mark.parametrize("shape,seed", [((4, 64), 0), ((16, 128), 1), ((8, 96), 2)])
def test_brute_force_tiny(shape, seed):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(shape) * np.exp(rng.uniform(-4, 4, (shape[0], 1)))).astype(np.float32)
    x[0, :32] = 0                                  # a zero block
    x[1, 5] = np.float32(7.5) * np.max(np.abs(x[1, :32]))   # a saturating maximum
    q, s = mxfp4.quantize(x)
    for r in range(shape[0]):
        for b in range(shape[1] // 32):
            codes, sc = _brute_block(x[r, 32 * b: 32 * b + 32])
            assert list(q[r, 32 * b: 32 * b + 32]) == codes
            assert s[r, b] == sc


def test_codes_in_range_and_error_bound():
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((64, 256)) * 3).astype(np.float32)
    q, s = mxfp4.quantize(x)
    assert q.max() <= 15 and s.max() <= 254
    assert not np.any(q == 8)                      # no negative zero
    xh = mxfp4.dequantize(q, s)
    X = np.repeat(mxfp4.e8m0_decode(s), 32, axis=1)
    err = np.abs(x.astype(np.float64) - xh)
    y = np.abs(x.astype(np.float64)) / X
    assert np.all(err[y <= 6] <= X[y <= 6])        # the largest half-gap of E2M1 (on [4, 6]) is 1
    assert np.all(err < 2 * X)                     # saturation: |y| < 8


def test_gemm_exact_integer_arithmetic():
    """MXFP4 x MXFP4 products: 2 e2m1 values are integers, scales powers of two."""
    rng = np.random.default_rng(9)
    A = rng.standard_normal((3, 64)).astype(np.float32)
    W = (rng.standard_normal((5, 64)) * 0.05).astype(np.float32)
    qa, sa = mxfp4.quantize(A)
    qw, sw = mxfp4.quantize(W)
    y = linalg.gemm(mxfp4.dequantize(qa, sa), mxfp4.dequantize(qw, sw))
    two_e = [0, 1, 2, 3, 4, 6, 8, 12]
    for m in range(3):
        for n in range(5):
            tot = Fraction(0)
            for k in range(64):
                ia = (-1 if qa[m, k] & 8 else 1) * two_e[qa[m, k] & 7]
                iw = (-1 if qw[n, k] & 8 else 1) * two_e[qw[n, k] & 7]
                tot += Fraction(ia * iw, 4) * Fraction(2) ** (int(sa[m, k // 32]) + int(sw[n, k // 32]) - 254)
            assert Fraction(y[m, n]) == tot
