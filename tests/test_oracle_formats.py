"""Pins for the oracle's number formats (CPU only).

The oracle's codecs are checked against things other than themselves:
torch's float8_e4m3fn casts (a library routine), brute force in exact
rational arithmetic, and hand-worked values from tests/golden/.
"""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import formats

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _e4m3_all_values_exact():
    """All non-negative finite E4M3 values as Fractions, from the OCP definition."""
    vals = []
    for code in range(0x7F):
        e, m = code >> 3, code & 7
        if e == 0:
            vals.append(Fraction(m, 2 ** 9))
        else:
            vals.append((1 + Fraction(m, 8)) * Fraction(2) ** (e - 7))
    return vals


def _nearest_even_brute(t: Fraction, vals):
    best = None
    for i, v in enumerate(vals):
        d = abs(t - v)
        if best is None or d < best[0] or (d == best[0] and i % 2 == 0):
            best = (d, i)
    return best[1]


def test_e4m3_decode_all_codes_match_torch():
    codes = np.arange(256, dtype=np.uint8)
    ours = formats.e4m3_decode(codes)
    ref = torch.from_numpy(codes.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(ours[ok], ref[ok])
    assert formats.E4M3_VALUES[-1] == 448.0 and len(formats.E4M3_VALUES) == 127


def test_e4m3_hand_worked():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "e4m3_hand.txt"))
            if l.strip() and not l.startswith("#")]
    t = np.array([float(a) for a, _ in rows], dtype=np.float32)
    want = np.array([int(b, 16) for _, b in rows], dtype=np.uint8)
    assert np.array_equal(formats.e4m3_rne_satfinite(t), want)


def test_e4m3_matches_torch_cast_in_range():
    rng = np.random.default_rng(1)
    t = np.exp2(rng.uniform(-12, np.log2(448), 200_000)).astype(np.float32)
    # exact midpoints between neighbouring codes, and one fp32 ulp either side
    v = formats.E4M3_VALUES
    mids = ((v[:-1] + v[1:]) / 2).astype(np.float32)
    t = np.concatenate([t, mids, np.nextafter(mids, np.float32(0)),
                        np.nextafter(mids, np.float32(1e9)), v.astype(np.float32)])
    t = t[t <= 448]
    ours = formats.e4m3_rne_satfinite(t)
    ref = torch.from_numpy(t).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(ours, ref)


def test_e4m3_saturates_above_448():
    t = np.array([448.0, 449.0, 463.9, 464.0, 480.0, 1e6, 3e38], dtype=np.float32)
    assert np.all(formats.e4m3_rne_satfinite(t) == 0x7E)


def test_e4m3_brute_force_rational():
    vals = _e4m3_all_values_exact()
    rng = np.random.default_rng(2)
    t = np.exp2(rng.uniform(-11, 9.2, 400)).astype(np.float32)
    t = np.minimum(t, np.float32(448))
    got = formats.e4m3_rne_satfinite(t)
    for ti, gi in zip(t, got):
        assert gi == _nearest_even_brute(Fraction(float(ti)), vals)


E2M1 = [Fraction(0), Fraction(1, 2), Fraction(1), Fraction(3, 2), Fraction(2),
        Fraction(3), Fraction(4), Fraction(6)]


def test_e2m1_brute_force_rational():
    rng = np.random.default_rng(3)
    y = np.concatenate([rng.uniform(0, 7, 3000),
                        [float(a + b) / 2 for a, b in zip(E2M1[:-1], E2M1[1:])]]).astype(np.float32)
    got = formats.e2m1_rne_sat(y)
    for yi, gi in zip(y, got):
        t = min(Fraction(float(yi)), Fraction(6))
        assert gi == _nearest_even_brute(t, E2M1)


def test_e2m1_decode_grid():
    codes = np.arange(16, dtype=np.uint8)
    v = formats.e2m1_decode(codes)
    assert list(v[:8]) == [0, 0.5, 1, 1.5, 2, 3, 4, 6]
    assert list(v[8:]) == [-0.0, -0.5, -1, -1.5, -2, -3, -4, -6]


def _fp16_rne_fraction(x: Fraction) -> Fraction:
    """fp16 round-to-nearest-even of an exact rational (normal and subnormal range)."""
    if x == 0:
        return Fraction(0)
    s = -1 if x < 0 else 1
    a = abs(x)
    e = 0
    while a >= 2:
        a /= 2
        e += 1
    while a < 1:
        a *= 2
        e -= 1
    e = max(e, -14)                        # subnormals share the 2**-24 quantum
    q = Fraction(2) ** (e - 10)
    n = abs(x) / q
    f = n.numerator // n.denominator
    r = n - f
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and f % 2 == 1):
        f += 1
    return s * f * q


def test_fp16_from_f64_single_rounding():
    rng = np.random.default_rng(4)
    # values just above fp16 midpoints: a double rounding through fp32 would
    # land on the midpoint and then round to even (down for half of them).
    base = rng.uniform(-1000, 1000, 2000).astype(np.float16).astype(np.float64)
    ulp = np.abs(np.spacing(base.astype(np.float16)).astype(np.float64))
    mids = base + ulp / 2
    tricky = mids + np.abs(mids) * 2.0 ** -40
    x = np.concatenate([tricky, mids, rng.normal(0, 0.05, 2000), rng.normal(0, 1e-5, 500)])
    got = formats.fp16_from_f64(x).astype(np.float64)
    for xi, gi in zip(x, got):
        assert Fraction(float(gi)) == _fp16_rne_fraction(Fraction(float(xi)))


def test_bf16_rne_from_f64_matches_torch_for_f32_inputs():
    rng = np.random.default_rng(5)
    x = rng.normal(0, 3, 50_000).astype(np.float32)
    ours = formats.bf16_rne_from_f64(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ours, ref)


def test_bf16_bits_decode_matches_torch():
    bits = np.arange(0, 65536, 7, dtype=np.uint16)
    bits = bits[(bits & 0x7F80) != 0x7F80]      # finite only
    ours = formats.f64_from_bf16_bits(bits)
    ref = torch.from_numpy(bits.astype(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ours, ref)
