"""Pins for the oracle's LUT formats (CPU only).

PER_ROW: exact reproduction of rows with at most 2**b distinct values,
brute-force bin means in rational arithmetic, brute-force nearest codes,
monotone entries, the mean of equal-count bin means equals the row mean.
PAPER_GRID: the printed grids (tests/golden/paper_grids.txt), sign
absorption (the block maximum always normalizes to +6), zero blocks,
brute-force nearest grid level, and the printed LUT3 grid's optimality
claim (a constrained Lloyd-Max fit under N(0,1) lands on it).
"""
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import formats, lut, nvfp4

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _printed_grids():
    g = {}
    for line in open(os.path.join(GOLDEN, "paper_grids.txt")):
        if line.strip() and not line.startswith("#"):
            k, *v = line.split()
            g[k] = [float(a) for a in v]
    return g


def test_default_grids_are_the_printed_ones():
    g = _printed_grids()
    for bits, key in ((3, "LUT3"), (2, "LUT2")):
        d = lut.default_grid(bits).astype(np.float64)
        p = np.array(g[key])
        assert np.all(np.abs(d - p) <= np.abs(p) * 2.0 ** -11)    # fp16 rounding only
        assert 0.0 in d and 6.0 in d and np.all(np.diff(d) > 0)


@pytest.mark.parametrize("bits", [2, 3])
def test_per_row_exact_on_few_distinct_values(bits):
    rng = np.random.default_rng(20)
    nb = 1 << bits
    K = 64 * nb
    vals = np.sort(rng.normal(0, 0.02, nb)).astype(np.float16).astype(np.float32)
    row = rng.permutation(np.repeat(vals, K // nb)).astype(np.float32)
    codes, table = lut.quantize_per_row(row[None, :], bits)
    assert np.array_equal(table[0].astype(np.float32), vals)
    assert np.array_equal(lut.dequantize_per_row(codes, table)[0], row.astype(np.float64))


def _fp16_rne(x: Fraction) -> Fraction:
    if x == 0:
        return Fraction(0)
    s, a, e = (-1 if x < 0 else 1), abs(x), 0
    while a >= 2:
        a /= 2
        e += 1
    while a < 1:
        a *= 2
        e -= 1
    q = Fraction(2) ** (max(e, -14) - 10)
    n = abs(x) / q
    f = n.numerator // n.denominator
    r = n - f
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and f % 2):
        f += 1
    return s * f * q


@pytest.mark.parametrize("bits", [2, 3])
def test_per_row_brute_force(bits):
    rng = np.random.default_rng(21 + bits)
    N, K = 6, 96
    W = (rng.standard_normal((N, K)) * 0.02 * np.exp(0.3 * rng.standard_normal((N, 1)))).astype(np.float32)
    W[0, :10] = W[0, 10]                                    # ties across a bin boundary
    codes, table = lut.quantize_per_row(W, bits)
    nb = 1 << bits
    cnt = K // nb
    for n in range(N):
        srt = sorted(Fraction(float(v)) for v in W[n])
        # fp16 of the exact bin mean; the oracle divides the correctly rounded
        # fp64 sum in fp64 first, which agrees except within ~2**-40 of an fp16 midpoint
        means = [_fp16_rne(sum(srt[j * cnt:(j + 1) * cnt]) / cnt) for j in range(nb)]
        assert [Fraction(float(v)) for v in table[n]] == means
        for k in range(K):
            w = Fraction(float(W[n, k]))
            best = min(range(nb), key=lambda j: (abs(w - means[j]), j))   # ties -> lower index
            assert codes[n, k] == best


def test_per_row_invariants():
    rng = np.random.default_rng(23)
    W = (rng.standard_normal((32, 512)) * 0.02).astype(np.float32)
    for bits in (2, 3):
        codes, table = lut.quantize_per_row(W, bits)
        t = table.astype(np.float64)
        assert np.all(np.diff(t, axis=1) >= 0)
        assert codes.max() < (1 << bits)
        # equal-count bins: the mean of the bin means is the row mean (up to fp16 rounding)
        tol = np.abs(t).max(axis=1) * 2.0 ** -11
        assert np.all(np.abs(t.mean(axis=1) - W.astype(np.float64).mean(axis=1)) <= tol)
        # every weight is at least as close to its entry as to any other
        d = np.abs(W[..., None].astype(np.float64) - t[:, None, :])
        own = np.take_along_axis(d, codes[..., None].astype(np.int64), axis=-1)[..., 0]
        assert np.all(own <= d.min(axis=-1))


@pytest.mark.parametrize("bits", [2, 3])
def test_paper_grid_sign_absorption_and_zero_blocks(bits):
    rng = np.random.default_rng(24)
    grid = lut.default_grid(bits)
    top = int(np.argmax(grid))
    W = (rng.standard_normal((64, 256)) * 0.02).astype(np.float32)
    W[3, 32:48] = 0
    codes, sb, G = lut.quantize_paper_grid(W, grid)
    assert G == np.float32(np.float32(np.abs(W).max()) / np.float32(2688))
    blk = W.reshape(64, 16, 16)
    i_star = np.argmax(np.abs(blk), axis=-1)
    c_star = np.take_along_axis(codes.reshape(64, 16, 16), i_star[..., None], -1)[..., 0]
    nz = np.abs(blk).max(-1) > 0
    assert np.all(c_star[nz] == top)                       # block maximum -> +6
    neg = np.take_along_axis(blk, i_star[..., None], -1)[..., 0] < 0
    assert np.all(((sb & 0x80) != 0) == (neg & nz))       # the scale carries the sign
    assert sb[3, 2] == 0 and np.all(codes[3, 32:48] == lut.zero_level(grid))


@pytest.mark.parametrize("bits", [2, 3])
def test_paper_grid_brute_force(bits):
    rng = np.random.default_rng(25)
    grid = lut.default_grid(bits)
    gF = [Fraction(float(g)) for g in grid.astype(np.float64)]
    W = (rng.standard_normal((4, 64)) * 0.05).astype(np.float32)
    codes, sb, G = lut.quantize_paper_grid(W, grid)
    S = (formats.e4m3_decode(sb).astype(np.float32) * G).astype(np.float32)
    for n in range(4):
        for k in range(64):
            y = Fraction(float(np.float32(W[n, k] / S[n, k // 16])))
            best = min(range(len(gF)), key=lambda j: (abs(y - gF[j]), j))
            assert codes[n, k] == best
    wh = lut.dequantize_paper_grid(codes, sb, G, grid)
    # normalized values lie in [-6.4, 6.4] (E4M3 rounding of the scale is within 1/16);
    # the error is at most the largest distance from that interval to the grid, times |S|
    g = grid.astype(np.float64)
    bound = max(np.max(np.diff(g)) / 2, 6.4 + g[0], 6.4 - g[-1])
    assert np.all(np.abs(wh - W).reshape(4, 4, 16).max(-1) <= bound * np.abs(S).astype(np.float64))


def _normalized_gaussian_blocks(n_blocks, seed=26):
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((n_blocks, 16)).astype(np.float32)
    G = np.float32(np.abs(W).max() / np.float32(2688))
    i_star = np.argmax(np.abs(W), axis=-1)
    w_star = W[np.arange(n_blocks), i_star]
    mag = formats.e4m3_rne_satfinite((np.abs(w_star) / np.float32(6 * G)).astype(np.float32))
    S = formats.e4m3_decode(mag) * np.sign(w_star) * float(G)
    return (W / S[:, None]).ravel()


def test_printed_lut3_grid_is_a_constrained_lloyd_max_fixed_point():
    """Paper: the grids minimize expected squared error over N(0,1) samples under
    two-level scaling, constrained to contain 0 and +6.  Starting from the printed
    LUT3 grid, constrained Lloyd iterations stay within 0.02 of it."""
    y = _normalized_gaussian_blocks(1 << 16)
    g = np.array(_printed_grids()["LUT3"])
    fixed = (g == 0) | (g == 6)
    for _ in range(60):
        mids = (g[:-1] + g[1:]) / 2
        idx = np.searchsorted(mids, y)
        for j in range(len(g)):
            if not fixed[j]:
                g[j] = y[idx == j].mean()
    assert np.max(np.abs(g - np.array(_printed_grids()["LUT3"]))) < 0.02


def test_autocast_reproduces_nvfp4_exact_tables():
    """LUT entries that NVFP4 represents exactly come back unchanged: every
    16-block holds the tensor's largest entry 6c with c = 7/256, so
    G = 6c/2688 = 2^-14 exactly, the block scale codes to 448 = 6c / (6G),
    S = 448 G = c, and each entry e*c (e an E2M1 magnitude) is a code."""
    rng = np.random.default_rng(50)
    c = np.float16(7.0 / 256.0)
    e2m1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])
    N, K = 6, 64
    table = np.zeros((N, 8), np.float16)
    for n in range(N):
        vals = np.sort(rng.choice(e2m1[:-1], 7, replace=True))
        table[n] = (np.concatenate([vals, [6.0]]) * np.float64(c)).astype(np.float16)
    codes = rng.integers(0, 8, (N, K)).astype(np.uint8)
    codes[:, ::16] = 7                                    # the largest entry in every block
    w_hat = lut.dequantize_per_row(codes, table)
    q, sc, G = lut.autocast_to_nvfp4(w_hat)
    assert G == np.float32(2.0 ** -14)
    assert np.all(sc == 0x7E)
    assert np.array_equal(nvfp4.dequantize(q, sc, G), w_hat)


def test_autocast_paper_grid_is_one_rounding():
    """PAPER_GRID entries grid * e4m3 * G are exact in fp64 and rounded once to
    fp32 before the NVFP4 rule; a given G is passed through."""
    W = (np.random.default_rng(51).standard_normal((8, 64)) * 0.02).astype(np.float32)
    grid = lut.default_grid(3)
    codes, sb, G = lut.quantize_paper_grid(W, grid)
    w_hat = lut.dequantize_paper_grid(codes, sb, G, grid)
    q, c, G2 = lut.autocast_to_nvfp4(w_hat, G=np.float32(0.001))
    q_ref, c_ref = nvfp4.quantize(w_hat.astype(np.float32), np.float32(0.001))
    assert G2 == np.float32(0.001) and np.array_equal(q, q_ref) and np.array_equal(c, c_ref)
