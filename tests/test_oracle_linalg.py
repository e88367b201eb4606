"""Pins for the oracle's fp64 GEMM / GEMV (CPU only).

Exact rational triple loops on tiny non-square shapes (a transposed operand
or a dropped G fails them), one-hot selections, and the exact special case
with unit scales, where every partial sum is a multiple of 1/4.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import formats, linalg, lut, nvfp4
from synth import bf16_bits_from_f32


def _rational_gemm(A, W):
    M, K = A.shape
    N = W.shape[0]
    return [[sum(Fraction(float(A[m, k])) * Fraction(float(W[n, k])) for k in range(K))
             for n in range(N)] for m in range(M)]


def test_nvfp4_gemm_matches_rational_triple_loop():
    rng = np.random.default_rng(30)
    M, N, K = 3, 5, 48
    X = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    qa, ca, Ga = nvfp4.quantize_dynamic(X)
    qw, cw, Gw = nvfp4.quantize_dynamic(W)
    Y = linalg.nvfp4_gemm(qa, ca, Ga, qw, cw, Gw)
    assert Y.shape == (M, N)
    A = nvfp4.dequantize(qa, ca, Ga)
    B = nvfp4.dequantize(qw, cw, Gw)
    ref = _rational_gemm(A, B)
    mag = _rational_gemm(np.abs(A), np.abs(B))
    for m in range(M):
        for n in range(N):
            # fp64 summation error bound: K * 2**-53 * sum |a_k w_k|
            assert abs(Fraction(float(Y[m, n])) - ref[m][n]) <= mag[m][n] * K * Fraction(1, 2 ** 53)


def test_gemm_exact_with_unit_scales():
    """All scales 1 and G = 1: the fp64 result equals the exact sum."""
    rng = np.random.default_rng(31)
    M, N, K = 4, 6, 64
    qa = rng.integers(0, 16, (M, K)).astype(np.uint8)
    qw = rng.integers(0, 16, (N, K)).astype(np.uint8)
    ones_a = np.full((M, K // 16), 0x38, np.uint8)
    ones_w = np.full((N, K // 16), 0x38, np.uint8)
    Y = linalg.nvfp4_gemm(qa, ones_a, 1.0, qw, ones_w, 1.0)
    ref = _rational_gemm(formats.e2m1_decode(qa), formats.e2m1_decode(qw))
    assert all(Fraction(float(Y[m, n])) == ref[m][n] for m in range(M) for n in range(N))


def test_one_hot_selects_rows_and_columns():
    rng = np.random.default_rng(32)
    A = rng.standard_normal((7, 32))
    W = np.zeros((3, 32))
    W[1, 5] = 1.0
    Y = linalg.gemm(A, W)
    assert np.array_equal(Y[:, 1], A[:, 5]) and not Y[:, 0].any() and not Y[:, 2].any()


def test_gemv_per_row_lut_rational():
    rng = np.random.default_rng(33)
    W = (rng.standard_normal((5, 64)) * 0.02).astype(np.float32)
    codes, table = lut.quantize_per_row(W, 3)
    x = bf16_bits_from_f32(rng.standard_normal((2, 64)).astype(np.float32))
    y = linalg.lut_gemv_per_row(x, codes, table)
    xv = formats.f64_from_bf16_bits(x)
    for b in range(2):
        for n in range(5):
            terms = [Fraction(float(xv[b, k])) * Fraction(float(table[n, codes[n, k]])) for k in range(64)]
            bound = sum(abs(t) for t in terms) * 64 * Fraction(1, 2 ** 53)
            assert abs(Fraction(float(y[b, n])) - sum(terms)) <= bound


def test_nvfp4a16_gemv_rational():
    """Weight-only NVFP4 GEMV against a loop over the format's definition:
    E2M1 value table, E4M3 decode, global scale."""
    rng = np.random.default_rng(35)
    W = (rng.standard_normal((4, 48)) * 0.02).astype(np.float32)
    q, c, G = nvfp4.quantize_dynamic(W)
    x = bf16_bits_from_f32(rng.standard_normal((2, 48)).astype(np.float32))
    y = linalg.nvfp4a16_gemv(x, q, c, G)
    e2m1 = [Fraction(v) for v in ("0", "1/2", "1", "3/2", "2", "3", "4", "6")]

    def e4m3(b):
        e, m = (int(b) >> 3) & 0xF, int(b) & 7
        return Fraction(m, 512) if e == 0 else Fraction(8 + m, 8) * Fraction(2) ** (e - 7)

    xv = formats.f64_from_bf16_bits(x)
    for b in range(2):
        for n in range(4):
            terms = []
            for k in range(48):
                code = int(q[n, k])
                w = (-1 if code & 8 else 1) * e2m1[code & 7] * e4m3(c[n, k // 16]) * Fraction(float(G))
                terms.append(Fraction(float(xv[b, k])) * w)
            bound = sum(abs(t) for t in terms) * 48 * Fraction(1, 2 ** 53)
            assert abs(Fraction(float(y[b, n])) - sum(terms)) <= bound


def test_gemv_paper_grid_rational():
    rng = np.random.default_rng(34)
    W = (rng.standard_normal((3, 32)) * 0.02).astype(np.float32)
    grid = lut.default_grid(3)
    codes, sb, G = lut.quantize_paper_grid(W, grid)
    x = bf16_bits_from_f32(rng.standard_normal((1, 32)).astype(np.float32))
    y = linalg.lut_gemv_paper(x, codes, sb, G, grid)
    xv = formats.f64_from_bf16_bits(x)
    d = formats.e4m3_decode(sb)
    for n in range(3):
        terms = [Fraction(float(xv[0, k])) * Fraction(float(grid[codes[n, k]])) *
                 Fraction(float(d[n, k // 16])) * Fraction(float(G)) for k in range(32)]
        bound = sum(abs(t) for t in terms) * 32 * Fraction(1, 2 ** 53)
        assert abs(Fraction(float(y[0, n])) - sum(terms)) <= bound


def test_silu_mul_values():
    """SwiGLU's silu(g) * u pinned by facts independent of the oracle's
    formula: other closed forms of the logistic function (the tanh form
    (1 + tanh(g/2)) / 2 for g >= 0, e^g / (1 + e^g) for g < 0, each free of
    cancellation on its side), the identity silu(g) - silu(-g) = g,
    silu(0) = 0, and the limits silu(g) -> g (g -> +inf) and -> 0 (g -> -inf)."""
    rng = np.random.default_rng(5)
    g = rng.standard_normal(1000) * 4
    u = rng.standard_normal(1000)
    sig = np.where(g >= 0, (1.0 + np.tanh(g / 2.0)) / 2.0, np.exp(np.minimum(g, 0)) / (1.0 + np.exp(np.minimum(g, 0))))
    other = g * sig * u
    out = linalg.silu_mul(g, u)
    assert np.max(np.abs(out - other) / np.maximum(np.abs(other), 1e-300)) < 1e-13
    ones = np.ones_like(g)
    assert np.allclose(linalg.silu_mul(g, ones) - linalg.silu_mul(-g, ones), g, rtol=0, atol=1e-13)
    assert linalg.silu_mul(np.array([0.0]), np.array([7.0]))[0] == 0.0
    big = linalg.silu_mul(np.array([60.0, -60.0]), np.array([1.0, 1.0]))
    assert big[0] == 60.0 and 0 > big[1] > -1e-20


def test_rel_fro():
    assert linalg.rel_fro(np.array([1.0, 2.0]), np.array([1.0, 2.0])) == 0.0
    assert abs(linalg.rel_fro(np.array([3.0, 4.0]) * 1.001, np.array([3.0, 4.0])) - 1e-3) < 1e-12


def test_elementwise_bound_holds_for_fp32_sums_and_catches_a_wrong_element():
    """The element-wise bound the GPU parity tests apply (tests/parity_bounds.py):
    an fp32 GEMM of exactly representable dequantized operands (NumPy float32
    matmul, any summation order) stays within it, and a single wrong output
    (one flipped code's worth) does not."""
    import parity_bounds as PB
    rng = np.random.default_rng(5)
    qa = rng.integers(0, 16, (24, 2048)).astype(np.uint8)
    qw = rng.integers(0, 16, (40, 2048)).astype(np.uint8)
    ca = rng.integers(0x30, 0x48, (24, 128)).astype(np.uint8)
    cw = rng.integers(0x30, 0x48, (40, 128)).astype(np.uint8)
    a_hat = nvfp4.dequantize(qa, ca, np.float32(0.01))
    w_hat = nvfp4.dequantize(qw, cw, np.float32(0.02))
    ref = linalg.gemm(a_hat, w_hat)
    y32 = np.matmul(a_hat.astype(np.float32), w_hat.astype(np.float32).T).astype(np.float64)
    bound = PB.fp32_sum_bound(PB.abs_products(a_hat, w_hat), 2048)
    PB.assert_within(y32, ref, bound, "fp32 matmul")
    bad = y32.copy()
    bad[3, 7] += 0.5 * abs(a_hat[3]).max() * abs(w_hat[7]).max()   # one product's worth of error
    with pytest.raises(AssertionError):
        PB.assert_within(bad, ref, bound, "perturbed")
