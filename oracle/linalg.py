"""fp64 products over dequantized operands (oracle; test infrastructure).

The prefill GEMM of the paper's W4A4 NVFP4 path computes
``Y = X_hat @ W_hat^T`` over the dequantized activations and weights (App. A
"NVFP4"; App. C "Compute and timing scope").  The decode GEMV of the
weight-only LUT formats computes ``y = x @ W_hat^T`` with the bf16
activations left unquantized (Sec. 2.3; App. C "Kernel specification").

Here both are a float64 ``numpy.matmul`` (BLAS dgemm).  Every product of two
dequantized NVFP4 values (at most 6 and 4 significant bits), of two MXFP4
values (at most 2 significant bits each) and every
product of a bf16 value with an fp16 LUT entry is exact in fp64; only the
fp64 summation rounds.  Pins (tests/test_oracle_linalg.py): a triple loop
in exact rational arithmetic on tiny shapes, one-hot rows and columns, and
non-square shapes that catch a transposed operand.
"""
from __future__ import annotations

import numpy as np

from . import formats, lut, mxfp4, nvfp4


def gemm(a_hat, w_hat) -> np.ndarray:
    """``Y[m, n] = sum_k A[m, k] * W[n, k]`` in fp64."""
    return np.matmul(np.asarray(a_hat, np.float64), np.asarray(w_hat, np.float64).T)


def nvfp4_gemm(a_codes, a_scales, G_a, w_codes, w_scales, G_w) -> np.ndarray:
    return gemm(nvfp4.dequantize(a_codes, a_scales, G_a), nvfp4.dequantize(w_codes, w_scales, G_w))


def mxfp4_gemm(a_codes, a_scales, w_codes, w_scales) -> np.ndarray:
    return gemm(mxfp4.dequantize(a_codes, a_scales), mxfp4.dequantize(w_codes, w_scales))


def gemv_bf16(x_bits, w_hat) -> np.ndarray:
    """``y[b, n] = sum_k x[b, k] * W[n, k]`` with bf16 activations, fp64."""
    return gemm(formats.f64_from_bf16_bits(x_bits), w_hat)


def lut_gemv_per_row(x_bits, codes, table) -> np.ndarray:
    return gemv_bf16(x_bits, lut.dequantize_per_row(codes, table))


def lut_gemv_paper(x_bits, codes, scale_bytes, G, grid) -> np.ndarray:
    return gemv_bf16(x_bits, lut.dequantize_paper_grid(codes, scale_bytes, G, grid))


def nvfp4a16_gemv(x_bits, codes, scale_codes, G) -> np.ndarray:
    """Weight-only NVFP4 decode (Sec. 2.3, format disaggregation: 16-bit
    activations, NVFP4 weights): ``y[b, n] = sum_k x[b, k] * w_hat[n, k]`` with
    the NVFP4 dequantization of App. A, in fp64."""
    return gemv_bf16(x_bits, nvfp4.dequantize(codes, scale_codes, G))


def silu_mul(g, u) -> np.ndarray:
    """SwiGLU's ``silu(g) * u = g / (1 + exp(-g)) * u`` in fp64."""
    g = np.asarray(g, np.float64)
    return g / (1.0 + np.exp(-g)) * np.asarray(u, np.float64)


def rel_fro(y, y_ref) -> float:
    """Relative Frobenius error ``||y - y_ref|| / ||y_ref||``."""
    y = np.asarray(y, np.float64)
    r = np.asarray(y_ref, np.float64)
    den = np.linalg.norm(r)
    num = np.linalg.norm(y - r)
    return float(num / den) if den > 0 else float(num)
