"""Element-wise error bounds for the GPU's fp32 sums (test infrastructure).

Every GEMM / GEMV of the hot path multiplies exactly representable operands
(dequantized NVFP4 / MXFP4 values in fp16 or fp8 MFMA inputs, fp16 table
entries against fp16-staged activations), so each product is exact and only
the fp32 accumulation rounds.  For a sum of K exact products p_k computed in
fp32 in any order, |fl(sum) - sum| <= (K - 1) u sum |p_k| with u = 2^-24
(round to nearest; a factor 2 covers hardware that truncates).  A constant
number of further fp32 roundings (global scale products, the split-K partial
sums, unscaling) adds a few u times the same magnitude.  Hence, per output
element,

    |y - y_ref| <= 2 (K + 8) 2^-24 sum_k |a_k w_k|            (fp32 outputs)

with sum_k |a_k w_k| taken from the oracle's dequantized operands.  A bf16
output rounds once more (half an ulp, at most 2^-9 relative to the fp32
value).  The batch activations of the decode GEMVs are staged in fp16 after
a power-of-two rescale; values more than 2^31 below the largest magnitude of
their slice become fp16 subnormals, truncated: an extra error of at most
2^-38 max|x| |w| per product.  PAPER_GRID weights fold the E4M3 block scale
into the fp16 operand: at most 2^-11 relative per weight.

The bound catches any wrong element, block or tile (errors of the order of
|y|), which the relative Frobenius check over a sample would average away.
"""
import numpy as np

U = 2.0 ** -24


def abs_products(a_hat, w_hat) -> np.ndarray:
    """sum_k |a[m, k]| |w[n, k]| in fp64 for a [M, K] and w [N, K]."""
    return np.abs(np.asarray(a_hat, np.float64)) @ np.abs(np.asarray(w_hat, np.float64)).T


def fp32_sum_bound(absprod, K: int) -> np.ndarray:
    return 2.0 * (K + 8) * U * np.asarray(absprod, np.float64)


def gemv_bound(x_f64, w_hat, K: int, folded_rel: float = 0.0) -> np.ndarray:
    """Bound for y[b, n] = sum_k x[b, k] w[n, k] with fp16-staged activations
    (subnormal truncation included) and, for PAPER_GRID, a relative error
    `folded_rel` per weight."""
    ap = abs_products(x_f64, w_hat)
    xmax = np.abs(x_f64).max(axis=1, keepdims=True)
    wmax = np.abs(np.asarray(w_hat, np.float64)).max(axis=1)[None, :]
    return fp32_sum_bound(ap, K) * (1.0 + folded_rel) + folded_rel * ap + K * 2.0 ** -38 * xmax * wmax


def assert_within(y, ref, bound, what: str, bf16: bool = False) -> None:
    """|y - ref| <= bound element by element (bf16 outputs: plus the output
    rounding, 2^-9 of |ref| + bound, taken as 2^-8 for safety)."""
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    bound = np.asarray(bound, np.float64)
    if bf16:
        bound = bound + 2.0 ** -8 * (np.abs(ref) + bound)
    err = np.abs(y - ref)
    bad = err > bound
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} elements beyond the element-wise bound; "
                             f"first at {idx.tolist()}: err {err[bad][:5]} bound {bound[bad][:5]}")
