"""GPU parity of the MXFP4 W4A4 prefill variant against the CPU oracle.

Bars: codes and E8M0 scale codes bit-exact (oracle.mxfp4.quantize, the OCP MX
conversion); GEMM fp32 outputs within 1e-3 relative Frobenius error of the
fp64 product of the dequantized operands, bf16 outputs against that product
rounded to bf16.  Inputs are seeded synthetic tensors (synth/).
"""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import dq_layout as L  # noqa: E402
import parity_bounds as PB  # noqa: E402

import synth  # noqa: E402
from oracle import formats, linalg, mxfp4  # noqa: E402

pytestmark = pytest.mark.gpu

TOL = 1e-3

try:
    import paper_2609_26333_amd as dq
except ImportError:  # pragma: no cover
    dq = None


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if dq is None or not torch.cuda.is_available():
        pytest.skip("needs the built HIP library and a GPU")


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def bf16_dev(bits):
    return dev(np.asarray(bits, np.uint16).view(np.int16))


def say(*a):
    print(*a, flush=True)


def _check_mx(t, rows, cols, q_ref, s_ref):
    q, s, qfull, sfull = L.mxfp4_unpack(host(t.codes), host(t.scales), rows, cols)
    assert np.array_equal(s, s_ref), f"scale codes differ at {np.argwhere(s != s_ref)[:5]}"
    assert np.array_equal(q, q_ref), f"codes differ at {np.argwhere(q != q_ref)[:5]}"
    assert not qfull[rows:].any() and not qfull[:, cols:].any()
    assert not sfull[rows:].any() and not sfull[:, cols // 32:].any()


def _upload(q, s):
    rows, cols = q.shape
    cb, sb = L.mxfp4_pack(q, s)
    t = dq.MxFp4Tensor.empty(rows, cols)
    t.codes[: cb.size].copy_(dev(cb))
    t.scales[: sb.size].copy_(dev(sb))
    return t


ACT_SHAPES = [(128, 512, 0), (100, 96, 1), (1, 32, 2), (33, 1056, 3), (2048, 4096, 5)]


@pytest.mark.parametrize("M,K,seed", ACT_SHAPES)
def test_mx_quantize_act(M, K, seed):
    say("mx act", M, K)
    xb = synth.random_bf16(100 + seed, (M, K), outlier_frac=0.005, outlier_factor=30)
    q_ref, s_ref = mxfp4.quantize_bf16_activations(xb)
    _check_mx(dq.dq_quantize_act_mxfp4(bf16_dev(xb)), M, K, q_ref, s_ref)


@pytest.mark.parametrize("N,K,seed", [(512, 512, 0), (72, 96, 1), (12288, 4096, 2)])
def test_mx_pack_weights(N, K, seed):
    say("mx pack", N, K)
    w = synth.random_f32(110 + seed, (N, K), 0.02)
    q_ref, s_ref = mxfp4.quantize(w)
    _check_mx(dq.dq_pack_mxfp4(dev(w)), N, K, q_ref, s_ref)


def test_mx_pack_special_values():
    """Blocks that reach every branch of the conversion: all zero, subnormal
    maxima (exponent clamped at -127), maxima near the fp32 limit, exact
    powers of two, E2M1 midpoints after scaling (ties to even) and values that
    saturate at 6."""
    rng = np.random.default_rng(120)
    w = (rng.standard_normal((64, 320)) * 0.5).astype(np.float32)
    w[0, :32] = 0.0
    w[1, :32] = np.float32(2.0 ** -140) * rng.integers(-8, 9, 32).astype(np.float32)
    w[2, :32] = np.float32(3.0e38) * rng.uniform(-1, 1, 32).astype(np.float32)
    w[3, :32] = np.float32(2.0) ** rng.integers(-10, 10, 32).astype(np.float32)
    # block max 4 -> e = 0: every E2M1 midpoint (0.25, 0.75, ..., 5) and saturation
    w[4, :32] = np.array([4.0, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, -0.25, -0.75, -1.25, -1.75, -2.5, -3.5,
                          -5.0, 0.0, 7.9, -7.9, 6.0, -6.0, 0.1, -0.1, 0.5, 1.5, 3.0, 2.0, 1.0, 0.0, -0.0,
                          4.5, 5.5, 7.0], np.float32)
    w[5, :32] = np.float32(2.0 ** -149)      # the smallest subnormal
    w[6, :32] = -0.0
    q_ref, s_ref = mxfp4.quantize(w)
    _check_mx(dq.dq_pack_mxfp4(dev(w)), 64, 320, q_ref, s_ref)


def test_mx_quantize_empty():
    t = dq.dq_quantize_act_mxfp4(torch.empty((0, 64), dtype=torch.int16, device="cuda"))
    assert t.rows == 0
    t = dq.dq_pack_mxfp4(torch.empty((16, 0), dtype=torch.float32, device="cuda"))
    assert t.cols == 0


GEMM_SHAPES = [(128, 512, 512), (100, 72, 96), (1, 1, 32), (300, 520, 1024), (257, 33, 64), (64, 256, 4096),
               (520, 300, 2080)]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_mx_gemm_oracle_operands(M, N, K):
    """GEMM alone: operands quantized by the oracle, laid out on the host."""
    say("mx gemm", M, N, K)
    xb = synth.random_bf16(130, (M, K), outlier_frac=0.01, outlier_factor=20)
    w = synth.random_f32(131, (N, K), 0.02)
    qa, sa = mxfp4.quantize_bf16_activations(xb)
    qw, sw = mxfp4.quantize(w)
    ref = linalg.mxfp4_gemm(qa, sa, qw, sw)
    A, W = _upload(qa, sa), _upload(qw, sw)
    y = host(dq.dq_prefill_gemm_mxfp4(A, W, out_kind=dq.OUT_F32))
    err = linalg.rel_fro(y, ref)
    say("  rel_fro", err)
    assert err <= TOL
    bound = PB.fp32_sum_bound(PB.abs_products(mxfp4.dequantize(qa, sa), mxfp4.dequantize(qw, sw)), K)
    PB.assert_within(y, ref, bound, "mx gemm f32")
    yb = host(dq.dq_prefill_gemm_mxfp4(A, W, out_kind=dq.OUT_BF16).float()).astype(np.float64)
    assert linalg.rel_fro(yb, formats.bf16_rne_from_f64(ref)) <= TOL
    PB.assert_within(yb, ref, bound, "mx gemm bf16", bf16=True)


def test_mx_gemm_exact_small_scales():
    """Scale codes in a narrow range around 127: every partial sum is a
    multiple of 2^-8 well below 2^16, so the fp32 accumulation is exact and
    the result must equal the fp64 one bit for bit."""
    rng = np.random.default_rng(132)
    M, N, K = 96, 160, 512
    qa = rng.integers(0, 16, (M, K)).astype(np.uint8)
    qw = rng.integers(0, 16, (N, K)).astype(np.uint8)
    qa[qa == 8] = 0
    qw[qw == 8] = 0
    sa = rng.integers(124, 131, (M, K // 32)).astype(np.uint8)
    sw = rng.integers(124, 131, (N, K // 32)).astype(np.uint8)
    ref = linalg.mxfp4_gemm(qa, sa, qw, sw)
    y = host(dq.dq_prefill_gemm_mxfp4(_upload(qa, sa), _upload(qw, sw)))
    assert np.array_equal(y.astype(np.float64), ref)


def test_mx_gemm_end_to_end_8b_up_sampled_rows():
    """The 8B up-projection at full size (M=2048, K=4096, N=12288) through the
    GPU quantizers and GEMM in the benchmark's launch configuration; 48 rows
    of the bf16 output checked against the oracle."""
    cfg = synth.UP_8B_M2048
    layer = cfg.layers[0]
    w = synth.layer_weight(cfg, layer)
    xb = synth.prefill_x(cfg, layer.k)
    W = dq.dq_pack_mxfp4(dev(w))
    A = dq.dq_quantize_act_mxfp4(bf16_dev(xb))
    Y = dq.dq_prefill_gemm_mxfp4(A, W, out_kind=dq.OUT_BF16)
    rows = np.sort(np.random.default_rng(133).choice(cfg.m, 48, replace=False))
    qa, sa = mxfp4.quantize_bf16_activations(xb[rows])
    qw, sw = mxfp4.quantize(w)
    ref = linalg.mxfp4_gemm(qa, sa, qw, sw)
    y = host(Y[torch.from_numpy(rows).cuda()].float()).astype(np.float64)
    err = linalg.rel_fro(y, formats.bf16_rne_from_f64(ref))
    say("  8B up sampled rel_fro", err)
    assert err <= TOL
    bound = PB.fp32_sum_bound(PB.abs_products(mxfp4.dequantize(qa, sa), mxfp4.dequantize(qw, sw)), layer.k)
    PB.assert_within(y, ref, bound, "mx 8B up gemm", bf16=True)


@pytest.mark.parametrize("M,N,K", [(0, 64, 64), (64, 0, 64), (40, 24, 0)])
def test_mx_gemm_empty(M, N, K):
    A, W = dq.MxFp4Tensor.empty(M, K), dq.MxFp4Tensor.empty(N, K)
    y = dq.dq_prefill_gemm_mxfp4(A, W)
    assert tuple(y.shape) == (M, N)
    if M * N:
        assert not host(y).any()
