"""GPU parity of the GEMM epilogues (requantization to NVFP4 for the next
layer, and SwiGLU between gate/up and down), through the C ABI.

* NVFP4 output: the epilogue quantizes exactly the fp32 values the plain
  fp32 output of the same GEMM holds, so its codes and scales must equal the
  oracle quantizer applied to that fp32 output, bit for bit.
* SwiGLU: the fp32 output is compared with the oracle's fp64
  ``silu(g) * u`` of the GEMM's own fp32 gate and up values; its NVFP4
  requantization is matched against the oracle's quantization of the fp64
  values with a boundary tolerance: a scale or code may differ only where
  the fp64 value lies within 1e-5 (relative) of a rounding boundary (the
  GPU's fp32 exponential is not the fp64 one).
* A chain of two GEMMs is checked per step: the oracle consumes the GPU's
  own intermediate codes.

Inputs are seeded synthetic tensors; no expected value comes from the GPU
path except the intermediates that the per-step checks hand to the oracle.
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
from oracle import formats, linalg, nvfp4  # noqa: E402

pytestmark = pytest.mark.gpu

TOL = 1e-3
BOUNDARY_REL = 1e-5

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


def unpack(t, rows, cols):
    q, c, qfull, cfull = L.nvfp4_unpack(host(t.codes), host(t.scales), rows, cols)
    return q, c, qfull, cfull


def interleave_gate_up(wg, wu):
    """[gate; up] weight rows in the epilogue's order: groups of 16 gate rows
    and 16 up rows alternate."""
    F, K = wg.shape
    return np.stack([wg.reshape(F // 16, 16, K), wu.reshape(F // 16, 16, K)], axis=1).reshape(2 * F, K)


def operands(M, N, K, seed):
    xb = synth.random_bf16(seed, (M, K), outlier_frac=0.01, outlier_factor=20)
    w = synth.random_f32(seed + 1, (N, K), 0.02)
    A = dq.dq_quantize_act_nvfp4(bf16_dev(xb))
    W = dq.dq_pack_nvfp4(dev(w))
    return xb, w, A, W


def g_dev(G):
    return dev(np.array([G], np.float32))


# ---------------------------------------------------------------- E4M3 / E2M1 boundaries
_E4M3_POS = formats.E4M3_VALUES[formats.E4M3_VALUES >= 0].astype(np.float64)
_E4M3_MIDS = np.concatenate([[2.0 ** -10], (_E4M3_POS[:-1] + _E4M3_POS[1:]) / 2])
_E2M1_MIDS = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])


def _near(v, mids, rel):
    v = np.abs(np.asarray(v, np.float64))
    d = np.min(np.abs(v[..., None] - mids), axis=-1)
    return d <= rel * np.maximum(v, np.min(mids))


def tolerant_match(q, c, h64, G, rel=BOUNDARY_REL):
    """Codes q / scales c (GPU) against the oracle quantization of the fp64
    values h64: every difference must sit at a rounding boundary.  Returns
    the number of differing scales and codes."""
    G = np.float32(G)
    q_ref, c_ref = nvfp4.quantize(h64.astype(np.float32), G)
    rows, cols = h64.shape
    den = float(np.float32(np.float32(6.0) * G))
    a64 = np.abs(h64).reshape(rows, cols // 16, 16).max(-1)
    bad_scale = c != c_ref
    assert _near(a64[bad_scale] / den, _E4M3_MIDS, rel).all(), "a block scale differs away from a boundary"
    # codes: compare within blocks whose scales agree, against the fp64 ratio
    S = formats.e4m3_decode(c).astype(np.float64) * float(G)
    y = h64.reshape(rows, cols // 16, 16) / np.where(S == 0, 1.0, S)[..., None]
    diff = (q != q_ref).reshape(rows, cols // 16, 16) & ~bad_scale[..., None]
    assert _near(y[diff], _E2M1_MIDS, rel).all(), "a code differs away from an E2M1 midpoint"
    return int(bad_scale.sum()), int(diff.sum())


# ---------------------------------------------------------------- a4: NVFP4 requantization
REQ_SHAPES = [(128, 512, 512, 0.7), (300, 640, 1024, 1.3), (33, 96, 256, 1.0), (1, 16, 64, 0.5),
              (257, 1040, 128, 1.0)]


@pytest.mark.parametrize("M,N,K,gfac", REQ_SHAPES)
def test_nvfp4_output_equals_quantized_f32_output(M, N, K, gfac):
    """gfac < 1 makes the static output scale smaller than the data needs:
    the top blocks saturate (scale 448, codes 6)."""
    say("requant", M, N, K, gfac)
    _, _, A, W = operands(M, N, K, 21)
    y32 = host(dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_F32))
    G_out = np.float32(nvfp4.global_scale(nvfp4.amax(y32)) * np.float32(gfac))
    Yq = dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_NVFP4, G_out_static=g_dev(G_out))
    q, c, qfull, cfull = unpack(Yq, M, N)
    q_ref, c_ref = nvfp4.quantize(y32, G_out)
    assert np.array_equal(c, c_ref), f"scales differ at {np.argwhere(c != c_ref)[:5]}"
    assert np.array_equal(q, q_ref), f"codes differ at {np.argwhere(q != q_ref)[:5]}"
    assert not qfull[M:].any() and not qfull[:, N:].any()
    assert not cfull[M:].any() and not cfull[:, N // 16:].any()
    assert host(Yq.G)[0] == G_out
    if gfac < 1:
        assert (c == 0x7E).any()


def test_nvfp4_output_zero_and_empty():
    M, N, K = 64, 128, 256
    W = dq.dq_pack_nvfp4(dev(synth.random_f32(3, (N, K), 0.02)))
    A = dq.dq_quantize_act_nvfp4(bf16_dev(np.zeros((M, K), np.uint16)))
    Yq = dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_NVFP4, G_out_static=g_dev(0.25))
    _, _, qfull, cfull = unpack(Yq, M, N)
    assert not qfull.any() and not cfull.any()
    A0 = dq.dq_quantize_act_nvfp4(bf16_dev(np.zeros((0, K), np.uint16)))
    Y0 = dq.dq_prefill_gemm(W, A=A0, out_kind=dq.OUT_NVFP4, G_out_static=g_dev(0.5))
    assert Y0.rows == 0 and host(Y0.G)[0] == np.float32(0.5)


# ---------------------------------------------------------------- SwiGLU
SW_SHAPES = [(128, 256, 512), (100, 48, 96), (64, 1040, 256), (1, 16, 64)]


def _swiglu_case(M, F, K, seed):
    xb = synth.random_bf16(seed, (M, K), outlier_frac=0.01, outlier_factor=20)
    wg = synth.random_f32(seed + 1, (F, K), 0.02)
    wu = synth.random_f32(seed + 2, (F, K), 0.02)
    A = dq.dq_quantize_act_nvfp4(bf16_dev(xb))
    W = dq.dq_pack_nvfp4(dev(interleave_gate_up(wg, wu)))   # one tensor: gate and up share G_w
    y32 = host(dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_F32))      # [M, 2F], interleaved
    y = y32.reshape(M, F // 16, 2, 16)
    h64 = linalg.silu_mul(y[:, :, 0, :].reshape(M, F), y[:, :, 1, :].reshape(M, F))
    return A, W, h64


@pytest.mark.parametrize("M,F,K", SW_SHAPES)
def test_swiglu_f32_and_bf16(M, F, K):
    say("swiglu", M, F, K)
    A, W, h64 = _swiglu_case(M, F, K, 31)
    h = host(dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_F32, epilogue_flags=dq.EPI_SWIGLU))
    assert h.shape == (M, F)
    err = linalg.rel_fro(h, h64)
    say("  rel_fro", err)
    assert err <= 1e-6
    # h64 is silu(g) u in fp64 from the GPU's own fp32 gate / up sums, so only
    # the epilogue's fp32 arithmetic differs: exp, one add, one division and
    # two products, a few units in the last place relative to h (plus an
    # absolute floor for gate values so negative that exp overflows)
    bound = 2.0 ** -19 * np.abs(h64) + 2.0 ** -120
    PB.assert_within(h, h64, bound, "swiglu f32")
    hb = dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_BF16, epilogue_flags=dq.EPI_SWIGLU)
    hbf = host(hb.float()).astype(np.float64)
    assert linalg.rel_fro(hbf, formats.bf16_rne_from_f64(h64)) <= TOL
    PB.assert_within(hbf, h64, bound, "swiglu bf16", bf16=True)


@pytest.mark.parametrize("M,F,K", [(128, 256, 512), (64, 1040, 256), (300, 512, 1024)])
def test_swiglu_nvfp4(M, F, K):
    say("swiglu nvfp4", M, F, K)
    A, W, h64 = _swiglu_case(M, F, K, 41)
    h32 = host(dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_F32, epilogue_flags=dq.EPI_SWIGLU))
    G_out = nvfp4.global_scale(nvfp4.amax(h64))
    Hq = dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_NVFP4, G_out_static=g_dev(G_out),
                            epilogue_flags=dq.EPI_SWIGLU)
    q, c, qfull, cfull = unpack(Hq, M, F)
    # same fp32 values as the fp32 SwiGLU output: exact
    q32, c32 = nvfp4.quantize(h32, G_out)
    assert np.array_equal(c, c32) and np.array_equal(q, q32)
    # against the fp64 SwiGLU: differences only at rounding boundaries
    n_s, n_q = tolerant_match(q, c, h64, G_out)
    say("  boundary differences: scales", n_s, "codes", n_q)
    assert n_s + n_q <= max(2, 1e-4 * q.size)
    assert not qfull[M:].any() and not cfull[M:].any()


def test_swiglu_rejects_odd_groups():
    M, K = 32, 64
    A = dq.dq_quantize_act_nvfp4(bf16_dev(np.zeros((M, K), np.uint16)))
    W = dq.dq_pack_nvfp4(dev(synth.random_f32(5, (48, K), 0.02)))   # 48 rows: not gate/up groups of 16
    with pytest.raises(dq.DQError):
        dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_F32, epilogue_flags=dq.EPI_SWIGLU)


# ---------------------------------------------------------------- chains, per step
def test_chain_two_layers_per_step():
    """GEMM 1 (NVFP4 output) feeds GEMM 2 directly; the oracle computes step 2
    from the GPU's step-1 codes."""
    M, K1, N1, N2 = 192, 512, 768, 320
    _, _, A, W1 = operands(M, N1, K1, 51)
    y1 = host(dq.dq_prefill_gemm(W1, A=A, out_kind=dq.OUT_F32))
    G1 = nvfp4.global_scale(nvfp4.amax(y1))
    Y1q = dq.dq_prefill_gemm(W1, A=A, out_kind=dq.OUT_NVFP4, G_out_static=g_dev(G1))
    w2 = synth.random_f32(52, (N2, N1), 0.02)
    W2 = dq.dq_pack_nvfp4(dev(w2))
    y2 = host(dq.dq_prefill_gemm(W2, A=Y1q, out_kind=dq.OUT_F32))
    q1, c1, _, _ = unpack(Y1q, M, N1)
    qw, cw, Gw = nvfp4.quantize_dynamic(w2)
    ref = linalg.nvfp4_gemm(q1, c1, G1, qw, cw, Gw)
    err = linalg.rel_fro(y2, ref)
    say("  chain step 2 rel_fro", err)
    assert err <= TOL
    bound = PB.fp32_sum_bound(PB.abs_products(nvfp4.dequantize(q1, c1, G1), nvfp4.dequantize(qw, cw, Gw)), N1)
    PB.assert_within(y2, ref, bound, "chain step 2")
