"""GPU parity at the benchmark's full sizes, through the C ABI.

* Decode: every linear of the 27B-class block (q/k/v 7168x5120, o 5120x5120,
  gate/up 34816x5120, down 5120x17408) packed on the GPU in LUT3 and LUT2
  (per-row tables) and multiplied at batch 1, 8 and 16 in the launch
  configuration of the decode sweep.  Per-row packing is row-independent, so
  sampled rows are checked bit for bit (codes and tables) against the
  oracle's packing of those rows, and the GEMV outputs of those rows against
  the oracle's fp64 GEMV (relative Frobenius error and an element-wise bound).
* Prefill: the W4A4 NVFP4 GEMM at M = 32768 on the 27B down-projection shape
  (K = 17408, N = 5120) and its MXFP4 variant, sampled rows and columns.
* The 27B block chained at M = 4096, checked per step (the oracle consumes the
  GPU's own intermediate codes): q/k/v (bf16 out), o (NVFP4 requantization
  with a static scale), gate/up (SwiGLU, NVFP4), down (bf16 out).
* The fallback GEMV kernel (activations too long for the one-launch kernel's
  LDS staging) in both table modes.

Inputs are the seeded synthetic tensors of synth/; no expected value comes
from the GPU except the intermediates that the per-step checks hand on.
"""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import dq_layout as L  # noqa: E402
import parity_bounds as PB  # noqa: E402
from test_gpu_epilogue import tolerant_match  # noqa: E402

import synth  # noqa: E402
from oracle import formats, linalg, lut, mxfp4, nvfp4  # noqa: E402

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


def g_dev(G):
    return dev(np.array([G], np.float32))


def say(*a):
    print(*a, flush=True)


def nvfp4_rows(t, rows):
    """Logical codes and scales of the given rows of a tiled NVFP4 tensor,
    copying only their 32-row tile rows to the host."""
    TC = (t.cols + 63) // 64
    TR = (t.rows + 31) // 32
    sel = torch.from_numpy(np.asarray(rows) // 32).cuda()
    cb = host(t.codes[: TR * TC * 1024].view(TR, TC * 1024)[sel]).reshape(-1)
    sb = host(t.scales[: TR * TC * 128].view(TR, TC * 128)[sel]).reshape(-1)
    q, c, _, _ = L.nvfp4_unpack(cb, sb, len(rows) * 32, t.cols)
    pick = np.arange(len(rows)) * 32 + np.asarray(rows) % 32
    return q[pick], c[pick]


STACK = synth.STACK_27B_M32768
BLOCK = synth.BLOCK_27B_M4096
LAYERS = {l.name: l for l in STACK.layers}


def sample_rows(n, count, seed):
    """Sorted sample of rows including the first, the last and the first row
    of the last 16-row tile."""
    rng = np.random.default_rng(seed)
    r = set(rng.choice(n, count, replace=False).tolist()) | {0, n - 1, (n - 1) // 16 * 16}
    return np.array(sorted(r))


_W_CACHE = {}


def layer_weight(name):
    if name not in _W_CACHE:
        _W_CACHE.clear()
        _W_CACHE[name] = synth.layer_weight(STACK, LAYERS[name])
    return _W_CACHE[name]


# ---------------------------------------------------------------- decode, 27B block
@pytest.mark.parametrize("bits", [3, 2])
@pytest.mark.parametrize("name", ["qkv", "o", "gate_up", "down"])
def test_lut_gemv_27b_block(name, bits):
    layer = LAYERS[name]
    N, K = layer.n, layer.k
    say("lut 27b", name, N, K, "bits", bits)
    w = layer_weight(name)
    Wq = dq.dq_pack_lut3(dev(w), bits=bits, mode=dq.LUT_PER_ROW)
    rows = sample_rows(N, 160, 200 + bits)
    codes_ref, table_ref = lut.quantize_per_row(w[rows], bits)
    codes = L.lut_codes_unpack(host(Wq.codes), N, K, bits)[rows]
    table = host(Wq.lut).view(np.uint16)[: N * (1 << bits)].reshape(N, 1 << bits)[rows]
    assert np.array_equal(table, table_ref.view(np.uint16)), "LUT entries differ"
    assert np.array_equal(codes, codes_ref), f"codes differ at {np.argwhere(codes != codes_ref)[:5]}"
    w_hat = lut.dequantize_per_row(codes_ref, table_ref)
    for B in (1, 8, 16):
        xb = synth.decode_x(STACK, K, B)
        x = bf16_dev(xb)
        ws_n = dq.dq_decode_gemv_workspace_size(B, Wq)
        ws = torch.empty(max(ws_n, 16), dtype=torch.uint8, device="cuda")
        y = host(dq.dq_decode_gemv(x, Wq, out_kind=dq.OUT_F32, workspace=ws))[:, rows]
        ref = linalg.lut_gemv_per_row(xb, codes_ref, table_ref)
        err = linalg.rel_fro(y, ref)
        say(f"  B={B} rel_fro {err:.2e}")
        assert err <= TOL
        PB.assert_within(y, ref, PB.gemv_bound(formats.f64_from_bf16_bits(xb), w_hat, K), f"{name} lut{bits} B={B}")
        if B == 8:
            yb = host(dq.dq_decode_gemv(x, Wq, out_kind=dq.OUT_BF16, workspace=ws).float())[:, rows]
            assert linalg.rel_fro(yb, formats.bf16_rne_from_f64(ref)) <= TOL
            PB.assert_within(yb, ref, PB.gemv_bound(formats.f64_from_bf16_bits(xb), w_hat, K),
                             f"{name} lut{bits} B={B} bf16", bf16=True)


# ---------------------------------------------------------------- prefill GEMM at M = 32768
def _calibrated_scale(cfg, K):
    calib = synth.prefill_x(cfg, K, m=2048, calib=True)
    return nvfp4.global_scale(nvfp4.amax(formats.f32_from_bf16_bits(calib)))


@pytest.fixture(scope="module")
def stack_prefill():
    layer = LAYERS["down"]
    say("M = 32768 prefill: generating X [32768, 17408] and W [5120, 17408]")
    w = synth.layer_weight(STACK, layer)
    xb = synth.prefill_x(STACK, layer.k)
    return w, xb, _calibrated_scale(STACK, layer.k)


def test_nvfp4_gemm_m32768_sampled(stack_prefill):
    """The NVFP4 prefill GEMM of the decode-sweep workload (M = 32768 tokens on
    the 27B down-projection), as the benchmark runs it: static-scale
    activation quantization, then the GEMM with bf16 output."""
    w, xb, G_x = stack_prefill
    M, K = xb.shape
    N = w.shape[0]
    W = dq.dq_pack_nvfp4(dev(w))
    A = dq.dq_quantize_act_nvfp4(bf16_dev(xb), G_static=g_dev(G_x))
    Y = dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_BF16)
    rng = np.random.default_rng(301)
    rows = np.sort(np.concatenate([rng.choice(M, 14, replace=False), [0, M - 1]]))
    cols = np.sort(np.concatenate([rng.choice(N, 510, replace=False), [0, N - 1]]))
    qa, ca, _ = nvfp4.quantize_bf16_activations(xb[rows], G_x)
    qa_g, ca_g = nvfp4_rows(A, rows)
    assert np.array_equal(qa_g, qa) and np.array_equal(ca_g, ca), "activation codes differ"
    Gw = nvfp4.global_scale(nvfp4.amax(w))
    assert host(W.G)[0] == Gw
    qw, cw = nvfp4.quantize(w[cols], Gw)
    a_hat, w_hat = nvfp4.dequantize(qa, ca, G_x), nvfp4.dequantize(qw, cw, Gw)
    ref = linalg.gemm(a_hat, w_hat)
    y = host(Y[torch.from_numpy(rows).cuda()][:, torch.from_numpy(cols).cuda()].float())
    err = linalg.rel_fro(y, formats.bf16_rne_from_f64(ref))
    say("  nvfp4 M=32768 sampled rel_fro", err)
    assert err <= TOL
    PB.assert_within(y, ref, PB.fp32_sum_bound(PB.abs_products(a_hat, w_hat), K), "nvfp4 gemm M=32768", bf16=True)


def test_mxfp4_gemm_m32768_sampled(stack_prefill):
    w, xb, _ = stack_prefill
    M, K = xb.shape
    N = w.shape[0]
    Wm = dq.dq_pack_mxfp4(dev(w))
    Am = dq.dq_quantize_act_mxfp4(bf16_dev(xb))
    Y = dq.dq_prefill_gemm_mxfp4(Am, Wm, out_kind=dq.OUT_BF16)
    rng = np.random.default_rng(302)
    rows = np.sort(np.concatenate([rng.choice(M, 14, replace=False), [0, M - 1]]))
    cols = np.sort(np.concatenate([rng.choice(N, 510, replace=False), [0, N - 1]]))
    qa, ca = mxfp4.quantize_bf16_activations(xb[rows])
    qw, cw = mxfp4.quantize(w[cols])
    a_hat, w_hat = mxfp4.dequantize(qa, ca), mxfp4.dequantize(qw, cw)
    ref = linalg.gemm(a_hat, w_hat)
    y = host(Y[torch.from_numpy(rows).cuda()][:, torch.from_numpy(cols).cuda()].float())
    err = linalg.rel_fro(y, formats.bf16_rne_from_f64(ref))
    say("  mxfp4 M=32768 sampled rel_fro", err)
    assert err <= TOL
    PB.assert_within(y, ref, PB.fp32_sum_bound(PB.abs_products(a_hat, w_hat), K), "mxfp4 gemm M=32768", bf16=True)


# ---------------------------------------------------------------- the 27B block chained at M = 4096
def test_block_chain_27b_m4096_per_step():
    """q/k/v and o from quantized activations (o's input is the synthetic
    attention stand-in), o requantized to NVFP4 in its epilogue with a static
    scale and fed to gate/up (standing in for the residual and the norm),
    gate/up with SwiGLU requantized for down, down with bf16 output.  Each
    step on sampled rows and output blocks against the oracle, from the GPU's
    own input codes."""
    L3 = {l.name: l for l in BLOCK.layers}
    M = BLOCK.m
    rng = np.random.default_rng(303)
    rows = np.sort(np.concatenate([rng.choice(M, 6, replace=False), [0, M - 1]]))
    rows_t = torch.from_numpy(rows).cuda()

    def weight(name):
        w = synth.layer_weight(BLOCK, L3[name])
        return w, dq.dq_pack_nvfp4(dev(w))

    # q/k/v
    say("chain: qkv")
    xb = synth.prefill_x(BLOCK, 5120)
    G_x = _calibrated_scale(BLOCK, 5120)
    w_qkv, W_qkv = weight("qkv")
    A = dq.dq_quantize_act_nvfp4(bf16_dev(xb), G_static=g_dev(G_x))
    Y_qkv = dq.dq_prefill_gemm(W_qkv, A=A, out_kind=dq.OUT_BF16)
    cols = np.sort(rng.choice(L3["qkv"].n, 384, replace=False))
    qa, ca, _ = nvfp4.quantize_bf16_activations(xb[rows], G_x)
    G_qkv = nvfp4.global_scale(nvfp4.amax(w_qkv))
    qw, cw = nvfp4.quantize(w_qkv[cols], G_qkv)
    a_hat, w_hat = nvfp4.dequantize(qa, ca, G_x), nvfp4.dequantize(qw, cw, G_qkv)
    ref = linalg.gemm(a_hat, w_hat)
    y = host(Y_qkv[rows_t][:, torch.from_numpy(cols).cuda()].float())
    assert linalg.rel_fro(y, formats.bf16_rne_from_f64(ref)) <= TOL
    PB.assert_within(y, ref, PB.fp32_sum_bound(PB.abs_products(a_hat, w_hat), 5120), "chain qkv", bf16=True)
    del Y_qkv, W_qkv, w_qkv

    # o, with NVFP4 requantization for the next layer; its static output scale
    # is calibrated on the oracle's result for the sampled rows
    say("chain: o")
    ab = synth.attn_out_standin(BLOCK, M, 5120)
    G_a = nvfp4.global_scale(nvfp4.amax(formats.f32_from_bf16_bits(ab[:512])))
    w_o, W_o = weight("o")
    qa, ca, _ = nvfp4.quantize_bf16_activations(ab[rows], G_a)
    qw, cw, G_wo = nvfp4.quantize_dynamic(w_o)
    a_hat, w_hat = nvfp4.dequantize(qa, ca, G_a), nvfp4.dequantize(qw, cw, G_wo)
    ref = linalg.gemm(a_hat, w_hat)
    G_o = np.float32(nvfp4.global_scale(nvfp4.amax(ref)))
    Ao = dq.dq_quantize_act_nvfp4(bf16_dev(ab), G_static=g_dev(G_a))
    y32 = dq.dq_prefill_gemm(W_o, A=Ao, out_kind=dq.OUT_F32)
    Hq_o = dq.dq_prefill_gemm(W_o, A=Ao, out_kind=dq.OUT_NVFP4, G_out_static=g_dev(G_o))
    y32_rows = host(y32[rows_t])
    assert linalg.rel_fro(y32_rows, ref) <= TOL
    PB.assert_within(y32_rows, ref, PB.fp32_sum_bound(PB.abs_products(a_hat, w_hat), 5120), "chain o")
    # the epilogue requantizes exactly the fp32 values of the plain output
    q_o, c_o = nvfp4_rows(Hq_o, rows)
    q_ref, c_ref = nvfp4.quantize(y32_rows, G_o)
    assert np.array_equal(c_o, c_ref) and np.array_equal(q_o, q_ref), "o requantization differs"
    del y32, W_o, w_o

    # gate/up with SwiGLU, from the GPU's o codes
    say("chain: gate_up")
    w_gu, W_gu = weight("gate_up")
    F = L3["gate_up"].n // 2
    G_h = np.float32(0.05)
    Hq = dq.dq_prefill_gemm(W_gu, A=Hq_o, out_kind=dq.OUT_NVFP4, G_out_static=g_dev(G_h),
                            epilogue_flags=dq.EPI_SWIGLU)
    fblocks = np.sort(rng.choice(F // 16, 40, replace=False))
    G_gu = nvfp4.global_scale(nvfp4.amax(w_gu))
    wrows = (fblocks[:, None, None] * 32 + np.arange(2)[None, :, None] * 16 + np.arange(16)[None, None, :]).reshape(-1)
    qw, cw = nvfp4.quantize(w_gu[wrows], G_gu)
    yg = linalg.nvfp4_gemm(q_o, c_o, G_o, qw, cw, G_gu).reshape(len(rows), len(fblocks), 2, 16)
    h64 = linalg.silu_mul(yg[:, :, 0, :], yg[:, :, 1, :]).reshape(len(rows), -1)
    q_h, c_h = nvfp4_rows(Hq, rows)
    fcols = (fblocks[:, None] * 16 + np.arange(16)[None, :]).reshape(-1)
    n_s, n_q = tolerant_match(q_h[:, fcols], c_h[:, fblocks], h64, G_h, rel=1e-5)
    say("  gate_up boundary differences: scales", n_s, "codes", n_q)
    assert n_s + n_q <= 4
    del W_gu, w_gu

    # down from the GPU's SwiGLU codes
    say("chain: down")
    w_dn, W_dn = weight("down")
    Y = dq.dq_prefill_gemm(W_dn, A=Hq, out_kind=dq.OUT_BF16)
    ncols = np.sort(rng.choice(L3["down"].n, 256, replace=False))
    G_dn = nvfp4.global_scale(nvfp4.amax(w_dn))
    qw, cw = nvfp4.quantize(w_dn[ncols], G_dn)
    a_hat, w_hat = nvfp4.dequantize(q_h, c_h, G_h), nvfp4.dequantize(qw, cw, G_dn)
    ref = linalg.gemm(a_hat, w_hat)
    y = host(Y[rows_t][:, torch.from_numpy(ncols).cuda()].float())
    err = linalg.rel_fro(y, formats.bf16_rne_from_f64(ref))
    say("  down rel_fro", err)
    assert err <= TOL
    PB.assert_within(y, ref, PB.fp32_sum_bound(PB.abs_products(a_hat, w_hat), 17408), "chain down", bf16=True)


# ---------------------------------------------------------------- the fallback GEMV kernel
@pytest.mark.parametrize("mode", [0, 1])
def test_lut_gemv_long_rows_fallback(mode):
    """K = 73728: batch-1 activations no longer fit the one-launch kernel's LDS
    staging, so the GEMV runs the piecewise kernel.  PER_ROW weights are
    packed on the host (the GPU packer sorts rows of at most 32768); the
    PAPER_GRID weights by the GPU packer."""
    N, K, B = 48, 73728, 1
    w = synth.random_f32(310 + mode, (N, K), 0.02)
    xb = synth.random_bf16(312, (B, K), outlier_frac=0.005, outlier_factor=30)
    if mode == dq.LUT_PER_ROW:
        codes, table = lut.quantize_per_row(w, 3)
        Wq = dq.LutWeight.empty(N, K, 3, dq.LUT_PER_ROW)
        cb = L.lut_codes_pack(codes, 3)
        Wq.codes[: cb.size].copy_(dev(cb))
        Wq.lut[: table.size].copy_(dev(table.view(np.int16).reshape(-1)))
        ref = linalg.lut_gemv_per_row(xb, codes, table)
        w_hat, folded = lut.dequantize_per_row(codes, table), 0.0
    else:
        grid = lut.default_grid(3)
        codes, sb, G = lut.quantize_paper_grid(w, grid)
        Wq = dq.dq_pack_lut3(dev(w), bits=3, mode=dq.LUT_PAPER_GRID)
        assert np.array_equal(L.lut_codes_unpack(host(Wq.codes), N, K, 3), codes)
        ref = linalg.lut_gemv_paper(xb, codes, sb, G, grid)
        w_hat, folded = lut.dequantize_paper_grid(codes, sb, G, grid), 2.0 ** -11
    y = host(dq.dq_decode_gemv(bf16_dev(xb), Wq))
    err = linalg.rel_fro(y, ref)
    say("  fallback rel_fro", err)
    assert err <= TOL
    PB.assert_within(y, ref, PB.gemv_bound(formats.f64_from_bf16_bits(xb), w_hat, K, folded), "fallback gemv")
