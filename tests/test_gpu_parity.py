"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars: codes, scales, LUT entries and global scales bit-exact; GEMM / GEMV
fp32 outputs within 1e-3 relative Frobenius error of the fp64 oracle (bf16
outputs against the oracle rounded to bf16) and, element by element, within
the fp32 summation bound of parity_bounds.py.  Inputs are seeded synthetic
tensors (synth/); no expected value comes from the GPU.
"""
import ctypes
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import dq_layout as L  # noqa: E402
import parity_bounds as PB  # noqa: E402

import synth  # noqa: E402
from oracle import formats, linalg, lut, nvfp4  # noqa: E402

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


# ---------------------------------------------------------------- a1: activation quantization
def _check_nvfp4(t, rows, cols, q_ref, c_ref, G_ref):
    q, c, qfull, cfull = L.nvfp4_unpack(host(t.codes), host(t.scales), rows, cols)
    assert np.array_equal(c, c_ref), f"scales differ at {np.argwhere(c != c_ref)[:5]}"
    assert np.array_equal(q, q_ref), f"codes differ at {np.argwhere(q != q_ref)[:5]}"
    # padding of the tiled layout holds zeros
    assert not qfull[rows:].any() and not qfull[:, cols:].any()
    assert not cfull[rows:].any() and not cfull[:, cols // 16:].any()
    assert host(t.G)[0] == np.float32(G_ref)


ACT_SHAPES = [(128, 512, 0), (100, 48, 1), (1, 16, 2), (33, 1040, 3), (2048, 4096, 5)]


@pytest.mark.parametrize("M,K,seed", ACT_SHAPES)
@pytest.mark.parametrize("static", [False, True])
def test_act_quant(M, K, seed, static):
    say("act_quant", M, K, seed, static)
    xb = synth.random_bf16(seed, (M, K), outlier_frac=0.01, outlier_factor=20)
    G_static = None
    if static:
        calib = synth.random_bf16(seed + 1000, (M, K), outlier_frac=0.01, outlier_factor=20)
        G_static = nvfp4.global_scale(nvfp4.amax(formats.f32_from_bf16_bits(calib)))
    q_ref, c_ref, G_ref = nvfp4.quantize_bf16_activations(xb, G_static)
    Gd = dev(np.array([G_static], np.float32)) if static else None
    t = dq.dq_quantize_act_nvfp4(bf16_dev(xb), G_static=Gd)
    _check_nvfp4(t, M, K, q_ref, c_ref, G_ref)


def test_act_quant_empty():
    t = dq.dq_quantize_act_nvfp4(bf16_dev(np.zeros((0, 64), np.uint16)))
    assert host(t.G)[0] == 1.0


def test_act_quant_midpoints_and_saturation():
    """Blocks whose elements sit exactly on E2M1 midpoints (and one bf16 ulp
    either side) after division by the block scale, plus saturated blocks."""
    rng = np.random.default_rng(7)
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
    rows = []
    for v in formats.E4M3_VALUES[8:126:3]:                # normal-range scales
        blk = np.concatenate([[6.0], mids, -mids, [0.0]]) * v
        rows.append(blk)
    x = np.array(rows, np.float32)
    xb = synth.bf16_bits_from_f32(x)
    nz = (xb & 0x7FFF) != 0                   # perturb nonzero magnitudes by one bf16 ulp
    up = np.where(nz, xb + 1, xb).astype(np.uint16)
    dn = np.where(nz, xb - 1, xb).astype(np.uint16)
    dn[:, 0] = xb[:, 0]
    up[:, 0] = xb[:, 0]
    sat = synth.bf16_bits_from_f32(np.float32(1e4) * rng.standard_normal((x.shape[0], 16)).astype(np.float32))
    allx = np.concatenate([np.concatenate([xb, up, dn, sat], axis=1)] * 2, axis=0)
    G = np.float32(1.0)
    q_ref, c_ref, _ = nvfp4.quantize_bf16_activations(allx, G)
    t = dq.dq_quantize_act_nvfp4(bf16_dev(allx), G_static=dev(np.array([G], np.float32)))
    _check_nvfp4(t, allx.shape[0], allx.shape[1], q_ref, c_ref, G)


# ---------------------------------------------------------------- a2: weight packing
@pytest.mark.parametrize("N,K,seed", [(512, 512, 0), (72, 48, 1), (12288, 4096, 2)])
def test_pack_nvfp4(N, K, seed):
    say("pack_nvfp4", N, K)
    w = synth.random_f32(seed, (N, K), 0.02)
    w *= np.exp(0.3 * synth.random_f32(seed + 1, (N, 1))).astype(np.float32)
    q_ref, c_ref, G_ref = nvfp4.quantize_dynamic(w)
    t = dq.dq_pack_nvfp4(dev(w))
    _check_nvfp4(t, N, K, q_ref, c_ref, G_ref)


def test_pack_nvfp4_shared_scale_and_fp32_midpoints():
    """A shared (overridden) global scale, and fp32 elements one ulp around
    every E2M1 midpoint (exercises the exact division)."""
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0], np.float32)
    rows = []
    for v in formats.E4M3_VALUES[8:126:5].astype(np.float32):
        base = np.concatenate([[6.0], mids, [-0.75, -5.0, 0.0, 1.0, 2.0, 3.0, 4.0, 0.5]]).astype(np.float32) * v
        rows += [base, np.nextafter(base, np.float32(np.inf)), np.nextafter(base, np.float32(-np.inf))]
    w = np.array(rows, np.float32)
    w[1::3, 0] = w[0::3, 0]
    w[2::3, 0] = w[0::3, 0]
    G = np.float32(1.0)
    q_ref, c_ref = nvfp4.quantize(w, G)
    t = dq.dq_pack_nvfp4(dev(w), G_override=dev(np.array([G], np.float32)))
    _check_nvfp4(t, w.shape[0], w.shape[1], q_ref, c_ref, G)


# ---------------------------------------------------------------- a3: GEMM
def _upload_nvfp4(q, c, G):
    rows, cols = q.shape
    t = dq.NvFp4Tensor.empty(rows, cols)
    cb, sb = L.nvfp4_pack(q, c)
    t.codes[: cb.size].copy_(dev(cb))
    t.scales[: sb.size].copy_(dev(sb))
    t.G.copy_(dev(np.array([G], np.float32)))
    return t


GEMM_SHAPES = [(128, 512, 512), (100, 72, 48), (1, 1, 16), (300, 520, 1024), (257, 33, 64), (64, 256, 4096),
               (200, 132, 128), (520, 392, 256)]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_gemm_oracle_operands(M, N, K):
    """GEMM alone: operands quantized by the oracle, laid out on the host."""
    say("gemm", M, N, K)
    xb = synth.random_bf16(11, (M, K), outlier_frac=0.01, outlier_factor=20)
    w = synth.random_f32(12, (N, K), 0.02)
    qa, ca, Ga = nvfp4.quantize_bf16_activations(xb)
    qw, cw, Gw = nvfp4.quantize_dynamic(w)
    ref = linalg.nvfp4_gemm(qa, ca, Ga, qw, cw, Gw)
    A, W = _upload_nvfp4(qa, ca, Ga), _upload_nvfp4(qw, cw, Gw)
    y = host(dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_F32))
    err = linalg.rel_fro(y, ref)
    say("  rel_fro", err)
    assert err <= TOL
    bound = PB.fp32_sum_bound(PB.abs_products(nvfp4.dequantize(qa, ca, Ga), nvfp4.dequantize(qw, cw, Gw)), K)
    PB.assert_within(y, ref, bound, "gemm f32")
    yb = dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_BF16)
    ybf = host(yb.float()).astype(np.float64)
    assert linalg.rel_fro(ybf, formats.bf16_rne_from_f64(ref)) <= TOL
    PB.assert_within(ybf, ref, bound, "gemm bf16", bf16=True)


def test_gemm_exact_unit_scales():
    """Unit block scales and G = 1: every partial sum is a multiple of 1/4 and
    small, so the fp32 result must equal the exact one."""
    rng = np.random.default_rng(13)
    M, N, K = 96, 160, 512
    qa = rng.integers(0, 16, (M, K)).astype(np.uint8)
    qw = rng.integers(0, 16, (N, K)).astype(np.uint8)
    qa[qa == 8] = 0
    qw[qw == 8] = 0
    ones_a = np.full((M, K // 16), 0x38, np.uint8)
    ones_w = np.full((N, K // 16), 0x38, np.uint8)
    ref = linalg.nvfp4_gemm(qa, ones_a, 1.0, qw, ones_w, 1.0)
    y = host(dq.dq_prefill_gemm(_upload_nvfp4(qw, ones_w, 1.0), A=_upload_nvfp4(qa, ones_a, 1.0)))
    assert np.array_equal(y.astype(np.float64), ref)


def test_gemm_end_to_end_8b_up_sampled_rows():
    """The 8B up-projection at full size (M=2048, K=4096, N=12288) through the
    GPU quantizers and GEMM in the benchmark's launch configuration; 48 rows
    of the output checked against the oracle."""
    cfg = synth.UP_8B_M2048
    layer = cfg.layers[0]
    w = synth.layer_weight(cfg, layer)
    xb = synth.prefill_x(cfg, layer.k)
    calib = synth.prefill_x(cfg, layer.k, calib=True)
    G_x = nvfp4.global_scale(nvfp4.amax(formats.f32_from_bf16_bits(calib)))
    W = dq.dq_pack_nvfp4(dev(w))
    A = dq.dq_quantize_act_nvfp4(bf16_dev(xb), G_static=dev(np.array([G_x], np.float32)))
    Y = dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_BF16)
    rows = np.sort(np.random.default_rng(14).choice(cfg.m, 48, replace=False))
    qa, ca, _ = nvfp4.quantize_bf16_activations(xb[rows], G_x)
    qw, cw, Gw = nvfp4.quantize_dynamic(w)
    ref = linalg.nvfp4_gemm(qa, ca, G_x, qw, cw, Gw)
    y = host(Y[torch.from_numpy(rows).cuda()].float()).astype(np.float64)
    err = linalg.rel_fro(y, formats.bf16_rne_from_f64(ref))
    say("  8B up sampled rel_fro", err)
    assert err <= TOL
    bound = PB.fp32_sum_bound(PB.abs_products(nvfp4.dequantize(qa, ca, G_x), nvfp4.dequantize(qw, cw, Gw)), layer.k)
    PB.assert_within(y, ref, bound, "8B up gemm", bf16=True)


@pytest.mark.parametrize("M,N,K,out", [(2048, 10240, 256, "bf16"), (1024, 20480, 128, "nvfp4"),
                                       (4096, 5120, 128, "swiglu")])
def test_gemm_tile_geometries_agree(M, N, K, out):
    """Shapes whose launch mixes 256x128 tiles (the leading columns) with
    128x128 tiles (the trailing columns, the last round): each output is
    accumulated over K in the same order in both, so slices of 32 rows (launched
    with 128x128 tiles only) equal the full call bit for bit; sampled rows of
    the full call also match the oracle."""
    say("geometries", M, N, K, out)
    xb = synth.random_bf16(90, (M, K), outlier_frac=0.01, outlier_factor=20)
    w = synth.random_f32(91, (N, K), 0.02)
    G_x = nvfp4.global_scale(nvfp4.amax(formats.f32_from_bf16_bits(xb)))
    Gd = dev(np.array([G_x], np.float32))
    W = dq.dq_pack_nvfp4(dev(w))
    kw = {}
    if out == "bf16":
        kw = dict(out_kind=dq.OUT_BF16)
    elif out == "nvfp4":
        kw = dict(out_kind=dq.OUT_NVFP4, G_out_static=dev(np.array([0.02], np.float32)))
    else:
        kw = dict(out_kind=dq.OUT_NVFP4, G_out_static=dev(np.array([0.02], np.float32)), epilogue_flags=dq.EPI_SWIGLU)
    Nout = N // 2 if out == "swiglu" else N

    def run(rows):
        A = dq.dq_quantize_act_nvfp4(bf16_dev(xb[rows]), G_static=Gd)
        Y = dq.dq_prefill_gemm(W, A=A, **kw)
        torch.cuda.synchronize()
        if out == "bf16":
            return host(Y.view(torch.int16))
        q, c, _, _ = L.nvfp4_unpack(host(Y.codes), host(Y.scales), len(rows), Nout)
        return np.concatenate([q, np.repeat(c, 16, axis=1)], axis=1)

    full = run(np.arange(M))
    for r0 in (0, M // 2 + 32, M - 32):
        rows = np.arange(r0, r0 + 32)
        assert np.array_equal(run(rows), full[rows]), f"rows {r0}..{r0 + 31} differ"
    if out == "bf16":
        rows = np.sort(np.random.default_rng(92).choice(M, 8, replace=False))
        qa, ca, _ = nvfp4.quantize_bf16_activations(xb[rows], G_x)
        qw, cw, Gw = nvfp4.quantize_dynamic(w)
        ref = linalg.nvfp4_gemm(qa, ca, G_x, qw, cw, Gw)
        y = formats.f64_from_bf16_bits(full[rows].view(np.uint16))
        err = linalg.rel_fro(y, formats.bf16_rne_from_f64(ref))
        say("  sampled rel_fro", err)
        assert err <= TOL
        bound = PB.fp32_sum_bound(PB.abs_products(nvfp4.dequantize(qa, ca, G_x), nvfp4.dequantize(qw, cw, Gw)), K)
        PB.assert_within(y, ref, bound, "geometries bf16", bf16=True)


@pytest.mark.parametrize("M,N,K", [(4096, 8192, 128), (4000, 8320, 192), (4096, 16640, 64), (4096, 8192, 80)])
def test_gemm_wide_tile_geometry_agrees(M, N, K):
    """bf16 outputs of grids of at least two rounds of 256x256 tiles run as
    one workgroup of four 128x128 wavefronts per compute unit (with a partial
    last round of 256x128 tiles in the trailing columns when N is not a whole
    number of rounds); 32-row slices launch the small-tile geometry.  Every
    output is accumulated over K in the same order, so the slices equal the
    full call bit for bit (ragged rows, edge columns and a K that ends inside
    a 64-column step included), and sampled rows of the full call match the
    oracle."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    assert ((M + 255) // 256) * ((N + 255) // 256) >= 2 * cus, "shape must take the 256x256 geometry"
    say("wide geometry", M, N, K)
    xb = synth.random_bf16(93, (M, K), outlier_frac=0.01, outlier_factor=20)
    w = synth.random_f32(94, (N, K), 0.02)
    G_x = nvfp4.global_scale(nvfp4.amax(formats.f32_from_bf16_bits(xb)))
    Gd = dev(np.array([G_x], np.float32))
    W = dq.dq_pack_nvfp4(dev(w))

    def run(rows):
        A = dq.dq_quantize_act_nvfp4(bf16_dev(xb[rows]), G_static=Gd)
        Y = dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_BF16)
        return host(Y.view(torch.int16))

    full = run(np.arange(M))
    for r0 in (0, 1056, M - 32):
        rows = np.arange(r0, r0 + 32)
        assert np.array_equal(run(rows), full[rows]), f"rows {r0}..{r0 + 31} differ"
    rows = np.sort(np.random.default_rng(95).choice(M, 6, replace=False))
    qa, ca, _ = nvfp4.quantize_bf16_activations(xb[rows], G_x)
    qw, cw, Gw = nvfp4.quantize_dynamic(w)
    ref = linalg.nvfp4_gemm(qa, ca, G_x, qw, cw, Gw)
    y = formats.f64_from_bf16_bits(full[rows].view(np.uint16))
    err = linalg.rel_fro(y, formats.bf16_rne_from_f64(ref))
    say("  sampled rel_fro", err)
    assert err <= TOL
    bound = PB.fp32_sum_bound(PB.abs_products(nvfp4.dequantize(qa, ca, G_x), nvfp4.dequantize(qw, cw, Gw)), K)
    PB.assert_within(y, ref, bound, "wide geometry", bf16=True)


FUSED_SHAPES = [(128, 512, 512), (300, 520, 1024), (1, 16, 64), (0, 32, 64)]


@pytest.mark.parametrize("M,N,K", FUSED_SHAPES)
def test_gemm_fused_act_quant(M, N, K):
    """X given instead of A (fused activation quantization with a static
    scale): the result equals quantize-then-GEMM bit for bit, and the oracle
    within tolerance; also with the NVFP4 epilogue."""
    say("fused", M, N, K)
    xb = synth.random_bf16(71, (M, K), outlier_frac=0.01, outlier_factor=20)
    calib = synth.random_bf16(1071, (max(M, 1), K), outlier_frac=0.01, outlier_factor=20)
    G_x = nvfp4.global_scale(nvfp4.amax(formats.f32_from_bf16_bits(calib)))
    w = synth.random_f32(72, (N, K), 0.02)
    W = dq.dq_pack_nvfp4(dev(w))
    Gd = dev(np.array([G_x], np.float32))
    y_f = host(dq.dq_prefill_gemm(W, X=bf16_dev(xb), G_x_static=Gd))
    A = dq.dq_quantize_act_nvfp4(bf16_dev(xb), G_static=Gd)
    y_u = host(dq.dq_prefill_gemm(W, A=A))
    assert np.array_equal(y_f, y_u)
    if M:
        qa, ca, _ = nvfp4.quantize_bf16_activations(xb, G_x)
        qw, cw, Gw = nvfp4.quantize_dynamic(w)
        ref = linalg.nvfp4_gemm(qa, ca, G_x, qw, cw, Gw)
        assert linalg.rel_fro(y_f, ref) <= TOL
        bound = PB.fp32_sum_bound(PB.abs_products(nvfp4.dequantize(qa, ca, G_x), nvfp4.dequantize(qw, cw, Gw)), K)
        PB.assert_within(y_f, ref, bound, "fused gemm")
    if N % 16 == 0:
        G_o = dev(np.array([0.01], np.float32))
        q_f = dq.dq_prefill_gemm(W, X=bf16_dev(xb), G_x_static=Gd, out_kind=dq.OUT_NVFP4, G_out_static=G_o)
        q_u = dq.dq_prefill_gemm(W, A=A, out_kind=dq.OUT_NVFP4, G_out_static=G_o)
        if M:   # (M = 0: the minimum allocations hold no data)
            assert torch.equal(q_f.codes, q_u.codes) and torch.equal(q_f.scales, q_u.scales)
        assert torch.equal(q_f.G, q_u.G)


def test_gemm_fused_down_27b_full_size_sampled():
    """The 27B-class down projection with fused activation quantization
    (M=8192, K=17408, N=5120) at full size; sampled rows and columns of the
    bf16 output against the oracle (weights quantized with the whole
    tensor's global scale)."""
    cfg = synth.DOWN_27B_M8192
    layer = cfg.layers[0]
    w = synth.layer_weight(cfg, layer)
    xb = synth.prefill_x(cfg, layer.k)
    calib = synth.prefill_x(cfg, layer.k, calib=True)
    G_x = nvfp4.global_scale(nvfp4.amax(formats.f32_from_bf16_bits(calib)))
    W = dq.dq_pack_nvfp4(dev(w))
    Y = dq.dq_prefill_gemm(W, X=bf16_dev(xb), G_x_static=dev(np.array([G_x], np.float32)), out_kind=dq.OUT_BF16)
    rng = np.random.default_rng(73)
    rows = np.sort(rng.choice(cfg.m, 16, replace=False))
    cols = np.sort(rng.choice(layer.n, 512, replace=False))
    qa, ca, _ = nvfp4.quantize_bf16_activations(xb[rows], G_x)
    Gw = nvfp4.global_scale(nvfp4.amax(w))
    qw, cw = nvfp4.quantize(w[cols], Gw)
    ref = linalg.nvfp4_gemm(qa, ca, G_x, qw, cw, Gw)
    y = host(Y[torch.from_numpy(rows).cuda()][:, torch.from_numpy(cols).cuda()].float()).astype(np.float64)
    err = linalg.rel_fro(y, formats.bf16_rne_from_f64(ref))
    say("  fused down sampled rel_fro", err)
    assert err <= TOL
    bound = PB.fp32_sum_bound(PB.abs_products(nvfp4.dequantize(qa, ca, G_x), nvfp4.dequantize(qw, cw, Gw)), layer.k)
    PB.assert_within(y, ref, bound, "fused down gemm", bf16=True)


def test_gemm_empty():
    W = dq.dq_pack_nvfp4(dev(synth.random_f32(1, (32, 64))))
    A = dq.dq_quantize_act_nvfp4(bf16_dev(np.zeros((0, 64), np.uint16)))
    y = dq.dq_prefill_gemm(W, A=A)
    assert y.shape == (0, 32)


# ---------------------------------------------------------------- a5 + a6: LUT pack and GEMV
def _lut_weight(N, K, seed):
    w = synth.random_f32(seed, (N, K), 0.02)
    return w * np.exp(0.3 * synth.random_f32(seed + 1, (N, 1))).astype(np.float32)


LUT_CASES = [(512, 512, 1, 3), (20, 96, 1, 3), (20, 96, 3, 2), (48, 4096, 4, 2), (12288, 4096, 1, 3),
             (12288, 4096, 4, 3), (12288, 4096, 1, 2), (12288, 4096, 4, 2), (64, 4096, 16, 3), (40, 17408, 16, 3),
             (5120, 17408, 1, 3), (33, 640, 1, 2), (33, 640, 2, 3),
             # K not a multiple of the 128-column chunk (a partial last chunk),
             # odd chunk counts, and batches on either side of the split plan's
             # task-count switch at 12
             (100, 4128, 1, 3), (100, 4128, 8, 2), (4112, 1056, 1, 3), (256, 4096, 12, 3), (96, 2080, 5, 3)]


@pytest.mark.parametrize("N,K,B,bits", LUT_CASES)
def test_lut_per_row_pack_and_gemv(N, K, B, bits):
    say("lut per_row", N, K, B, bits)
    w = _lut_weight(N, K, 20 + bits)
    codes_ref, lut_ref = lut.quantize_per_row(w, bits)
    Wq = dq.dq_pack_lut3(dev(w), bits=bits, mode=dq.LUT_PER_ROW)
    codes = L.lut_codes_unpack(host(Wq.codes), N, K, bits)
    table = host(Wq.lut).view(np.uint16)[: N * (1 << bits)].reshape(N, 1 << bits)
    assert np.array_equal(table, lut_ref.view(np.uint16)), "LUT entries differ"
    assert np.array_equal(codes, codes_ref), f"codes differ at {np.argwhere(codes != codes_ref)[:5]}"
    xb = synth.random_bf16(30 + B, (B, K), outlier_frac=0.005, outlier_factor=30)
    ref = linalg.lut_gemv_per_row(xb, codes_ref, lut_ref)
    y = host(dq.dq_decode_gemv(bf16_dev(xb), Wq, out_kind=dq.OUT_F32))
    err = linalg.rel_fro(y, ref)
    say("  gemv rel_fro", err)
    assert err <= TOL
    PB.assert_within(y, ref, PB.gemv_bound(formats.f64_from_bf16_bits(xb), lut.dequantize_per_row(codes_ref, lut_ref), K),
                     "lut per-row gemv")
    if K <= 4096:
        yb = host(dq.dq_decode_gemv(bf16_dev(xb), Wq, out_kind=dq.OUT_BF16).float()).astype(np.float64)
        assert linalg.rel_fro(yb, formats.bf16_rne_from_f64(ref)) <= TOL


@pytest.mark.parametrize("N,K,B,bits", [(512, 512, 1, 3), (20, 96, 2, 3), (37, 1024, 1, 2), (256, 4096, 4, 3)])
def test_lut_paper_grid_pack_and_gemv(N, K, B, bits):
    say("lut paper", N, K, B, bits)
    w = _lut_weight(N, K, 40 + bits)
    w[min(3, N - 1), :16] = 0.0                                   # a zero block
    grid = lut.default_grid(bits)
    codes_ref, sb_ref, G_ref = lut.quantize_paper_grid(w, grid)
    Wq = dq.dq_pack_lut3(dev(w), bits=bits, mode=dq.LUT_PAPER_GRID)
    codes = L.lut_codes_unpack(host(Wq.codes), N, K, bits)
    sb = L.lut_scales_unpack(host(Wq.scales), N, K)
    assert host(Wq.G)[0] == G_ref
    assert np.array_equal(host(Wq.lut).view(np.uint16)[: 1 << bits], grid.view(np.uint16))
    assert np.array_equal(sb, sb_ref), f"scales differ at {np.argwhere(sb != sb_ref)[:5]}"
    assert np.array_equal(codes, codes_ref), f"codes differ at {np.argwhere(codes != codes_ref)[:5]}"
    xb = synth.random_bf16(50 + B, (B, K), outlier_frac=0.005, outlier_factor=30)
    ref = linalg.lut_gemv_paper(xb, codes_ref, sb_ref, G_ref, grid)
    y = host(dq.dq_decode_gemv(bf16_dev(xb), Wq))
    err = linalg.rel_fro(y, ref)
    say("  gemv rel_fro", err)
    assert err <= TOL
    w_hat = lut.dequantize_paper_grid(codes_ref, sb_ref, G_ref, grid)
    PB.assert_within(y, ref, PB.gemv_bound(formats.f64_from_bf16_bits(xb), w_hat, K, 2.0 ** -11), "lut paper gemv")


def test_lut_paper_grid_custom_grid():
    grid = np.array([-3.0, -1.0, 0.0, 0.5, 1.0, 2.0, 4.0, 6.0], np.float16)
    w = _lut_weight(32, 256, 60)
    codes_ref, sb_ref, G_ref = lut.quantize_paper_grid(w, grid)
    Wq = dq.dq_pack_lut3(dev(w), bits=3, mode=dq.LUT_PAPER_GRID, grid=grid)
    assert np.array_equal(L.lut_codes_unpack(host(Wq.codes), 32, 256, 3), codes_ref)
    assert np.array_equal(L.lut_scales_unpack(host(Wq.scales), 32, 256), sb_ref)


def test_gemv_large_activations_rescaled():
    """Activations far outside fp16 range are rescaled per slice by a power of two."""
    N, K = 64, 1024
    w = _lut_weight(N, K, 70)
    codes_ref, lut_ref = lut.quantize_per_row(w, 3)
    x = synth.random_f32(71, (2, K))
    x[0] *= np.float32(1e6)
    x[1] *= np.float32(1e-6)
    xb = synth.bf16_bits_from_f32(x)
    ref = linalg.lut_gemv_per_row(xb, codes_ref, lut_ref)
    Wq = dq.dq_pack_lut3(dev(w), bits=3)
    y = host(dq.dq_decode_gemv(bf16_dev(xb), Wq))
    for b in range(2):
        assert linalg.rel_fro(y[b], ref[b]) <= TOL
    PB.assert_within(y, ref, PB.gemv_bound(formats.f64_from_bf16_bits(xb), lut.dequantize_per_row(codes_ref, lut_ref), K),
                     "rescaled activations gemv")


def test_gemv_workspace_and_pool_paths_agree():
    """B >= 2 with split-K partials: a caller workspace and the library's own
    pool (NULL workspace) run the same kernels and give identical outputs."""
    N, K, B = 7168, 5120, 8
    say("gemv workspace vs pool", N, K, B)
    w = _lut_weight(N, K, 80)
    Wq = dq.dq_pack_lut3(dev(w), bits=3)
    xb = synth.random_bf16(81, (B, K), outlier_frac=0.005, outlier_factor=30)
    x = bf16_dev(xb)
    n = dq.dq_decode_gemv_workspace_size(B, Wq)
    assert n > 0
    ws = torch.full((n + 64,), 0xFF, dtype=torch.uint8, device="cuda")   # stale contents must not matter
    y_ws = dq.dq_decode_gemv(x, Wq, workspace=ws)
    y_ws2 = dq.dq_decode_gemv(x, Wq, workspace=ws)
    y_pool = torch.empty_like(y_ws)
    lib = dq.lib()
    d = Wq.desc()
    assert lib.dq_decode_gemv(x.data_ptr(), B, ctypes.byref(d), dq.OUT_F32, y_pool.data_ptr(), None, 0,
                              torch.cuda.current_stream().cuda_stream) == dq.DQ_OK
    assert torch.equal(y_ws, y_pool) and torch.equal(y_ws, y_ws2)
    codes_ref, lut_ref = lut.quantize_per_row(w, 3)
    ref = linalg.lut_gemv_per_row(xb, codes_ref, lut_ref)
    assert linalg.rel_fro(host(y_ws), ref) <= TOL
    PB.assert_within(host(y_ws), ref, PB.gemv_bound(formats.f64_from_bf16_bits(xb),
                                                    lut.dequantize_per_row(codes_ref, lut_ref), K), "workspace gemv")


# ---------------------------------------------------------------- NVFP4A16 decode GEMV
# one-launch kernel (four wavefronts per row tile up to 64 K steps, else
# eight): batch <= 8 with the activation slices in LDS and at most one
# resident round of row tiles; the K-group kernel otherwise ((5120, 5120, 16),
# (64, 4096, 8), (34816, 2048, 1))
NV_GEMV_CASES = [(512, 512, 1), (100, 96, 3), (33, 1040, 2), (7168, 5120, 1), (5120, 17408, 1), (5120, 5120, 16),
                 (12288, 4096, 4), (64, 4096, 8), (17408, 2048, 1), (34816, 2048, 1), (16384, 208, 8), (40, 16, 1)]


@pytest.mark.parametrize("N,K,B", NV_GEMV_CASES)
def test_nvfp4a16_gemv(N, K, B):
    """Weight-only NVFP4 decode: the GPU's own NVFP4 weight packing, bf16 x,
    against the oracle's fp64 GEMV over the oracle-dequantized weights."""
    say("nvfp4a16 gemv", N, K, B)
    w = _lut_weight(N, K, 90)
    qw, cw, Gw = nvfp4.quantize_dynamic(w)
    Wq = dq.dq_pack_nvfp4(dev(w))
    q_g, c_g, _, _ = L.nvfp4_unpack(host(Wq.codes), host(Wq.scales), N, K)
    assert np.array_equal(q_g, qw) and np.array_equal(c_g, cw) and host(Wq.G)[0] == Gw
    xb = synth.random_bf16(91 + B, (B, K), outlier_frac=0.005, outlier_factor=30)
    ref = linalg.nvfp4a16_gemv(xb, qw, cw, Gw)
    y = host(dq.dq_decode_gemv_nvfp4(bf16_dev(xb), Wq, out_kind=dq.OUT_F32))
    err = linalg.rel_fro(y, ref)
    say("  rel_fro", err)
    assert err <= TOL
    PB.assert_within(y, ref, PB.gemv_bound(formats.f64_from_bf16_bits(xb), nvfp4.dequantize(qw, cw, Gw), K),
                     "nvfp4a16 gemv")
    if K <= 5120:
        yb = host(dq.dq_decode_gemv_nvfp4(bf16_dev(xb), Wq, out_kind=dq.OUT_BF16).float()).astype(np.float64)
        assert linalg.rel_fro(yb, formats.bf16_rne_from_f64(ref)) <= TOL


def test_nvfp4a16_gemv_empty_and_pool():
    """K = 0 gives zeros; a small batch runs in one launch without a
    workspace; with K split over workgroups (batch 12) a NULL workspace
    (library pool) gives the same result as a caller workspace."""
    W0 = dq.NvFp4Tensor.empty(40, 0)
    y0 = dq.dq_decode_gemv_nvfp4(torch.zeros((2, 0), dtype=torch.int16, device="cuda"), W0)
    assert tuple(y0.shape) == (2, 40) and not host(y0).any()
    assert dq.dq_decode_gemv_nvfp4_workspace_size(2, dq.NvFp4Tensor.empty(5120, 5120)) == 0
    N, K, B = 5120, 5120, 12
    w = _lut_weight(N, K, 92)
    Wq = dq.dq_pack_nvfp4(dev(w))
    xb = synth.random_bf16(93, (B, K), outlier_frac=0.005, outlier_factor=30)
    x = bf16_dev(xb)
    assert dq.dq_decode_gemv_nvfp4_workspace_size(B, Wq) > 0
    y_ws = dq.dq_decode_gemv_nvfp4(x, Wq)
    y_pool = torch.empty_like(y_ws)
    d = Wq.desc()
    assert dq.lib().dq_decode_gemv_nvfp4(x.data_ptr(), B, ctypes.byref(d), dq.OUT_F32, y_pool.data_ptr(), None, 0,
                                         torch.cuda.current_stream().cuda_stream) == dq.DQ_OK
    assert torch.equal(y_ws, y_pool)


# ---------------------------------------------------------------- LUT -> NVFP4 autocast
@pytest.mark.parametrize("N,K,bits,mode", [(512, 512, 3, 0), (20, 96, 3, 0), (300, 1024, 2, 0), (12288, 4096, 3, 0),
                                           (37, 1024, 3, 1), (64, 4096, 2, 1)])
def test_lut_autocast_to_nvfp4(N, K, bits, mode):
    """The GPU's own LUT packing, re-quantized to NVFP4 on the GPU, against
    the oracle's autocast of the oracle's LUT weight: codes, scales and G
    bit-exact; then the prefill GEMM on the autocast weights."""
    say("autocast", N, K, bits, mode)
    w = _lut_weight(N, K, 100 + bits)
    if mode == dq.LUT_PER_ROW:
        codes_ref, table = lut.quantize_per_row(w, bits)
        w_hat = lut.dequantize_per_row(codes_ref, table)
    else:
        grid = lut.default_grid(bits)
        codes_ref, sb, G_l = lut.quantize_paper_grid(w, grid)
        w_hat = lut.dequantize_paper_grid(codes_ref, sb, G_l, grid)
    q_ref, c_ref, G_ref = lut.autocast_to_nvfp4(w_hat)
    Wl = dq.dq_pack_lut3(dev(w), bits=bits, mode=mode)
    Wn = dq.dq_autocast_lut_to_nvfp4(Wl)
    q, c, qfull, cfull = L.nvfp4_unpack(host(Wn.codes), host(Wn.scales), N, K)
    assert host(Wn.G)[0] == G_ref
    assert np.array_equal(c, c_ref), f"scales differ at {np.argwhere(c != c_ref)[:5]}"
    assert np.array_equal(q, q_ref), f"codes differ at {np.argwhere(q != q_ref)[:5]}"
    assert not qfull[N:].any() and not cfull[N:].any()
    if N * K <= 1 << 22:
        xb = synth.random_bf16(110, (64, K), outlier_frac=0.01, outlier_factor=20)
        qa, ca, Ga = nvfp4.quantize_bf16_activations(xb)
        A = _upload_nvfp4(qa, ca, Ga)
        y = host(dq.dq_prefill_gemm(Wn, A=A, out_kind=dq.OUT_F32))
        ref = linalg.nvfp4_gemm(qa, ca, Ga, q_ref, c_ref, G_ref)
        assert linalg.rel_fro(y, ref) <= TOL
        bound = PB.fp32_sum_bound(PB.abs_products(nvfp4.dequantize(qa, ca, Ga), nvfp4.dequantize(q_ref, c_ref, G_ref)), K)
        PB.assert_within(y, ref, bound, "autocast gemm")


def test_lut_autocast_static_scale():
    w = _lut_weight(48, 256, 111)
    Wl = dq.dq_pack_lut3(dev(w), bits=3)
    G = np.float32(3.0e-4)
    Wn = dq.dq_autocast_lut_to_nvfp4(Wl, G_override=dev(np.array([G], np.float32)))
    codes_ref, table = lut.quantize_per_row(w, 3)
    q_ref, c_ref, _ = lut.autocast_to_nvfp4(lut.dequantize_per_row(codes_ref, table), G=G)
    q, c, _, _ = L.nvfp4_unpack(host(Wn.codes), host(Wn.scales), 48, 256)
    assert host(Wn.G)[0] == G and np.array_equal(q, q_ref) and np.array_equal(c, c_ref)


# ---------------------------------------------------------------- RMSNorm + NVFP4 activation quantization
from oracle import norm  # noqa: E402

NORM_SHAPES = [(128, 512, 0), (33, 1040, 1), (1, 16, 2), (2048, 4096, 3), (300, 5120, 4), (40, 8192, 5),
               (40, 8256, 6)]


def _norm_case(M, K, seed):
    xb = synth.random_bf16(120 + seed, (M, K), outlier_frac=0.005, outlier_factor=30)
    gb = synth.bf16_bits_from_f32((1.0 + 0.2 * synth.random_f32(121 + seed, (1, K))).astype(np.float32))[0]
    return xb, gb


@pytest.mark.parametrize("M,K,seed", NORM_SHAPES)
@pytest.mark.parametrize("static", [False, True])
def test_rmsnorm_quantize_act(M, K, seed, static):
    """Fused RMSNorm + NVFP4 activation quantization against the oracle's
    fp32 RMSNorm and a1 quantizer (static scale with K <= 8192: the one-pass
    kernel; K = 8256 or a dynamic scale: statistics pass, then the tile
    quantizer).  Both follow the same fp32 operation
    order; only the fp64 sum of squares may round differently (tree vs
    exactly rounded), so a differing code or scale is accepted only at a
    rounding boundary of the oracle's normalized values, and at most one in
    10^4."""
    from test_gpu_epilogue import tolerant_match
    say("rmsnorm quant", M, K, static)
    xb, gb = _norm_case(M, K, seed)
    eps = 1e-5
    G_s = np.float32(0.0125) if static else None
    q_ref, c_ref, G_ref, y = norm.quantize_rmsnorm_bf16(xb, gb, eps, G_s)
    t = dq.dq_rmsnorm_quantize_act_nvfp4(bf16_dev(xb), bf16_dev(gb), eps,
                                         G_static=dev(np.array([G_s], np.float32)) if static else None)
    q, c, qfull, cfull = L.nvfp4_unpack(host(t.codes), host(t.scales), M, K)
    G = host(t.G)[0]
    assert G == G_ref
    n_s, n_q = tolerant_match(q, c, y.astype(np.float64), G)
    say("  differing scales / codes", n_s, n_q)
    assert n_s + n_q <= max(1, M * K // 10000)
    assert not qfull[M:].any() and not cfull[M:].any()


def test_rmsnorm_quantize_act_empty():
    t = dq.dq_rmsnorm_quantize_act_nvfp4(torch.empty((0, 64), dtype=torch.int16, device="cuda"),
                                         torch.ones(64, dtype=torch.bfloat16, device="cuda"))
    assert t.rows == 0 and host(t.G)[0] == 1.0
