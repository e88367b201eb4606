"""C-ABI contract checks that need no GPU: the library loads, exports every
function include/dq.h declares, and rejects invalid arguments on the host
before any HIP call (DQ_ERR_INVALID_ARG / DQ_ERR_UNSUPPORTED)."""
import ctypes
import os
import re

import pytest

import paper_2609_26333_amd as dq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "dq.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dq_[a-z0-9_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = _declared()
    assert len(names) >= 10
    lib = ctypes.CDLL(dq.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(dq.EXPORTED)


def test_version_and_status_strings():
    assert dq.abi_version() == 3
    lib = dq.lib()
    assert lib.dq_status_string(0) == b"DQ_OK"
    assert lib.dq_status_string(-1) == b"DQ_ERR_INVALID_ARG"
    assert lib.dq_status_string(-2) == b"DQ_ERR_UNSUPPORTED"
    assert lib.dq_status_string(-3) == b"DQ_ERR_HIP"


def test_size_queries():
    assert dq.nvfp4_sizes(100, 48) == (128 * 64 // 2, 128 * 64 // 16)
    assert dq.nvfp4_sizes(0, 0) == (0, 0)
    assert dq.lut_sizes(3, dq.LUT_PER_ROW, 20, 96) == (2 * 1 * 64 * 12, 32 * 8 * 2, 0)
    assert dq.lut_sizes(2, dq.LUT_PAPER_GRID, 16, 256) == (1 * 2 * 64 * 8, 8, 2 * 128)
    with pytest.raises(dq.DQError) as e:
        dq.nvfp4_sizes(4, 24)
    assert e.value.status == dq.DQ_ERR_INVALID_ARG
    with pytest.raises(dq.DQError):
        dq.lut_sizes(4, 0, 16, 32)
    with pytest.raises(dq.DQError):
        dq.lut_sizes(3, 0, 16, 48)
    assert dq.mxfp4_sizes(100, 96) == (128 * 128 // 2, 128 * 128 // 32)
    assert dq.mxfp4_sizes(130, 64) == (160 * 64 // 2, 256 * 64 // 32)
    assert dq.mxfp4_sizes(0, 0) == (0, 0)
    # fused prefill staging: the NVFP4 copy of X (tile-rounded) plus its global scale
    assert dq.dq_prefill_gemm_workspace_size(100, 48) == 128 * 64 // 2 + 128 * 64 // 16 + 16
    assert dq.dq_prefill_gemm_workspace_size(0, 64) == 16
    with pytest.raises(dq.DQError):
        dq.dq_prefill_gemm_workspace_size(4, 24)
    with pytest.raises(dq.DQError):
        dq.mxfp4_sizes(4, 48)


def test_mxfp4_arguments_rejected_on_host():
    lib = dq.lib()
    fake = 1 << 20
    mx = lambda r, c, codes=fake, scales=fake: dq._MxFp4(codes, scales, r, c)   # noqa: E731
    P = ctypes.byref
    # K % 32, descriptor shape, NULL / misaligned buffers
    assert lib.dq_pack_mxfp4(fake, 4, 48, P(mx(4, 48)), None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_pack_mxfp4(fake, 4, 64, P(mx(4, 32)), None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_pack_mxfp4(fake, 4, 64, P(mx(4, 64, codes=None)), None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_pack_mxfp4(fake + 4, 4, 64, P(mx(4, 64)), None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_quantize_act_mxfp4(fake, 4, 64, P(mx(4, 64, scales=fake + 8)), None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_quantize_act_mxfp4(None, 4, 64, P(mx(4, 64)), None) == dq.DQ_ERR_INVALID_ARG
    # GEMM: K mismatch, bad out_kind, NULL Y
    assert lib.dq_prefill_gemm_mxfp4(P(mx(4, 64)), P(mx(8, 128)), 0, fake, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_prefill_gemm_mxfp4(P(mx(4, 64)), P(mx(8, 64)), dq.OUT_NVFP4, fake, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_prefill_gemm_mxfp4(P(mx(4, 64)), P(mx(8, 64)), 0, None, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_prefill_gemm_mxfp4(None, P(mx(8, 64)), 0, fake, None) == dq.DQ_ERR_INVALID_ARG
    # GEMM: K of 2^23 and beyond is not implemented (32-bit row-panel offsets)
    big = 1 << 23
    assert lib.dq_prefill_gemm_mxfp4(P(mx(4, big)), P(mx(8, big)), 0, fake, None) == dq.DQ_ERR_UNSUPPORTED


def _nv(rows, cols, codes=16, scales=16, G=16):
    return dq._NvFp4(codes, scales, G, rows, cols)


def test_invalid_arguments_rejected_on_host():
    lib = dq.lib()
    fake = 1 << 20                       # never dereferenced: validation fails first
    d = _nv(4, 24, fake, fake, fake)
    # K % 16 != 0
    assert lib.dq_quantize_act_nvfp4(fake, 4, 24, None, ctypes.byref(d), None) == dq.DQ_ERR_INVALID_ARG
    assert b"16" in lib.dq_last_error()
    # misaligned input
    d = _nv(4, 32, fake, fake, fake)
    assert lib.dq_quantize_act_nvfp4(fake + 2, 4, 32, None, ctypes.byref(d), None) == dq.DQ_ERR_INVALID_ARG
    # descriptor shape mismatch
    d = _nv(5, 32, fake, fake, fake)
    assert lib.dq_pack_nvfp4(fake, 4, 32, None, ctypes.byref(d), None) == dq.DQ_ERR_INVALID_ARG
    # NULL descriptor buffer
    d = _nv(4, 32, fake, 0, fake)
    assert lib.dq_pack_nvfp4(fake, 4, 32, None, ctypes.byref(d), None) == dq.DQ_ERR_INVALID_ARG
    # GEMM: both A and X / neither
    a = _nv(4, 32, fake, fake, fake)
    w = _nv(8, 32, fake, fake, fake)
    assert lib.dq_prefill_gemm(ctypes.byref(a), fake, fake, ctypes.byref(w), 4, 0, fake, None, None, 0,
                               None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_prefill_gemm(None, None, None, ctypes.byref(w), 4, 0, fake, None, None, 0,
                               None, 0, None) == dq.DQ_ERR_INVALID_ARG
    # GEMM: fused path with a workspace that is too small or misaligned
    need = dq.dq_prefill_gemm_workspace_size(4, 32)
    assert lib.dq_prefill_gemm(None, fake, fake, ctypes.byref(w), 4, 0, fake, None, None, 0, fake, need - 1,
                               None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_prefill_gemm(None, fake, fake, ctypes.byref(w), 4, 0, fake, None, None, 0, fake + 8, need,
                               None) == dq.DQ_ERR_INVALID_ARG
    # GEMM: K of 2^23 and beyond is not implemented (32-bit row-panel offsets)
    big = 1 << 23
    a3, w3 = _nv(4, big, fake, fake, fake), _nv(8, big, fake, fake, fake)
    assert lib.dq_prefill_gemm(ctypes.byref(a3), None, None, ctypes.byref(w3), 4, 0, fake, None, None, 0,
                               None, 0, None) == dq.DQ_ERR_UNSUPPORTED
    # GEMM: K mismatch between A and W
    a2 = _nv(4, 48, fake, fake, fake)
    assert lib.dq_prefill_gemm(ctypes.byref(a2), None, None, ctypes.byref(w), 4, 0, fake, None, None, 0,
                               None, 0, None) == dq.DQ_ERR_INVALID_ARG
    # GEMM: bad out kind, bad flag
    assert lib.dq_prefill_gemm(ctypes.byref(a), None, None, ctypes.byref(w), 4, 7, fake, None, None, 0,
                               None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_prefill_gemm(ctypes.byref(a), None, None, ctypes.byref(w), 4, 0, fake, None, None, 4,
                               None, 0, None) == dq.DQ_ERR_INVALID_ARG
    # SwiGLU needs gate/up groups of 16 rows (W rows % 32 == 0)
    w48 = _nv(48, 32, fake, fake, fake)
    assert lib.dq_prefill_gemm(ctypes.byref(a), None, None, ctypes.byref(w48), 4, 0, fake, None, None,
                               dq.EPI_SWIGLU, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    # NVFP4 output: Y must be NULL, Yq and G_out given, Yq shaped [M, N] ([M, N/2] with SwiGLU)
    w64 = _nv(64, 32, fake, fake, fake)
    yq = _nv(4, 64, fake, fake, fake)
    yq_sw = _nv(4, 32, fake, fake, fake)
    assert lib.dq_prefill_gemm(ctypes.byref(a), None, None, ctypes.byref(w64), 4, dq.OUT_NVFP4, fake, fake,
                               ctypes.byref(yq), 0, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_prefill_gemm(ctypes.byref(a), None, None, ctypes.byref(w64), 4, dq.OUT_NVFP4, None, None,
                               ctypes.byref(yq), 0, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_prefill_gemm(ctypes.byref(a), None, None, ctypes.byref(w64), 4, dq.OUT_NVFP4, None, fake,
                               None, 0, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_prefill_gemm(ctypes.byref(a), None, None, ctypes.byref(w64), 4, dq.OUT_NVFP4, None, fake,
                               ctypes.byref(yq_sw), 0, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_prefill_gemm(ctypes.byref(a), None, None, ctypes.byref(w64), 4, dq.OUT_NVFP4, None, fake,
                               ctypes.byref(yq), dq.EPI_SWIGLU, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    # Yq with a plain output
    assert lib.dq_prefill_gemm(ctypes.byref(a), None, None, ctypes.byref(w64), 4, 0, fake, None,
                               ctypes.byref(yq), 0, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    # NVFP4 output columns must be a multiple of 16 (here 40 / 2 = 20 after SwiGLU is refused first;
    # 24 rows without SwiGLU)
    w24 = _nv(24, 32, fake, fake, fake)
    yq24 = _nv(4, 24, fake, fake, fake)
    assert lib.dq_prefill_gemm(ctypes.byref(a), None, None, ctypes.byref(w24), 4, dq.OUT_NVFP4, None, fake,
                               ctypes.byref(yq24), 0, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    # GEMV: batch out of range, bad bits
    lw = dq._Lut(fake, fake, None, None, 16, 128, 3, 0)
    assert lib.dq_decode_gemv(fake, 0, ctypes.byref(lw), 0, fake, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_decode_gemv(fake, 17, ctypes.byref(lw), 0, fake, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    lw_bad = dq._Lut(fake, fake, None, None, 16, 128, 4, 0)
    assert lib.dq_decode_gemv(fake, 1, ctypes.byref(lw_bad), 0, fake, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    # workspace: none at B = 1, split-K partials at B >= 2; a short one is refused
    ws = ctypes.c_size_t(123)
    big = dq._Lut(fake, fake, None, None, 7168, 5120, 3, 0)
    assert lib.dq_decode_gemv_workspace_size(1, ctypes.byref(big), ctypes.byref(ws)) == dq.DQ_OK and ws.value == 0
    assert lib.dq_decode_gemv_workspace_size(16, ctypes.byref(big), ctypes.byref(ws)) == dq.DQ_OK and ws.value > 0
    assert lib.dq_decode_gemv_workspace_size(17, ctypes.byref(big), ctypes.byref(ws)) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_decode_gemv(fake, 16, ctypes.byref(big), 0, fake, fake, ws.value - 16, None) == dq.DQ_ERR_INVALID_ARG
    # the no-allocation GEMV: same argument checks; partial sums beyond its static scratch are refused
    assert lib.dq_decode_gemv_noalloc(fake, 17, ctypes.byref(big), 0, fake, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_decode_gemv_noalloc(fake, 1, ctypes.byref(lw_bad), 0, fake, None) == dq.DQ_ERR_INVALID_ARG
    huge = dq._Lut(fake, fake, None, None, 131072, 5120, 3, 0)
    assert lib.dq_decode_gemv_workspace_size(16, ctypes.byref(huge), ctypes.byref(ws)) == dq.DQ_OK
    assert ws.value > dq.NOALLOC_SCRATCH_BYTES
    assert lib.dq_decode_gemv_noalloc(fake, 16, ctypes.byref(huge), 0, fake, None) == dq.DQ_ERR_UNSUPPORTED
    assert b"scratch" in lib.dq_last_error()
    # NVFP4A16 GEMV: batch range, K % 16, short workspace
    wn = _nv(7168, 5120, fake, fake, fake)
    assert lib.dq_decode_gemv_nvfp4(fake, 0, ctypes.byref(wn), 0, fake, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_decode_gemv_nvfp4(fake, 17, ctypes.byref(wn), 0, fake, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_decode_gemv_nvfp4(fake, 1, ctypes.byref(_nv(16, 24, fake, fake, fake)), 0, fake, None, 0,
                                    None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_decode_gemv_nvfp4(fake, 1, None, 0, fake, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    # batch 1 runs in one launch without a workspace; batch 16 splits K
    assert lib.dq_decode_gemv_nvfp4_workspace_size(1, ctypes.byref(wn), ctypes.byref(ws)) == dq.DQ_OK and ws.value == 0
    assert lib.dq_decode_gemv_nvfp4_workspace_size(16, ctypes.byref(wn), ctypes.byref(ws)) == dq.DQ_OK and ws.value > 0
    assert lib.dq_decode_gemv_nvfp4(fake, 16, ctypes.byref(wn), 0, fake, fake, ws.value - 16,
                                    None) == dq.DQ_ERR_INVALID_ARG
    # fused RMSNorm quantizer: K % 16, negative / non-finite eps, NULL gamma
    dn = _nv(4, 64, fake, fake, fake)
    assert lib.dq_rmsnorm_quantize_act_nvfp4(fake, fake, 1e-6, 4, 24, None, ctypes.byref(_nv(4, 24, fake, fake, fake)),
                                             None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_rmsnorm_quantize_act_nvfp4(fake, fake, -1.0, 4, 64, None, ctypes.byref(dn), None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_rmsnorm_quantize_act_nvfp4(fake, fake, float("nan"), 4, 64, None, ctypes.byref(dn),
                                             None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_rmsnorm_quantize_act_nvfp4(fake, None, 1e-6, 4, 64, None, ctypes.byref(dn), None, 0, None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_rmsnorm_quantize_act_nvfp4(fake, fake, 1e-6, 4, 64, None, ctypes.byref(dn), fake, 8,
                                             None) == dq.DQ_ERR_INVALID_ARG
    # autocast: output shape must match W
    assert lib.dq_autocast_lut_to_nvfp4(ctypes.byref(lw), None, ctypes.byref(_nv(16, 64, fake, fake, fake)),
                                        None) == dq.DQ_ERR_INVALID_ARG
    assert lib.dq_autocast_lut_to_nvfp4(None, None, ctypes.byref(_nv(16, 128, fake, fake, fake)),
                                        None) == dq.DQ_ERR_INVALID_ARG
    # PAPER_GRID without scales / G
    lw_p = dq._Lut(fake, fake, None, None, 16, 128, 3, 1)
    assert lib.dq_decode_gemv(fake, 1, ctypes.byref(lw_p), 0, fake, None, 0, None) == dq.DQ_ERR_INVALID_ARG
    # LUT pack: K % 32, PER_ROW K limit, bad grid
    lo = dq._Lut(fake, fake, None, None, 16, 48, 3, 0)
    assert lib.dq_pack_lut3(fake, 16, 48, 3, 0, None, ctypes.byref(lo), None) == dq.DQ_ERR_INVALID_ARG
    lo = dq._Lut(fake, fake, None, None, 16, 65536, 3, 0)
    assert lib.dq_pack_lut3(fake, 16, 65536, 3, 0, None, ctypes.byref(lo), None) == dq.DQ_ERR_UNSUPPORTED
    lp = dq._Lut(fake, fake, fake, fake, 16, 128, 2, 1)
    bad_grid = (ctypes.c_uint16 * 4)(0x4000, 0x3C00, 0x0000, 0x4600)      # not ascending
    assert lib.dq_pack_lut3(fake, 16, 128, 2, 1, bad_grid, ctypes.byref(lp), None) == dq.DQ_ERR_INVALID_ARG
    no_zero = (ctypes.c_uint16 * 4)(0xC000, 0x3C00, 0x4000, 0x4600)
    assert lib.dq_pack_lut3(fake, 16, 128, 2, 1, no_zero, ctypes.byref(lp), None) == dq.DQ_ERR_INVALID_ARG


def test_oracle_is_not_imported_by_the_product():
    """The binding and the C sources never reach into oracle/."""
    pkg = os.path.join(ROOT, "paper_2609_26333_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".hpp", ".h")):
                txt = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in txt and "from oracle" not in txt, f
