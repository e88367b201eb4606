"""The no-allocation decode GEMV (dq_decode_gemv_noalloc), through the C ABI:
its split-K partial sums live in the library's static per-GPU scratch, and
its output must equal dq_decode_gemv's (same kernels, a caller workspace)
bit for bit, on two calls in a row, the second with a smaller input, and on
a batch-1 call (no partial sums).  The oracle confirms the first call."""
import ctypes
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import parity_bounds as PB  # noqa: E402

import synth  # noqa: E402
from oracle import formats, linalg, lut  # noqa: E402

pytestmark = pytest.mark.gpu

try:
    import paper_2609_26333_amd as dq
except ImportError:  # pragma: no cover
    dq = None


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if dq is None or not torch.cuda.is_available():
        pytest.skip("needs the built HIP library and a GPU")


def _case(N, K, B, seed):
    w = synth.random_f32(seed, (N, K), 0.02)
    Wq = dq.dq_pack_lut3(torch.from_numpy(w).cuda(), bits=3)
    xb = synth.random_bf16(seed + 1, (B, K), outlier_frac=0.005, outlier_factor=30)
    return w, Wq, torch.from_numpy(xb.view(np.int16)).cuda(), xb


def _both(Wq, x, B, out_kind):
    lib = dq.lib()
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    dt = torch.float32 if out_kind == dq.OUT_F32 else torch.bfloat16
    y_ref = torch.full((B, Wq.rows), 7.0, dtype=dt, device="cuda")
    y_na = torch.full((B, Wq.rows), -3.0, dtype=dt, device="cuda")
    n = dq.dq_decode_gemv_workspace_size(B, Wq)
    ws = torch.empty(max(n, 16), dtype=torch.uint8, device="cuda")
    d = Wq.desc()
    assert lib.dq_decode_gemv(x.data_ptr(), B, ctypes.byref(d), out_kind, y_ref.data_ptr(), ws.data_ptr(), n,
                              s) == dq.DQ_OK
    assert lib.dq_decode_gemv_noalloc(x.data_ptr(), B, ctypes.byref(d), out_kind, y_na.data_ptr(), s) == dq.DQ_OK
    torch.cuda.synchronize()
    return n, y_ref, y_na


def test_noalloc_gemv_matches_workspace_gemv_twice_then_batch1():
    # first call: batch 16 on the 27B q/k/v shape (K split over workgroups: partial sums in the scratch)
    w, Wq, x, xb = _case(7168, 5120, 16, 401)
    n1, y_ref, y_na = _both(Wq, x, 16, dq.OUT_F32)
    assert 0 < n1 <= dq.NOALLOC_SCRATCH_BYTES
    assert torch.equal(y_ref, y_na)
    codes, table = lut.quantize_per_row(w, 3)
    ref = linalg.lut_gemv_per_row(xb, codes, table)
    assert linalg.rel_fro(y_na.cpu().numpy(), ref) <= 1e-3
    PB.assert_within(y_na.cpu().numpy(), ref,
                     PB.gemv_bound(formats.f64_from_bf16_bits(xb), lut.dequantize_per_row(codes, table), 5120),
                     "noalloc gemv")
    # second call, smaller: batch 4 on a 1040 x 4096 weight, bf16 output; the scratch still
    # holds the first call's partial sums, which must not leak into this result
    _, Wq2, x2, _ = _case(1040, 4096, 4, 402)
    n2, y_ref2, y_na2 = _both(Wq2, x2, 4, dq.OUT_BF16)
    assert 0 < n2 < n1
    assert torch.equal(y_ref2, y_na2)
    # batch 1: one launch, no partial sums
    _, Wq3, x3, _ = _case(512, 512, 1, 403)
    n3, y_ref3, y_na3 = _both(Wq3, x3, 1, dq.OUT_F32)
    assert n3 == 0 and torch.equal(y_ref3, y_na3)
