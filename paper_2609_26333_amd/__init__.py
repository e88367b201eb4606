"""Python binding of libdq: the MI355X hot path of disaggregated quantization.

Thin argument marshalling over the C ABI in ``include/dq.h`` (same call names).
Every step of the path runs in the gfx950 kernels of ``libdq.so``; there is no
CPU fallback: importing this package fails if the library is not built
(``python paper_2609_26333_amd/build.py``).

PyTorch supplies device memory and the current HIP stream only.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdq.so")

DQ_OK = 0
DQ_ERR_INVALID_ARG = -1
DQ_ERR_UNSUPPORTED = -2
DQ_ERR_HIP = -3
OUT_F32, OUT_BF16, OUT_NVFP4 = 0, 1, 2
LUT_PER_ROW, LUT_PAPER_GRID = 0, 1
EPI_SWIGLU = 1


class DQError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


class _NvFp4(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p), ("G", ctypes.c_void_p),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64)]


class _MxFp4(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p), ("rows", ctypes.c_int64),
                ("cols", ctypes.c_int64)]


class _Lut(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_void_p), ("lut", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("G", ctypes.c_void_p), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("bits", ctypes.c_int32), ("mode", ctypes.c_int32)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2609_26333_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I32, S = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int32
    SZ = ctypes.POINTER(ctypes.c_size_t)
    sig = {
        "dq_abi_version": (I32, []),
        "dq_status_string": (ctypes.c_char_p, [S]),
        "dq_last_error": (ctypes.c_char_p, []),
        "dq_nvfp4_sizes": (S, [I64, I64, SZ, SZ]),
        "dq_lut_sizes": (S, [I32, I32, I64, I64, SZ, SZ, SZ]),
        "dq_pack_nvfp4": (S, [P, I64, I64, P, ctypes.POINTER(_NvFp4), P]),
        "dq_pack_lut3": (S, [P, I64, I64, I32, I32, P, ctypes.POINTER(_Lut), P]),
        "dq_quantize_act_nvfp4": (S, [P, I64, I64, P, ctypes.POINTER(_NvFp4), P]),
        "dq_prefill_gemm_workspace_size": (S, [I64, I64, SZ]),
        "dq_prefill_gemm": (S, [ctypes.POINTER(_NvFp4), P, P, ctypes.POINTER(_NvFp4), I64, I32, P, P,
                                ctypes.POINTER(_NvFp4), I32, P, ctypes.c_size_t, P]),
        "dq_autocast_lut_to_nvfp4": (S, [ctypes.POINTER(_Lut), P, ctypes.POINTER(_NvFp4), P]),
        "dq_rmsnorm_quantize_act_nvfp4": (S, [P, P, ctypes.c_float, I64, I64, P, ctypes.POINTER(_NvFp4), P,
                                              ctypes.c_size_t, P]),
        "dq_decode_gemv_nvfp4_workspace_size": (S, [I64, ctypes.POINTER(_NvFp4), SZ]),
        "dq_decode_gemv_nvfp4": (S, [P, I64, ctypes.POINTER(_NvFp4), I32, P, P, ctypes.c_size_t, P]),
        "dq_mxfp4_sizes": (S, [I64, I64, SZ, SZ]),
        "dq_pack_mxfp4": (S, [P, I64, I64, ctypes.POINTER(_MxFp4), P]),
        "dq_quantize_act_mxfp4": (S, [P, I64, I64, ctypes.POINTER(_MxFp4), P]),
        "dq_prefill_gemm_mxfp4": (S, [ctypes.POINTER(_MxFp4), ctypes.POINTER(_MxFp4), I32, P, P]),
        "dq_decode_gemv_workspace_size": (S, [I64, ctypes.POINTER(_Lut), SZ]),
        "dq_decode_gemv": (S, [P, I64, ctypes.POINTER(_Lut), I32, P, P, ctypes.c_size_t, P]),
        "dq_decode_gemv_noalloc": (S, [P, I64, ctypes.POINTER(_Lut), I32, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()
EXPORTED = ("dq_abi_version", "dq_status_string", "dq_last_error", "dq_nvfp4_sizes", "dq_lut_sizes",
            "dq_pack_nvfp4", "dq_pack_lut3", "dq_quantize_act_nvfp4", "dq_prefill_gemm",
            "dq_prefill_gemm_workspace_size",
            "dq_decode_gemv_workspace_size", "dq_decode_gemv", "dq_mxfp4_sizes", "dq_pack_mxfp4",
            "dq_quantize_act_mxfp4", "dq_prefill_gemm_mxfp4", "dq_decode_gemv_nvfp4_workspace_size",
            "dq_decode_gemv_nvfp4", "dq_autocast_lut_to_nvfp4", "dq_rmsnorm_quantize_act_nvfp4",
            "dq_decode_gemv_noalloc")


def lib() -> ctypes.CDLL:
    return _lib


def _check(status: int, call: str) -> None:
    if status != DQ_OK:
        raise DQError(status, f"{call}: {_lib.dq_status_string(status).decode()}: {_lib.dq_last_error().decode()}")


def abi_version() -> int:
    return _lib.dq_abi_version()


def _stream(stream=None) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


# ---------------------------------------------------------------- sizes
def nvfp4_sizes(rows: int, cols: int):
    c, s = ctypes.c_size_t(), ctypes.c_size_t()
    _check(_lib.dq_nvfp4_sizes(rows, cols, ctypes.byref(c), ctypes.byref(s)), "dq_nvfp4_sizes")
    return c.value, s.value


def mxfp4_sizes(rows: int, cols: int):
    c, s = ctypes.c_size_t(), ctypes.c_size_t()
    _check(_lib.dq_mxfp4_sizes(rows, cols, ctypes.byref(c), ctypes.byref(s)), "dq_mxfp4_sizes")
    return c.value, s.value


def lut_sizes(bits: int, mode: int, rows: int, cols: int):
    c, l, s = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    _check(_lib.dq_lut_sizes(bits, mode, rows, cols, ctypes.byref(c), ctypes.byref(l), ctypes.byref(s)),
           "dq_lut_sizes")
    return c.value, l.value, s.value


# ---------------------------------------------------------------- tensors
@dataclasses.dataclass
class NvFp4Tensor:
    """NVFP4 tensor in the tiled device layout of dq.h (uint8 buffers + fp32 G)."""
    codes: torch.Tensor
    scales: torch.Tensor
    G: torch.Tensor
    rows: int
    cols: int

    @staticmethod
    def empty(rows: int, cols: int, device="cuda") -> "NvFp4Tensor":
        cb, sb = nvfp4_sizes(rows, cols)
        return NvFp4Tensor(torch.empty(max(cb, 16), dtype=torch.uint8, device=device),
                           torch.empty(max(sb, 16), dtype=torch.uint8, device=device),
                           torch.empty(1, dtype=torch.float32, device=device), rows, cols)

    def desc(self) -> _NvFp4:
        return _NvFp4(self.codes.data_ptr(), self.scales.data_ptr(), self.G.data_ptr(), self.rows, self.cols)


@dataclasses.dataclass
class MxFp4Tensor:
    """MXFP4 tensor in the tiled device layout of dq.h (uint8 codes and E8M0 scales)."""
    codes: torch.Tensor
    scales: torch.Tensor
    rows: int
    cols: int

    @staticmethod
    def empty(rows: int, cols: int, device="cuda") -> "MxFp4Tensor":
        cb, sb = mxfp4_sizes(rows, cols)
        return MxFp4Tensor(torch.empty(max(cb, 16), dtype=torch.uint8, device=device),
                           torch.empty(max(sb, 16), dtype=torch.uint8, device=device), rows, cols)

    def desc(self) -> _MxFp4:
        return _MxFp4(self.codes.data_ptr(), self.scales.data_ptr(), self.rows, self.cols)


@dataclasses.dataclass
class LutWeight:
    """LUT weight (PER_ROW or PAPER_GRID) in the tiled device layout of dq.h."""
    codes: torch.Tensor
    lut: torch.Tensor
    scales: Optional[torch.Tensor]
    G: Optional[torch.Tensor]
    rows: int
    cols: int
    bits: int
    mode: int

    @staticmethod
    def empty(rows: int, cols: int, bits: int = 3, mode: int = LUT_PER_ROW, device="cuda") -> "LutWeight":
        cb, lb, sb = lut_sizes(bits, mode, rows, cols)
        scales = torch.empty(max(sb, 16), dtype=torch.uint8, device=device) if mode == LUT_PAPER_GRID else None
        G = torch.empty(1, dtype=torch.float32, device=device) if mode == LUT_PAPER_GRID else None
        return LutWeight(torch.empty(max(cb, 16), dtype=torch.uint8, device=device),
                         torch.empty(max(lb // 2, 8), dtype=torch.int16, device=device), scales, G,
                         rows, cols, bits, mode)

    def desc(self) -> _Lut:
        return _Lut(self.codes.data_ptr(), self.lut.data_ptr(), _ptr(self.scales), _ptr(self.G),
                    self.rows, self.cols, self.bits, self.mode)

    def nbytes(self) -> int:
        n = self.codes.numel() + self.lut.numel() * 2
        if self.scales is not None:
            n += self.scales.numel() + 4
        return n


def _as_u16(x: torch.Tensor) -> torch.Tensor:
    if x.dtype == torch.bfloat16:
        return x.view(torch.int16)
    if x.dtype in (torch.int16, torch.uint16):
        return x
    raise TypeError("activations must be bf16 (or their 16-bit patterns)")


# ---------------------------------------------------------------- calls
def dq_pack_nvfp4(W: torch.Tensor, G_override: Optional[torch.Tensor] = None, out: Optional[NvFp4Tensor] = None,
                  stream=None) -> NvFp4Tensor:
    assert W.dtype == torch.float32 and W.is_contiguous() and W.dim() == 2
    N, K = W.shape
    out = NvFp4Tensor.empty(N, K, W.device) if out is None else out
    d = out.desc()
    _check(_lib.dq_pack_nvfp4(W.data_ptr(), N, K, _ptr(G_override), ctypes.byref(d), _stream(stream)),
           "dq_pack_nvfp4")
    return out


def dq_pack_lut3(W: torch.Tensor, bits: int = 3, mode: int = LUT_PER_ROW, grid=None,
                 out: Optional[LutWeight] = None, stream=None) -> LutWeight:
    assert W.dtype == torch.float32 and W.is_contiguous() and W.dim() == 2
    N, K = W.shape
    out = LutWeight.empty(N, K, bits, mode, W.device) if out is None else out
    d = out.desc()
    gbuf = None
    if grid is not None:
        import numpy as np
        g = np.ascontiguousarray(np.asarray(grid, dtype=np.float16).view(np.uint16))
        gbuf = ctypes.cast((ctypes.c_uint16 * len(g))(*[int(v) for v in g]), ctypes.c_void_p)
    _check(_lib.dq_pack_lut3(W.data_ptr(), N, K, bits, mode, gbuf, ctypes.byref(d), _stream(stream)),
           "dq_pack_lut3")
    return out


def dq_quantize_act_nvfp4(X: torch.Tensor, G_static: Optional[torch.Tensor] = None,
                          out: Optional[NvFp4Tensor] = None, stream=None) -> NvFp4Tensor:
    X = _as_u16(X)
    assert X.is_contiguous() and X.dim() == 2
    M, K = X.shape
    out = NvFp4Tensor.empty(M, K, X.device) if out is None else out
    d = out.desc()
    _check(_lib.dq_quantize_act_nvfp4(X.data_ptr(), M, K, _ptr(G_static), ctypes.byref(d), _stream(stream)),
           "dq_quantize_act_nvfp4")
    return out


def dq_prefill_gemm_workspace_size(M: int, K: int) -> int:
    """Workspace bytes of dq_prefill_gemm's fused path (X given) for an [M, K] activation."""
    out = ctypes.c_size_t()
    _check(_lib.dq_prefill_gemm_workspace_size(M, K, ctypes.byref(out)), "dq_prefill_gemm_workspace_size")
    return out.value


def dq_prefill_gemm(W: NvFp4Tensor, A: Optional[NvFp4Tensor] = None, X: Optional[torch.Tensor] = None,
                    G_x_static: Optional[torch.Tensor] = None, out_kind: int = OUT_F32,
                    Y: Optional[torch.Tensor] = None, G_out_static: Optional[torch.Tensor] = None,
                    Yq: Optional[NvFp4Tensor] = None, epilogue_flags: int = 0, stream=None,
                    workspace: Optional[torch.Tensor] = None):
    M = A.rows if A is not None else X.shape[0]
    if X is not None and workspace is None:
        # the NVFP4 copy of X, from torch's stream-ordered caching allocator
        workspace = torch.empty(max(dq_prefill_gemm_workspace_size(M, W.cols), 16), dtype=torch.uint8,
                                device=W.codes.device)
    ws_ptr, ws_bytes = (workspace.data_ptr(), workspace.numel() * workspace.element_size()) \
        if workspace is not None else (None, 0)
    n_out = W.rows // 2 if (epilogue_flags & EPI_SWIGLU) else W.rows
    dev = W.codes.device
    if out_kind == OUT_NVFP4:
        Yq = NvFp4Tensor.empty(M, n_out, dev) if Yq is None else Yq
    elif Y is None:
        Y = torch.empty((M, n_out), dtype=torch.float32 if out_kind == OUT_F32 else torch.bfloat16, device=dev)
    da = A.desc() if A is not None else None
    dw = W.desc()
    dyq = Yq.desc() if Yq is not None else None
    xp = _as_u16(X).data_ptr() if X is not None else None
    _check(_lib.dq_prefill_gemm(ctypes.byref(da) if da is not None else None, xp, _ptr(G_x_static),
                                ctypes.byref(dw), M, out_kind, _ptr(Y), _ptr(G_out_static),
                                ctypes.byref(dyq) if dyq is not None else None, epilogue_flags, ws_ptr, ws_bytes,
                                _stream(stream)),
           "dq_prefill_gemm")
    return Yq if out_kind == OUT_NVFP4 else Y


def dq_rmsnorm_quantize_act_nvfp4(X: torch.Tensor, gamma: torch.Tensor, eps: float = 1e-6,
                                  G_static: Optional[torch.Tensor] = None, out: Optional[NvFp4Tensor] = None,
                                  stream=None) -> NvFp4Tensor:
    X, gamma = _as_u16(X), _as_u16(gamma)
    assert X.is_contiguous() and X.dim() == 2 and gamma.is_contiguous() and gamma.numel() == X.shape[1]
    M, K = X.shape
    out = NvFp4Tensor.empty(M, K, X.device) if out is None else out
    d = out.desc()
    ws = torch.empty(max(4 * M, 16), dtype=torch.uint8, device=X.device)   # per-row statistics
    _check(_lib.dq_rmsnorm_quantize_act_nvfp4(X.data_ptr() if X.numel() else None,
                                              gamma.data_ptr() if gamma.numel() else None, eps, M, K,
                                              _ptr(G_static), ctypes.byref(d), ws.data_ptr(), ws.numel(),
                                              _stream(stream)), "dq_rmsnorm_quantize_act_nvfp4")
    return out


def dq_autocast_lut_to_nvfp4(W: LutWeight, G_override: Optional[torch.Tensor] = None,
                             out: Optional[NvFp4Tensor] = None, stream=None) -> NvFp4Tensor:
    out = NvFp4Tensor.empty(W.rows, W.cols, W.codes.device) if out is None else out
    dw, do = W.desc(), out.desc()
    _check(_lib.dq_autocast_lut_to_nvfp4(ctypes.byref(dw), _ptr(G_override), ctypes.byref(do), _stream(stream)),
           "dq_autocast_lut_to_nvfp4")
    return out


def dq_pack_mxfp4(W: torch.Tensor, out: Optional[MxFp4Tensor] = None, stream=None) -> MxFp4Tensor:
    assert W.dtype == torch.float32 and W.is_contiguous() and W.dim() == 2
    N, K = W.shape
    out = MxFp4Tensor.empty(N, K, W.device) if out is None else out
    d = out.desc()
    _check(_lib.dq_pack_mxfp4(W.data_ptr(), N, K, ctypes.byref(d), _stream(stream)), "dq_pack_mxfp4")
    return out


def dq_quantize_act_mxfp4(X: torch.Tensor, out: Optional[MxFp4Tensor] = None, stream=None) -> MxFp4Tensor:
    X = _as_u16(X)
    assert X.is_contiguous() and X.dim() == 2
    M, K = X.shape
    out = MxFp4Tensor.empty(M, K, X.device) if out is None else out
    d = out.desc()
    _check(_lib.dq_quantize_act_mxfp4(X.data_ptr(), M, K, ctypes.byref(d), _stream(stream)),
           "dq_quantize_act_mxfp4")
    return out


def dq_prefill_gemm_mxfp4(A: MxFp4Tensor, W: MxFp4Tensor, out_kind: int = OUT_F32,
                          Y: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    if Y is None:
        Y = torch.empty((A.rows, W.rows), dtype=torch.float32 if out_kind == OUT_F32 else torch.bfloat16,
                        device=W.codes.device)
    da, dw = A.desc(), W.desc()
    _check(_lib.dq_prefill_gemm_mxfp4(ctypes.byref(da), ctypes.byref(dw), out_kind, Y.data_ptr(), _stream(stream)),
           "dq_prefill_gemm_mxfp4")
    return Y


_gemv_ws_cache: dict = {}


def dq_decode_gemv_nvfp4_workspace_size(B: int, W: NvFp4Tensor) -> int:
    """Workspace bytes dq_decode_gemv_nvfp4 needs for batch B."""
    key = ("nvfp4", B, W.rows, W.cols, W.codes.device.index)
    n = _gemv_ws_cache.get(key)
    if n is None:
        out = ctypes.c_size_t()
        _check(_lib.dq_decode_gemv_nvfp4_workspace_size(B, ctypes.byref(W.desc()), ctypes.byref(out)),
               "dq_decode_gemv_nvfp4_workspace_size")
        n = _gemv_ws_cache[key] = out.value
    return n


def dq_decode_gemv_nvfp4(x: torch.Tensor, W: NvFp4Tensor, out_kind: int = OUT_F32, y: Optional[torch.Tensor] = None,
                         stream=None, workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    x = _as_u16(x)
    assert x.is_contiguous() and x.dim() == 2
    B = x.shape[0]
    if y is None:
        y = torch.empty((B, W.rows), dtype=torch.float32 if out_kind == OUT_F32 else torch.bfloat16,
                        device=x.device)
    if workspace is None:
        n = dq_decode_gemv_nvfp4_workspace_size(B, W)
        if n:
            workspace = torch.empty(n, dtype=torch.uint8, device=x.device)
    ws_ptr, ws_bytes = (workspace.data_ptr(), workspace.numel() * workspace.element_size()) if workspace is not None \
        else (None, 0)
    d = W.desc()
    _check(_lib.dq_decode_gemv_nvfp4(x.data_ptr(), B, ctypes.byref(d), out_kind, y.data_ptr(), ws_ptr, ws_bytes,
                                     _stream(stream)), "dq_decode_gemv_nvfp4")
    return y


def dq_decode_gemv_workspace_size(B: int, W: LutWeight) -> int:
    """Workspace bytes dq_decode_gemv needs for batch B (0 for B = 1)."""
    key = (B, W.rows, W.cols, W.bits, W.mode, W.codes.device.index)
    n = _gemv_ws_cache.get(key)
    if n is None:
        out = ctypes.c_size_t()
        _check(_lib.dq_decode_gemv_workspace_size(B, ctypes.byref(W.desc()), ctypes.byref(out)),
               "dq_decode_gemv_workspace_size")
        n = _gemv_ws_cache[key] = out.value
    return n


def dq_decode_gemv(x: torch.Tensor, W: LutWeight, out_kind: int = OUT_F32, y: Optional[torch.Tensor] = None,
                   stream=None, workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    x = _as_u16(x)
    assert x.is_contiguous() and x.dim() == 2
    B = x.shape[0]
    if y is None:
        y = torch.empty((B, W.rows), dtype=torch.float32 if out_kind == OUT_F32 else torch.bfloat16,
                        device=x.device)
    if workspace is None:
        # torch's caching allocator hands out stream-ordered memory
        n = dq_decode_gemv_workspace_size(B, W)
        if n:
            workspace = torch.empty(n, dtype=torch.uint8, device=x.device)
    ws_ptr, ws_bytes = (workspace.data_ptr(), workspace.numel() * workspace.element_size()) if workspace is not None \
        else (None, 0)
    d = W.desc()
    _check(_lib.dq_decode_gemv(x.data_ptr(), B, ctypes.byref(d), out_kind, y.data_ptr(), ws_ptr, ws_bytes,
                               _stream(stream)), "dq_decode_gemv")
    return y


NOALLOC_SCRATCH_BYTES = 16 << 20


def dq_decode_gemv_noalloc(x: torch.Tensor, W: LutWeight, out_kind: int = OUT_F32,
                           y: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """dq_decode_gemv without a workspace: split-K partial sums go to the
    library's static per-GPU scratch (calls overlapping on one GPU race)."""
    x = _as_u16(x)
    assert x.is_contiguous() and x.dim() == 2
    B = x.shape[0]
    if y is None:
        y = torch.empty((B, W.rows), dtype=torch.float32 if out_kind == OUT_F32 else torch.bfloat16,
                        device=x.device)
    d = W.desc()
    _check(_lib.dq_decode_gemv_noalloc(x.data_ptr(), B, ctypes.byref(d), out_kind, y.data_ptr(), _stream(stream)),
           "dq_decode_gemv_noalloc")
    return y


__all__ = [n for n in dir() if n.startswith(("dq_", "DQ", "OUT_", "LUT_", "EPI_")) or n in
           ("NvFp4Tensor", "MxFp4Tensor", "LutWeight", "nvfp4_sizes", "mxfp4_sizes", "lut_sizes", "abi_version", "lib", "EXPORTED",
            "NOALLOC_SCRATCH_BYTES")]
