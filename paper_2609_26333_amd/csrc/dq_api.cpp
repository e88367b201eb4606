// C ABI of libdq (declared in include/dq.h): host-side argument validation,
// size queries and dispatch to the kernel launchers.  Validation runs before
// any HIP call, so rejected calls launch nothing.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "dq.h"
#include "dq_internal.hpp"

namespace {

thread_local char g_last_error[512] = "";

dq_status fail(dq_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

dq_status ok() {
  g_last_error[0] = '\0';
  return DQ_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int64_t rup(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

dq_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  if (e == hipErrorNotSupported) return fail(DQ_ERR_UNSUPPORTED, "%s: configuration not supported", what);
  return fail(DQ_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

dq_status check_nvfp4(const dq_nvfp4_t* t, const char* name, int64_t rows, int64_t cols) {
  if (t == nullptr) return fail(DQ_ERR_INVALID_ARG, "%s is NULL", name);
  if (t->codes == nullptr || t->scales == nullptr || t->G == nullptr)
    return fail(DQ_ERR_INVALID_ARG, "%s has a NULL buffer", name);
  if (!aligned(t->codes, 16) || !aligned(t->scales, 16) || !aligned(t->G, 4))
    return fail(DQ_ERR_INVALID_ARG, "%s buffers must be 16-byte aligned (G 4-byte)", name);
  if (t->rows != rows || t->cols != cols)
    return fail(DQ_ERR_INVALID_ARG, "%s is %lldx%lld, expected %lldx%lld", name, (long long)t->rows,
                (long long)t->cols, (long long)rows, (long long)cols);
  return DQ_OK;
}

dq::NvFp4View view(const dq_nvfp4_t* t) { return dq::NvFp4View{t->codes, t->scales, t->G, t->rows, t->cols}; }

dq_status check_mxfp4(const dq_mxfp4_t* t, const char* name, int64_t rows, int64_t cols) {
  if (t == nullptr) return fail(DQ_ERR_INVALID_ARG, "%s is NULL", name);
  if (t->rows < 0 || t->cols < 0 || t->cols % 32 != 0)
    return fail(DQ_ERR_INVALID_ARG, "%s: rows >= 0 and cols %% 32 == 0 required", name);
  if (rows >= 0 && (t->rows != rows || t->cols != cols))
    return fail(DQ_ERR_INVALID_ARG, "%s is %lldx%lld, expected %lldx%lld", name, (long long)t->rows,
                (long long)t->cols, (long long)rows, (long long)cols);
  if (t->rows * t->cols > 0 && (t->codes == nullptr || t->scales == nullptr))
    return fail(DQ_ERR_INVALID_ARG, "%s has a NULL buffer", name);
  if (!aligned(t->codes, 16) || !aligned(t->scales, 16))
    return fail(DQ_ERR_INVALID_ARG, "%s buffers must be 16-byte aligned", name);
  return DQ_OK;
}

dq::MxView view(const dq_mxfp4_t* t) { return dq::MxView{t->codes, t->scales, t->rows, t->cols}; }

dq_status check_lut(const dq_lut_t* t, const char* name) {
  if (t == nullptr) return fail(DQ_ERR_INVALID_ARG, "%s is NULL", name);
  if (t->bits != 2 && t->bits != 3) return fail(DQ_ERR_INVALID_ARG, "%s.bits must be 2 or 3", name);
  if (t->mode != DQ_LUT_PER_ROW && t->mode != DQ_LUT_PAPER_GRID)
    return fail(DQ_ERR_INVALID_ARG, "%s.mode is not a DQ_LUT_* value", name);
  if (t->rows < 0 || t->cols < 0 || t->cols % 32 != 0)
    return fail(DQ_ERR_INVALID_ARG, "%s: rows >= 0 and cols %% 32 == 0 required", name);
  if (t->codes == nullptr || t->lut == nullptr) return fail(DQ_ERR_INVALID_ARG, "%s has a NULL buffer", name);
  if (!aligned(t->codes, 16) || !aligned(t->lut, 16))
    return fail(DQ_ERR_INVALID_ARG, "%s buffers must be 16-byte aligned", name);
  if (t->mode == DQ_LUT_PAPER_GRID) {
    if (t->scales == nullptr || t->G == nullptr)
      return fail(DQ_ERR_INVALID_ARG, "%s: PAPER_GRID needs scales and G", name);
    if (!aligned(t->scales, 16) || !aligned(t->G, 4))
      return fail(DQ_ERR_INVALID_ARG, "%s: scales must be 16-byte aligned, G 4-byte", name);
  }
  return DQ_OK;
}

dq::LutView view(const dq_lut_t* t) {
  return dq::LutView{t->codes, t->lut, t->scales, t->G, t->rows, t->cols, t->bits, t->mode};
}

double f16_value(uint16_t h) {
  const int e = (h >> 10) & 0x1F, m = h & 0x3FF;
  double v = e == 0 ? m * (1.0 / (1 << 24)) : (1.0 + m / 1024.0) * (double)(1ll << e) / (double)(1 << 15);
  return (h & 0x8000) ? -v : v;
}

}  // namespace

namespace dq {

int num_cus() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n > 0) return n;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
  cached[dev].store(n, std::memory_order_relaxed);
  return n;
}

hipError_t pool_alloc_async(void** p, size_t bytes, hipStream_t s) {
  static std::atomic<hipMemPool_t> pools[64];
  static std::mutex mu;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipMallocAsync(p, bytes, s);
  hipMemPool_t pool = pools[dev].load(std::memory_order_acquire);
  if (pool == nullptr) {
    std::lock_guard<std::mutex> lock(mu);
    pool = pools[dev].load(std::memory_order_relaxed);
    if (pool == nullptr) {
      hipMemPoolProps props{};
      props.allocType = hipMemAllocationTypePinned;
      props.location.type = hipMemLocationTypeDevice;
      props.location.id = dev;
      e = hipMemPoolCreate(&pool, &props);
      if (e != hipSuccess) return e;
      uint64_t keep = UINT64_MAX;   // never trim: later calls reuse the memory
      e = hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
      if (e != hipSuccess) return e;
      pools[dev].store(pool, std::memory_order_release);
    }
  }
  return hipMallocFromPoolAsync(p, bytes, pool, s);
}

}  // namespace dq

extern "C" {

int dq_abi_version(void) { return DQ_ABI_VERSION; }

const char* dq_status_string(dq_status s) {
  switch (s) {
    case DQ_OK: return "DQ_OK";
    case DQ_ERR_INVALID_ARG: return "DQ_ERR_INVALID_ARG";
    case DQ_ERR_UNSUPPORTED: return "DQ_ERR_UNSUPPORTED";
    case DQ_ERR_HIP: return "DQ_ERR_HIP";
    default: return "DQ_ERR_UNKNOWN";
  }
}

const char* dq_last_error(void) { return g_last_error; }

dq_status dq_nvfp4_sizes(int64_t rows, int64_t cols, size_t* code_bytes, size_t* scale_bytes) {
  if (code_bytes == nullptr || scale_bytes == nullptr) return fail(DQ_ERR_INVALID_ARG, "NULL output pointer");
  if (rows < 0 || cols < 0 || cols % 16 != 0)
    return fail(DQ_ERR_INVALID_ARG, "rows >= 0, cols >= 0 and cols %% 16 == 0 required");
  const int64_t r = rup(rows, 32), c = rup(cols, 64);
  *code_bytes = (size_t)(r * c / 2);
  *scale_bytes = (size_t)(r * c / 16);
  return ok();
}

dq_status dq_mxfp4_sizes(int64_t rows, int64_t cols, size_t* code_bytes, size_t* scale_bytes) {
  if (code_bytes == nullptr || scale_bytes == nullptr) return fail(DQ_ERR_INVALID_ARG, "NULL output pointer");
  if (rows < 0 || cols < 0 || cols % 32 != 0)
    return fail(DQ_ERR_INVALID_ARG, "rows >= 0, cols >= 0 and cols %% 32 == 0 required");
  const int64_t c = rup(cols, 64);
  *code_bytes = (size_t)(rup(rows, 32) * c / 2);
  *scale_bytes = (size_t)(rup(rows, 128) * c / 32);
  return ok();
}

dq_status dq_lut_sizes(int bits, int mode, int64_t rows, int64_t cols, size_t* code_bytes, size_t* lut_bytes,
                       size_t* scale_bytes) {
  if (code_bytes == nullptr || lut_bytes == nullptr || scale_bytes == nullptr)
    return fail(DQ_ERR_INVALID_ARG, "NULL output pointer");
  if (bits != 2 && bits != 3) return fail(DQ_ERR_INVALID_ARG, "bits must be 2 or 3");
  if (mode != DQ_LUT_PER_ROW && mode != DQ_LUT_PAPER_GRID) return fail(DQ_ERR_INVALID_ARG, "bad LUT mode");
  if (rows < 0 || cols < 0 || cols % 32 != 0)
    return fail(DQ_ERR_INVALID_ARG, "rows >= 0, cols >= 0 and cols %% 32 == 0 required");
  const int64_t tr = rup(rows, 16) / 16, tc = rup(cols, 128) / 128;
  const int64_t gb = bits == 3 ? 12 : 8;
  *code_bytes = (size_t)(tr * tc * 64 * gb);
  if (mode == DQ_LUT_PER_ROW) {
    *lut_bytes = (size_t)(tr * 16 * (1 << bits) * 2);
    *scale_bytes = 0;
  } else {
    *lut_bytes = (size_t)((1 << bits) * 2);
    *scale_bytes = (size_t)(tr * tc * 128);
  }
  return ok();
}

dq_status dq_pack_nvfp4(const float* W, int64_t N, int64_t K, const float* G_override, const dq_nvfp4_t* out,
                        void* stream) {
  if (W == nullptr && N * K > 0) return fail(DQ_ERR_INVALID_ARG, "W is NULL");
  if (!aligned(W, 16)) return fail(DQ_ERR_INVALID_ARG, "W must be 16-byte aligned");
  if (N < 0 || K < 0 || K % 16 != 0) return fail(DQ_ERR_INVALID_ARG, "N >= 0, K >= 0, K %% 16 == 0 required");
  if (G_override != nullptr && !aligned(G_override, 4)) return fail(DQ_ERR_INVALID_ARG, "G_override misaligned");
  dq_status st = check_nvfp4(out, "out", N, K);
  if (st != DQ_OK) return st;
  return hip_status(dq::launch_pack_nvfp4(W, N, K, G_override, view(out), (hipStream_t)stream), "dq_pack_nvfp4");
}

dq_status dq_pack_lut3(const float* W, int64_t N, int64_t K, int bits, int mode, const uint16_t* grid,
                       const dq_lut_t* out, void* stream) {
  if (W == nullptr && N * K > 0) return fail(DQ_ERR_INVALID_ARG, "W is NULL");
  if (!aligned(W, 16)) return fail(DQ_ERR_INVALID_ARG, "W must be 16-byte aligned");
  if (N < 0 || K < 0 || K % 32 != 0) return fail(DQ_ERR_INVALID_ARG, "N >= 0, K >= 0, K %% 32 == 0 required");
  if (bits != 2 && bits != 3) return fail(DQ_ERR_INVALID_ARG, "bits must be 2 or 3");
  if (mode != DQ_LUT_PER_ROW && mode != DQ_LUT_PAPER_GRID) return fail(DQ_ERR_INVALID_ARG, "bad LUT mode");
  dq_status st = check_lut(out, "out");
  if (st != DQ_OK) return st;
  if (out->rows != N || out->cols != K || out->bits != bits || out->mode != mode)
    return fail(DQ_ERR_INVALID_ARG, "out descriptor does not match N, K, bits, mode");
  if (mode == DQ_LUT_PER_ROW && K > 32768)
    return fail(DQ_ERR_UNSUPPORTED, "PER_ROW packing sorts a row in LDS: K <= 32768");
  if (mode == DQ_LUT_PER_ROW && K == 0 && N > 0)
    return fail(DQ_ERR_INVALID_ARG, "PER_ROW needs K > 0 (bin means of empty rows are undefined)");
  if (mode == DQ_LUT_PAPER_GRID && grid != nullptr) {
    int zeros = 0;
    for (int i = 0; i < (1 << bits); ++i) {
      if ((grid[i] & 0x7FFF) == 0) ++zeros;
      if ((grid[i] & 0x7C00) == 0x7C00) return fail(DQ_ERR_INVALID_ARG, "grid must be finite");
      if (i > 0 && !(f16_value(grid[i]) > f16_value(grid[i - 1])))
        return fail(DQ_ERR_INVALID_ARG, "grid must be strictly ascending");
    }
    if (zeros != 1) return fail(DQ_ERR_INVALID_ARG, "grid must contain exactly one zero level");
  }
  return hip_status(dq::launch_pack_lut(W, N, K, grid, view(out), (hipStream_t)stream), "dq_pack_lut3");
}

dq_status dq_rmsnorm_quantize_act_nvfp4(const uint16_t* X, const uint16_t* gamma, float eps, int64_t M, int64_t K,
                                        const float* G_static, const dq_nvfp4_t* out, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  if (M < 0 || K < 0 || K % 16 != 0) return fail(DQ_ERR_INVALID_ARG, "M >= 0, K >= 0, K %% 16 == 0 required");
  if ((X == nullptr && M * K > 0) || !aligned(X, 16)) return fail(DQ_ERR_INVALID_ARG, "X must be 16-byte aligned");
  if ((gamma == nullptr && K > 0) || !aligned(gamma, 16))
    return fail(DQ_ERR_INVALID_ARG, "gamma must be 16-byte aligned");
  if (!(eps >= 0.0f) || eps > 3.0e38f) return fail(DQ_ERR_INVALID_ARG, "eps must be finite and >= 0");
  if (G_static != nullptr && !aligned(G_static, 4)) return fail(DQ_ERR_INVALID_ARG, "G_static misaligned");
  if (workspace != nullptr && (!aligned(workspace, 16) || workspace_bytes < (size_t)M * 4))
    return fail(DQ_ERR_INVALID_ARG, "workspace must be 16-byte aligned and hold 4 M bytes");
  dq_status st = check_nvfp4(out, "out", M, K);
  if (st != DQ_OK) return st;
  return hip_status(dq::launch_rmsnorm_quantize_act(X, gamma, eps, M, K, G_static, view(out), workspace,
                                                    (hipStream_t)stream),
                    "dq_rmsnorm_quantize_act_nvfp4");
}

dq_status dq_autocast_lut_to_nvfp4(const dq_lut_t* W, const float* G_override, const dq_nvfp4_t* out,
                                   void* stream) {
  dq_status st = check_lut(W, "W");
  if (st != DQ_OK) return st;
  if (G_override != nullptr && !aligned(G_override, 4)) return fail(DQ_ERR_INVALID_ARG, "G_override misaligned");
  st = check_nvfp4(out, "out", W->rows, W->cols);
  if (st != DQ_OK) return st;
  return hip_status(dq::launch_autocast_lut(view(W), G_override, view(out), (hipStream_t)stream),
                    "dq_autocast_lut_to_nvfp4");
}

dq_status dq_quantize_act_nvfp4(const uint16_t* X, int64_t M, int64_t K, const float* G_static,
                                const dq_nvfp4_t* out, void* stream) {
  if (X == nullptr && M * K > 0) return fail(DQ_ERR_INVALID_ARG, "X is NULL");
  if (!aligned(X, 16)) return fail(DQ_ERR_INVALID_ARG, "X must be 16-byte aligned");
  if (M < 0 || K < 0 || K % 16 != 0) return fail(DQ_ERR_INVALID_ARG, "M >= 0, K >= 0, K %% 16 == 0 required");
  if (G_static != nullptr && !aligned(G_static, 4)) return fail(DQ_ERR_INVALID_ARG, "G_static misaligned");
  dq_status st = check_nvfp4(out, "out", M, K);
  if (st != DQ_OK) return st;
  return hip_status(dq::launch_quantize_act(X, M, K, G_static, view(out), (hipStream_t)stream),
                    "dq_quantize_act_nvfp4");
}

// Bytes of the NVFP4 copy of X that the fused path of dq_prefill_gemm stages:
// codes and scales in the tiled layout, plus 16 bytes for its global scale.
static size_t fused_staging_bytes(int64_t M, int64_t K) {
  const int64_t r = rup(M, 32), c = rup(K, 64);
  return (size_t)(r * c / 2) + (size_t)(r * c / 16) + 16;
}

dq_status dq_prefill_gemm_workspace_size(int64_t M, int64_t K, size_t* bytes) {
  if (bytes == nullptr) return fail(DQ_ERR_INVALID_ARG, "bytes is NULL");
  if (M < 0 || K < 0 || K % 16 != 0) return fail(DQ_ERR_INVALID_ARG, "M >= 0, K >= 0, K %% 16 == 0 required");
  *bytes = fused_staging_bytes(M, K);
  return ok();
}

dq_status dq_prefill_gemm(const dq_nvfp4_t* A, const uint16_t* X, const float* G_x_static, const dq_nvfp4_t* W,
                          int64_t M, int out_kind, void* Y, const float* G_out_static, const dq_nvfp4_t* Yq,
                          int epilogue_flags, void* workspace, size_t workspace_bytes, void* stream) {
  // exactly one of A and X; an empty fused call (M == 0) may pass X = NULL
  if (A != nullptr && X != nullptr) return fail(DQ_ERR_INVALID_ARG, "give exactly one of A and X");
  if (A == nullptr && X == nullptr && !(M == 0 && G_x_static != nullptr))
    return fail(DQ_ERR_INVALID_ARG, "give exactly one of A and X");
  if (W == nullptr) return fail(DQ_ERR_INVALID_ARG, "W is NULL");
  if (M < 0) return fail(DQ_ERR_INVALID_ARG, "M < 0");
  const int64_t N = W->rows, K = W->cols;
  dq_status st = check_nvfp4(W, "W", N, K);
  if (st != DQ_OK) return st;
  if (N < 0 || K < 0 || K % 16 != 0) return fail(DQ_ERR_INVALID_ARG, "W: rows >= 0 and cols %% 16 == 0 required");
  if (K >= ((int64_t)1 << 23)) return fail(DQ_ERR_UNSUPPORTED, "K < 2^23 required (32-bit row-panel offsets)");
  if (A != nullptr) {
    st = check_nvfp4(A, "A", M, K);
    if (st != DQ_OK) return st;
  } else {
    if (G_x_static == nullptr || !aligned(G_x_static, 4))
      return fail(DQ_ERR_INVALID_ARG, "the fused path needs an aligned G_x_static");
    if (!aligned(X, 16)) return fail(DQ_ERR_INVALID_ARG, "X must be 16-byte aligned");
    if (workspace != nullptr && (!aligned(workspace, 16) || workspace_bytes < fused_staging_bytes(M, K)))
      return fail(DQ_ERR_INVALID_ARG, "workspace must be 16-byte aligned and hold dq_prefill_gemm_workspace_size() bytes");
  }
  if (epilogue_flags & ~DQ_EPI_SWIGLU) return fail(DQ_ERR_INVALID_ARG, "unknown epilogue flag");
  const bool swiglu = (epilogue_flags & DQ_EPI_SWIGLU) != 0;
  if (swiglu && N % 32 != 0) return fail(DQ_ERR_INVALID_ARG, "SwiGLU needs W rows %% 32 == 0 (gate/up groups of 16)");
  const int64_t Nout = swiglu ? N / 2 : N;
  if (out_kind != DQ_OUT_F32 && out_kind != DQ_OUT_BF16 && out_kind != DQ_OUT_NVFP4)
    return fail(DQ_ERR_INVALID_ARG, "bad out_kind");
  if (out_kind == DQ_OUT_NVFP4) {
    if (Y != nullptr) return fail(DQ_ERR_INVALID_ARG, "NVFP4 output: Y must be NULL");
    if (G_out_static == nullptr || !aligned(G_out_static, 4))
      return fail(DQ_ERR_INVALID_ARG, "NVFP4 output needs an aligned G_out_static");
    if (Yq == nullptr) return fail(DQ_ERR_INVALID_ARG, "NVFP4 output needs Yq");
    if (Nout % 16 != 0) return fail(DQ_ERR_INVALID_ARG, "NVFP4 output needs output columns %% 16 == 0");
    st = check_nvfp4(Yq, "Yq", M, Nout);
    if (st != DQ_OK) return st;
  } else {
    if (Yq != nullptr) return fail(DQ_ERR_INVALID_ARG, "Yq is only used with NVFP4 output");
    if (Y == nullptr && M * Nout > 0) return fail(DQ_ERR_INVALID_ARG, "Y is NULL");
    if (!aligned(Y, 16)) return fail(DQ_ERR_INVALID_ARG, "Y must be 16-byte aligned");
  }
  dq::GemmArgs a{};
  hipStream_t hs = (hipStream_t)stream;
  void* staging = nullptr;   // pooled staging to release after the GEMM
  if (A) {
    a.A = view(A);
  } else {
    // Fused activation quantization: one streaming pass of X into the NVFP4
    // copy in the workspace (or in stream-ordered pool staging), then the
    // GEMM, all on `stream`.
    const int64_t r = rup(M, 32), c = rup(K, 64);
    const size_t code_bytes = (size_t)(r * c / 2), scale_bytes = (size_t)(r * c / 16);
    void* base_ptr = workspace;
    if (base_ptr == nullptr) {
      hipError_t e = dq::pool_alloc_async(&staging, fused_staging_bytes(M, K), hs);
      if (e != hipSuccess) return hip_status(e, "dq_prefill_gemm (staging)");
      base_ptr = staging;
    }
    uint8_t* base = static_cast<uint8_t*>(base_ptr);
    a.A = dq::NvFp4View{base, base + code_bytes, reinterpret_cast<float*>(base + code_bytes + scale_bytes), M, K};
    hipError_t e = dq::launch_quantize_act(X, M, K, G_x_static, a.A, hs);
    if (e != hipSuccess) {
      if (staging != nullptr) (void)hipFreeAsync(staging, hs);
      return hip_status(e, "dq_prefill_gemm (activation quantization)");
    }
  }
  a.X = X;
  a.G_x = G_x_static;
  a.W = view(W);
  a.M = M;
  a.N = N;
  a.K = K;
  a.out_kind = out_kind;
  a.Y = Y;
  a.G_out = G_out_static;
  if (Yq) a.Yq = view(Yq);
  a.flags = epilogue_flags;
  hipError_t e = dq::launch_gemm(a, hs);
  if (staging != nullptr) {
    const hipError_t f = hipFreeAsync(staging, hs);
    if (e == hipSuccess) e = f;
  }
  return hip_status(e, "dq_prefill_gemm");
}

dq_status dq_decode_gemv_nvfp4_workspace_size(int64_t B, const dq_nvfp4_t* W, size_t* bytes) {
  if (W == nullptr) return fail(DQ_ERR_INVALID_ARG, "W is NULL");
  if (W->rows < 0 || W->cols < 0 || W->cols % 16 != 0)
    return fail(DQ_ERR_INVALID_ARG, "W: rows >= 0, cols >= 0 and cols %% 16 == 0 required");
  if (B < 1 || B > 16) return fail(DQ_ERR_INVALID_ARG, "1 <= B <= 16 required");
  if (bytes == nullptr) return fail(DQ_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = dq::gemv_nvfp4_workspace_bytes(B, W->rows, W->cols);
  return DQ_OK;
}

dq_status dq_decode_gemv_nvfp4(const uint16_t* x, int64_t B, const dq_nvfp4_t* W, int out_kind, void* y,
                               void* workspace, size_t workspace_bytes, void* stream) {
  if (W == nullptr) return fail(DQ_ERR_INVALID_ARG, "W is NULL");
  dq_status st = check_nvfp4(W, "W", W->rows, W->cols);
  if (st != DQ_OK) return st;
  if (W->rows < 0 || W->cols < 0 || W->cols % 16 != 0)
    return fail(DQ_ERR_INVALID_ARG, "W: rows >= 0, cols >= 0 and cols %% 16 == 0 required");
  if (B < 1 || B > 16) return fail(DQ_ERR_INVALID_ARG, "1 <= B <= 16 required");
  if ((x == nullptr && W->cols > 0) || !aligned(x, 16))
    return fail(DQ_ERR_INVALID_ARG, "x must be 16-byte aligned and non-NULL unless K == 0");
  if (out_kind != DQ_OUT_F32 && out_kind != DQ_OUT_BF16) return fail(DQ_ERR_INVALID_ARG, "bad out_kind");
  if (y == nullptr && W->rows > 0) return fail(DQ_ERR_INVALID_ARG, "y is NULL");
  if (!aligned(y, 16)) return fail(DQ_ERR_INVALID_ARG, "y must be 16-byte aligned");
  if (workspace != nullptr) {
    if (!aligned(workspace, 16)) return fail(DQ_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    if (workspace_bytes < dq::gemv_nvfp4_workspace_bytes(B, W->rows, W->cols))
      return fail(DQ_ERR_INVALID_ARG, "workspace smaller than dq_decode_gemv_nvfp4_workspace_size()");
  }
  return hip_status(dq::launch_gemv_nvfp4(x, B, view(W), out_kind, y, workspace, (hipStream_t)stream),
                    "dq_decode_gemv_nvfp4");
}

dq_status dq_pack_mxfp4(const float* W, int64_t N, int64_t K, const dq_mxfp4_t* out, void* stream) {
  if (W == nullptr && N * K > 0) return fail(DQ_ERR_INVALID_ARG, "W is NULL");
  if (!aligned(W, 16)) return fail(DQ_ERR_INVALID_ARG, "W must be 16-byte aligned");
  if (N < 0 || K < 0 || K % 32 != 0) return fail(DQ_ERR_INVALID_ARG, "N >= 0, K >= 0, K %% 32 == 0 required");
  dq_status st = check_mxfp4(out, "out", N, K);
  if (st != DQ_OK) return st;
  return hip_status(dq::launch_mx_quantize(W, false, N, K, view(out), (hipStream_t)stream), "dq_pack_mxfp4");
}

dq_status dq_quantize_act_mxfp4(const uint16_t* X, int64_t M, int64_t K, const dq_mxfp4_t* out, void* stream) {
  if (X == nullptr && M * K > 0) return fail(DQ_ERR_INVALID_ARG, "X is NULL");
  if (!aligned(X, 16)) return fail(DQ_ERR_INVALID_ARG, "X must be 16-byte aligned");
  if (M < 0 || K < 0 || K % 32 != 0) return fail(DQ_ERR_INVALID_ARG, "M >= 0, K >= 0, K %% 32 == 0 required");
  dq_status st = check_mxfp4(out, "out", M, K);
  if (st != DQ_OK) return st;
  return hip_status(dq::launch_mx_quantize(X, true, M, K, view(out), (hipStream_t)stream), "dq_quantize_act_mxfp4");
}

dq_status dq_prefill_gemm_mxfp4(const dq_mxfp4_t* A, const dq_mxfp4_t* W, int out_kind, void* Y, void* stream) {
  dq_status st = check_mxfp4(W, "W", -1, -1);
  if (st != DQ_OK) return st;
  if (A == nullptr) return fail(DQ_ERR_INVALID_ARG, "A is NULL");
  st = check_mxfp4(A, "A", A->rows, W->cols);
  if (st != DQ_OK) return st;
  if (out_kind != DQ_OUT_F32 && out_kind != DQ_OUT_BF16) return fail(DQ_ERR_INVALID_ARG, "bad out_kind");
  if (W->cols >= ((int64_t)1 << 23)) return fail(DQ_ERR_UNSUPPORTED, "K < 2^23 required (32-bit row-panel offsets)");
  if (Y == nullptr && A->rows * W->rows > 0) return fail(DQ_ERR_INVALID_ARG, "Y is NULL");
  if (!aligned(Y, 16)) return fail(DQ_ERR_INVALID_ARG, "Y must be 16-byte aligned");
  dq::MxGemmArgs a{};
  a.A = view(A);
  a.W = view(W);
  a.M = A->rows;
  a.N = W->rows;
  a.K = W->cols;
  a.out_kind = out_kind;
  a.Y = Y;
  return hip_status(dq::launch_mx_gemm(a, (hipStream_t)stream), "dq_prefill_gemm_mxfp4");
}

dq_status dq_decode_gemv_workspace_size(int64_t B, const dq_lut_t* W, size_t* bytes) {
  dq_status st = check_lut(W, "W");
  if (st != DQ_OK) return st;
  if (B < 1 || B > 16) return fail(DQ_ERR_INVALID_ARG, "1 <= B <= 16 required");
  if (bytes == nullptr) return fail(DQ_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = dq::gemv_workspace_bytes(B, view(W));
  return DQ_OK;
}

static dq_status check_gemv(const uint16_t* x, int64_t B, const dq_lut_t* W, int out_kind, void* y) {
  dq_status st = check_lut(W, "W");
  if (st != DQ_OK) return st;
  if (B < 1 || B > 16) return fail(DQ_ERR_INVALID_ARG, "1 <= B <= 16 required");
  if ((x == nullptr && W->cols > 0) || !aligned(x, 16))
    return fail(DQ_ERR_INVALID_ARG, "x must be 16-byte aligned and non-NULL unless K == 0");
  if (out_kind != DQ_OUT_F32 && out_kind != DQ_OUT_BF16) return fail(DQ_ERR_INVALID_ARG, "bad out_kind");
  if (y == nullptr && W->rows > 0) return fail(DQ_ERR_INVALID_ARG, "y is NULL");
  if (!aligned(y, 16)) return fail(DQ_ERR_INVALID_ARG, "y must be 16-byte aligned");
  return DQ_OK;
}

dq_status dq_decode_gemv_noalloc(const uint16_t* x, int64_t B, const dq_lut_t* W, int out_kind, void* y,
                                 void* stream) {
  dq_status st = check_gemv(x, B, W, out_kind, y);
  if (st != DQ_OK) return st;
  const size_t need = dq::gemv_workspace_bytes(B, view(W));
  if (need > dq::gemv_noalloc_scratch_bytes())
    return fail(DQ_ERR_UNSUPPORTED, "dq_decode_gemv_noalloc: this call needs %zu bytes of scratch, the library's "
                "static scratch holds %zu; use dq_decode_gemv with a workspace", need,
                dq::gemv_noalloc_scratch_bytes());
  void* ws = nullptr;
  hipError_t e = dq::gemv_noalloc_scratch(&ws);
  if (e != hipSuccess) return hip_status(e, "dq_decode_gemv_noalloc (scratch address)");
  return hip_status(dq::launch_gemv(x, B, view(W), out_kind, y, ws, (hipStream_t)stream), "dq_decode_gemv_noalloc");
}

dq_status dq_decode_gemv(const uint16_t* x, int64_t B, const dq_lut_t* W, int out_kind, void* y, void* workspace,
                         size_t workspace_bytes, void* stream) {
  dq_status st = check_gemv(x, B, W, out_kind, y);
  if (st != DQ_OK) return st;
  if (workspace != nullptr) {
    if (!aligned(workspace, 16)) return fail(DQ_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    if (workspace_bytes < dq::gemv_workspace_bytes(B, view(W)))
      return fail(DQ_ERR_INVALID_ARG, "workspace smaller than dq_decode_gemv_workspace_size()");
  }
  return hip_status(dq::launch_gemv(x, B, view(W), out_kind, y, workspace, (hipStream_t)stream), "dq_decode_gemv");
}

}  // extern "C"
