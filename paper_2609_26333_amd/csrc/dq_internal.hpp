// Internal launcher interface between the C ABI (dq_api.cpp) and the kernel
// translation units.  Views carry validated device pointers and logical sizes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dq {

struct NvFp4View {
  uint8_t* codes;
  uint8_t* scales;
  float* G;
  int64_t rows, cols;
};

struct LutView {
  uint8_t* codes;
  uint16_t* lut;
  uint8_t* scales;
  float* G;
  int64_t rows, cols;
  int bits, mode;
};

// a1 / a2: NVFP4 quantization (quant.hip)
hipError_t launch_quantize_act(const uint16_t* X, int64_t M, int64_t K, const float* G_static,
                               const NvFp4View& out, hipStream_t s);
hipError_t launch_pack_nvfp4(const float* W, int64_t N, int64_t K, const float* G_override,
                             const NvFp4View& out, hipStream_t s);

// G = fp32(max|x| / 2688) of n fp32 values into *G (1 when all are zero):
// the global scale of the NVFP4 weight rule, shared by the paper-grid LUT
// packer (quant.hip)
hipError_t launch_global_scale_f32(const float* x, int64_t n, float* G, hipStream_t s);

// a5: LUT packing (pack_lut.hip)
hipError_t launch_pack_lut(const float* W, int64_t N, int64_t K, const uint16_t* grid_host,
                           const LutView& out, hipStream_t s);

// RMSNorm fused with the NVFP4 activation quantizer (quant.hip): per-row
// statistics into the workspace ws (4 M bytes; NULL: pooled staging), then
// the tile quantizer on the normalized values; G_static == nullptr takes G
// from the normalized tensor's amax
hipError_t launch_rmsnorm_quantize_act(const uint16_t* X, const uint16_t* gamma, float eps, int64_t M, int64_t K,
                                       const float* G_static, const NvFp4View& out, void* ws, hipStream_t s);

// LUT -> NVFP4 autocast (pack_lut.hip): dequantize to a pooled fp32
// staging copy, then the NVFP4 weight packing
hipError_t launch_autocast_lut(const LutView& w, const float* G_override, const NvFp4View& out, hipStream_t s);

// a3 / a4: NVFP4 GEMM (gemm.hip)
struct GemmArgs {
  NvFp4View A;            // valid when X == nullptr
  const uint16_t* X;      // fused activation quantization input, or nullptr
  const float* G_x;       // static activation scale for the fused path
  NvFp4View W;
  int64_t M, N, K;
  int out_kind;
  void* Y;
  const float* G_out;     // static output scale (NVFP4 output)
  NvFp4View Yq;
  int flags;
};
hipError_t launch_gemm(const GemmArgs& a, hipStream_t s);

// MXFP4 (mxfp4.hip): codes and E8M0 scales in the 32x64-tile layout of dq.h
struct MxView {
  uint8_t* codes;
  uint8_t* scales;
  int64_t rows, cols;
};
// x: bf16 bits (is_bf16) or fp32, [rows, cols] row-major
hipError_t launch_mx_quantize(const void* x, bool is_bf16, int64_t rows, int64_t cols, const MxView& out,
                              hipStream_t s);
struct MxGemmArgs {
  MxView A, W;
  int64_t M, N, K;
  int out_kind;   // 0 fp32, 1 bf16
  void* Y;
};
hipError_t launch_mx_gemm(const MxGemmArgs& a, hipStream_t s);

// Number of compute units of the current device (queried once per device).
int num_cus();

// Stream-ordered staging from the library's memory pool on the current
// device (created on first use; it keeps freed memory for later calls instead
// of returning it at every free).  Release with hipFreeAsync on the same
// stream.
hipError_t pool_alloc_async(void** p, size_t bytes, hipStream_t s);

// Column split of an M x N GEMM between workgroup tiles of bm_full x bn_full
// (columns 0 .. split-1) and smaller tiles of bm_half x bn_half (the rest),
// `slots` resident workgroups: the split minimises the modelled time, a round
// of full tiles costing 1 and a round of small tiles half_cost, ties going to
// more full tiles.  Returns a multiple of bn_full, or N.
constexpr double kHalfRound = 0.65;
inline int64_t gemm_column_split(int64_t M, int64_t N, int64_t bm_full, int64_t bn_full, int64_t bm_half,
                                 int64_t bn_half, int64_t slots, double half_cost) {
  const int64_t tm = (M + bm_full - 1) / bm_full, tmh = (M + bm_half - 1) / bm_half;
  const int64_t panels = (N + bn_full - 1) / bn_full;
  int64_t best = panels;
  double best_cost = 1e300;
  for (int64_t p = panels; p >= 0; --p) {
    const int64_t split = p * bn_full < N ? p * bn_full : N;
    const int64_t full = tm * p, half = tmh * ((N - split + bn_half - 1) / bn_half);
    const double cost = (double)((full + slots - 1) / slots) + half_cost * (double)((half + slots - 1) / slots);
    if (cost < best_cost - 1e-9) {
      best_cost = cost;
      best = p;
    }
  }
  return best * bn_full < N ? best * bn_full : N;
}

// NVFP4A16 decode GEMV (gemv_nvfp4.hip): bf16 x [B, K] times NVFP4 weights
// [N, K].  ws: workspace of at least gemv_nvfp4_workspace_bytes(B, N, K)
// bytes, or NULL to take it from the pool.
size_t gemv_nvfp4_workspace_bytes(int64_t B, int64_t N, int64_t K);
hipError_t launch_gemv_nvfp4(const uint16_t* x, int64_t B, const NvFp4View& w, int out_kind, void* y, void* ws,
                             hipStream_t s);

// a6: LUT GEMV (gemv.hip).  ws: workspace of at least
// gemv_workspace_bytes(B, w) bytes, or NULL to take it from the pool.
size_t gemv_workspace_bytes(int64_t B, const LutView& w);
// The no-allocation variant's per-device static scratch (gemv.hip): its size,
// and its device address on the current device (looked up on first use).
size_t gemv_noalloc_scratch_bytes();
hipError_t gemv_noalloc_scratch(void** ptr);
hipError_t launch_gemv(const uint16_t* x, int64_t B, const LutView& w, int out_kind, void* y, void* ws,
                       hipStream_t s);

}  // namespace dq
