// W4A4 NVFP4 GEMM on gfx950 (paper App. A "NVFP4"; App. C "Compute and
// timing scope": the prefill projections).
//
//   Y[m, n] = G_a * G_w * sum_k e_a[m,k] s_a[m,k/16] * e_w[n,k] s_w[n,k/16]
//
// gfx950's block-scaled MFMA (v_mfma_scale_*_f8f6f4) takes one power-of-two
// (E8M0) scale per 32 elements, while NVFP4 carries an E4M3 scale (3 mantissa
// bits) per 16.  The product of an E2M1 element and an E4M3 scale has at most
// 6 significant bits and lies in [2^-10, 2688], so it is exact in fp16.  This
// kernel therefore dequantizes both operands exactly to fp16 in registers
// (hardware E2M1 -> fp16 conversion, then one packed fp16 multiply by the
// block scale) and accumulates v_mfma_f32_32x32x16_f16 products in fp32.  The
// global scales are applied once in the epilogue.
//
// Structure: a 256-thread workgroup covers a 256x256 output tile as 2x2
// wavefronts of 128x128; each wavefront keeps 4x4 32x32 fp32 accumulator
// blocks.  Operands stream straight from the tiled NVFP4 layout: one 32-row x
// 64-column tile is 1 KiB of codes, read by one wavefront-wide 16-byte load
// (lane l: row l%32, columns 32*(l/32) .. +31 of the tile), plus 2 scale bytes
// per lane.  Within a 64-column step, MFMA sub-step s consumes columns
// 32*(l/32) + 8s .. +7 on both operands (a permutation of K shared by A and W,
// which leaves the sum unchanged).  The next step's operands are loaded while
// the current step's MFMAs run.
#include "dq_device.hpp"
#include "dq_internal.hpp"

namespace dq {

namespace {

constexpr int kWaveM = 128;
constexpr int kWaveN = 128;
constexpr int kBlkM = 256;
constexpr int kBlkN = 256;

struct Operand {
  uint4_t code[4];
  uint32_t scale[4];
};

__device__ inline void load_operand(const uint8_t* __restrict__ codes, const uint8_t* __restrict__ scales,
                                    int64_t tile_row0, int64_t n_tile_rows, int64_t kt, int64_t KT,
                                    int lane, Operand& op) {
  const int lane_code = (lane & 31) * 32 + (lane >> 5) * 16;
  const int lane_scale = (lane & 31) * 4 + (lane >> 5) * 2;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int64_t tr = tile_row0 + b;
    if (tr < n_tile_rows) {
      const int64_t tile = tr * KT + kt;
      op.code[b] = *reinterpret_cast<const uint4_t*>(codes + tile * 1024 + lane_code);
      op.scale[b] = *reinterpret_cast<const uint16_t*>(scales + tile * 128 + lane_scale);
    } else {
      op.code[b] = uint4_t{0u, 0u, 0u, 0u};
      op.scale[b] = 0u;
    }
  }
}

// 8 E2M1 codes (one dword) times an fp16 block scale -> 8 exact fp16 values.
__device__ inline half8_t dequant8(uint32_t w, half2_t s) {
  half2_t p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 0) * s;
  half2_t p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 1) * s;
  half2_t p2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 2) * s;
  half2_t p3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 3) * s;
  return half8_t{p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

// two E4M3 scale bytes (lo: columns +0..15, hi: +16..31) -> fp16 broadcast pairs
__device__ inline void scale_pairs(uint32_t sc, half2_t& lo, half2_t& hi) {
  half2_t s = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sc, 1.0f, false);
  lo = half2_t{s[0], s[0]};
  hi = half2_t{s[1], s[1]};
}

template <int OUT>
__global__ __launch_bounds__(256, 1) void nvfp4_gemm_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales, const float* __restrict__ Ga,
    const uint8_t* __restrict__ w_codes, const uint8_t* __restrict__ w_scales, const float* __restrict__ Gw,
    int64_t M, int64_t N, int64_t a_tile_rows, int64_t w_tile_rows, int64_t KT, void* __restrict__ Y,
    int64_t tiles_n) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t bm = blockIdx.x / tiles_n, bn = blockIdx.x % tiles_n;
  const int64_t m0 = bm * kBlkM + (wave & 1) * kWaveM;
  const int64_t n0 = bn * kBlkN + (wave >> 1) * kWaveN;
  const int64_t a_tr0 = m0 / 32, w_tr0 = n0 / 32;

  float16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = float16_t{};

  Operand a_cur, w_cur, a_nxt, w_nxt;
  load_operand(a_codes, a_scales, a_tr0, a_tile_rows, 0, KT, lane, a_cur);
  load_operand(w_codes, w_scales, w_tr0, w_tile_rows, 0, KT, lane, w_cur);

  for (int64_t kt = 0; kt < KT; ++kt) {
    if (kt + 1 < KT) {
      load_operand(a_codes, a_scales, a_tr0, a_tile_rows, kt + 1, KT, lane, a_nxt);
      load_operand(w_codes, w_scales, w_tr0, w_tile_rows, kt + 1, KT, lane, w_nxt);
    }
    half2_t a_s[4][2], w_s[4][2];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      scale_pairs(a_cur.scale[b], a_s[b][0], a_s[b][1]);
      scale_pairs(w_cur.scale[b], w_s[b][0], w_s[b][1]);
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      half8_t af[4], wf[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        af[b] = dequant8(a_cur.code[b][s], a_s[b][s >> 1]);
        wf[b] = dequant8(w_cur.code[b][s], w_s[b][s >> 1]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[i], wf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) {
      a_cur = a_nxt;
      w_cur = w_nxt;
    }
  }

  const float g = (*Ga) * (*Gw);
  const int col_in = lane & 31;
  const int row_off = 4 * (lane >> 5);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t col = n0 + j * 32 + col_in;
      if (col >= N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + i * 32 + 8 * (r >> 2) + row_off + (r & 3);
        if (row < M) {
          const float v = acc[i][j][r] * g;
          if (OUT == 0)
            reinterpret_cast<float*>(Y)[row * N + col] = v;
          else
            reinterpret_cast<uint16_t*>(Y)[row * N + col] = (uint16_t)f32_to_bf16_rne(v);
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s) {
  if (a.M == 0 || a.N == 0) return hipSuccess;
  const int64_t a_tile_rows = round_up(a.M, 32) / 32;
  const int64_t w_tile_rows = round_up(a.N, 32) / 32;
  const int64_t KT = round_up(a.K, 64) / 64;
  const int64_t tiles_m = (a.M + kBlkM - 1) / kBlkM, tiles_n = (a.N + kBlkN - 1) / kBlkN;
  const dim3 grid((unsigned)(tiles_m * tiles_n));
  if (a.out_kind == 0)
    hipLaunchKernelGGL(nvfp4_gemm_kernel<0>, grid, dim3(256), 0, s, a.A.codes, a.A.scales, a.A.G,
                       a.W.codes, a.W.scales, a.W.G, a.M, a.N, a_tile_rows, w_tile_rows, KT, a.Y, tiles_n);
  else
    hipLaunchKernelGGL(nvfp4_gemm_kernel<1>, grid, dim3(256), 0, s, a.A.codes, a.A.scales, a.A.G,
                       a.W.codes, a.W.scales, a.W.G, a.M, a.N, a_tile_rows, w_tile_rows, KT, a.Y, tiles_n);
  return hipGetLastError();
}

}  // namespace dq
