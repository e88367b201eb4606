// MXFP4 W4A4 prefill on gfx950: the quantizer (weights and bf16
// activations) and the block-scaled GEMM.
//
// The paper runs MXFP4 in place of NVFP4 for a model released natively in
// that format (Sec. 4, the accuracy table and the evaluation arms).  The
// format is the OCP Microscaling one: E2M1 elements, one E8M0 (power-of-two)
// scale per 32 consecutive elements along K, no tensor scale.
//
// Quantization of a block with largest magnitude a:
//   e = floor(log2 a) - 2 (E2M1's largest power of two is 4), clamped to
//   [-127, 127], and -127 for an all-zero block; scale code e + 127;
//   q_i = E2M1(x_i * 2^-e), nearest with ties to even, saturating at 6,
//   magnitude-zero codes carry sign 0.
// x_i * 2^-e is exact in fp32 (a power-of-two scaling whose result is never
// subnormal for a non-zero code), and the E2M1 rounding is the hardware
// conversion at unit scale, as in the NVFP4 quantizer.
//
// GEMM:  Y[m, n] = sum_b 2^(sa[m,b] + sw[n,b] - 254) sum_{k in b} e_a[m,k] e_w[n,k]
// maps one-to-one onto v_mfma_scale_f32_32x32x64_f8f6f4 with FP4 operands:
// lane l of a 32x64 operand tile holds row l%32, columns 32*(l/32)..+31 (16
// bytes, low nibble first) and the E8M0 scale of exactly that 32-block, so
// the raw code bytes and scale bytes are the MFMA operands (no dequantization
// at all).  Element products and the block scaling are exact; the only
// rounding is the fp32 accumulation.
//
// Structure (same staging scheme as the NVFP4 kernel):
//  * a workgroup of WM x WN wavefronts covers a (32*TM*WM) x (32*TN*WN)
//    output tile, each wavefront 32*TM x 32*TN (TM x TN blocks of 32x32);
//  * a ring of LDS stages, one 64-column K step each (code tiles of 1 KiB,
//    scale tiles of 64 bytes), filled by direct global->LDS loads up to S
//    steps ahead of the consumer, one workgroup barrier per K step;
//  * the operands of K step kt+1 are read from LDS into registers while the
//    MFMAs of step kt run;
//  * workgroups are numbered so that the 8 XCDs each own a contiguous range
//    of output tiles (column-panel-major).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "dq_device.hpp"
#include "dq_internal.hpp"

namespace dq {

namespace {

typedef int int8v_t __attribute__((ext_vector_type(8)));

// floor(log2 a) for a finite a > 0 (normal or subnormal fp32)
__device__ inline int floor_log2(float a) {
  const uint32_t b = __float_as_uint(a);
  const int E = (int)(b >> 23);
  return E != 0 ? E - 127 : -149 + (31 - (int)__clz(b));
}

// ---------------------------------------------------------------- quantizer
// One wavefront per 32x64 tile: lane l = row l%32, columns 32*(l/32)..+31 of
// the tile (one MX block).  Codes: the lane's 16 bytes at 32*(l%32) +
// 16*(l/32) of the tile (row-major 32 bytes per row); scales: byte l of the
// tile's 64.  Rows past `rows` and columns past `cols` produce zero codes and
// scale code 0.
template <typename T>
__device__ inline void load_block(const T* __restrict__ src, float (&v)[32]);

template <>
__device__ inline void load_block<uint16_t>(const uint16_t* __restrict__ src, float (&v)[32]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint4_t w = *reinterpret_cast<const uint4_t*>(src + 8 * q);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[8 * q + 2 * i] = bf16_lo(w[i]);
      v[8 * q + 2 * i + 1] = bf16_hi(w[i]);
    }
  }
}

template <>
__device__ inline void load_block<float>(const float* __restrict__ src, float (&v)[32]) {
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const float4_t w = *reinterpret_cast<const float4_t*>(src + 4 * q);
    v[4 * q] = w[0];
    v[4 * q + 1] = w[1];
    v[4 * q + 2] = w[2];
    v[4 * q + 3] = w[3];
  }
}

template <typename T>
__global__ __launch_bounds__(256) void mx_quantize_kernel(const T* __restrict__ x, int64_t rows, int64_t cols,
                                                          int64_t tiles_r, int64_t tiles_c,
                                                          uint8_t* __restrict__ codes, uint8_t* __restrict__ scales) {
  const int lane = threadIdx.x & 63;
  const int64_t tile = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tile >= tiles_r * tiles_c) return;
  const int64_t tr = tile / tiles_c, tc = tile - tr * tiles_c;
  const int r = lane & 31, h = lane >> 5;
  const int64_t row = tr * 32 + r, col = tc * 64 + h * 32;
  float v[32];
  if (row < rows && col < cols) {
    load_block<T>(x + row * cols + col, v);
  } else {
#pragma unroll
    for (int i = 0; i < 32; ++i) v[i] = 0.0f;
  }
  float a = 0.0f;
#pragma unroll
  for (int i = 0; i < 32; ++i) a = fmaxf(a, fabsf(v[i]));
  int e = a > 0.0f ? floor_log2(a) - 2 : -127;
  e = e < -127 ? -127 : (e > 127 ? 127 : e);
  // 2^-e as fp32: -e lies in [-125, 127] for finite inputs (a < 2^128 gives
  // e <= 125), so the biased exponent 127 - e is in [2, 254]
  const float p = __uint_as_float((uint32_t)(127 - e) << 23);
  uint4_t out;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t w = 0u;
    w = cvt_pk_fp4<0>(w, v[8 * q] * p, v[8 * q + 1] * p);
    w = cvt_pk_fp4<1>(w, v[8 * q + 2] * p, v[8 * q + 3] * p);
    w = cvt_pk_fp4<2>(w, v[8 * q + 4] * p, v[8 * q + 5] * p);
    w = cvt_pk_fp4<3>(w, v[8 * q + 6] * p, v[8 * q + 7] * p);
    out[q] = fp4_canonical_zero(w);
  }
  *reinterpret_cast<uint4_t*>(codes + tile * 1024 + r * 32 + h * 16) = out;
  scales[tile * 64 + lane] = (uint8_t)(e + 127);
}

// ---------------------------------------------------------------- GEMM
constexpr int kMxLdsBudget = 150 * 1024;

template <int TM, int TN, int WM, int WN>
struct MxGeo {
  static constexpr int tm = TM, tn = TN, wm = WM, wn = WN;
  static constexpr int waves = WM * WN;
  static constexpr int threads = 64 * waves;
  static constexpr int bm = 32 * TM * WM;
  static constexpr int bn = 32 * TN * WN;
  static constexpr int at = bm / 32;   // A tiles per K step
  static constexpr int wt = bn / 32;   // W tiles per K step
  // one stage = one 64-column K step: A codes, W codes, A scales, W scales
  static constexpr int a_codes = 0;
  static constexpr int w_codes = at * 1024;
  static constexpr int a_scales = w_codes + wt * 1024;
  static constexpr int w_scales = a_scales + at * 64;
  static constexpr int bytes = w_scales + wt * 64;
  static constexpr int stages_fit = kMxLdsBudget / bytes;
  static constexpr int stages = stages_fit < 6 ? stages_fit : 6;
  // direct loads per stage: one per code tile; one dword load covers 4 scale tiles
  static constexpr int code_loads = at + wt;
  static constexpr int scale_loads = (at + wt) / 4;
  static_assert((at + wt) % 4 == 0 && at % 4 == 0, "scale tiles are loaded four at a time");
  static_assert(code_loads % waves == 0 && scale_loads <= waves, "uniform load distribution");
  static constexpr int loads_per_wave = code_loads / waves + 1;   // + one scale load (some waves: a dummy)
  static_assert(stages >= 4, "LDS ring needs four stages");
};

template <int n>
__device__ inline void mx_wait_vm() {
  __builtin_amdgcn_s_waitcnt((n & 0xF) | (0x7 << 4) | (0xF << 8) | ((n >> 4) << 14));
}

__device__ inline void mx_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <class Gm, int OUT>
__global__ __launch_bounds__(Gm::threads, 1) void mxfp4_gemm_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales, const uint8_t* __restrict__ w_codes,
    const uint8_t* __restrict__ w_scales, int64_t M, int64_t N, int64_t a_tiles_r, int64_t w_tiles_r, int64_t KT,
    void* __restrict__ Y, int64_t tiles_m, int64_t tiles_n, int64_t n_off) {
  constexpr int S = Gm::stages;
  constexpr int TM = Gm::tm, TN = Gm::tn;
  constexpr int L = Gm::loads_per_wave;
  extern __shared__ __align__(16) uint8_t smem[];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t nb = tiles_m * tiles_n;
  int64_t logical = blockIdx.x;
  if (nb % 8 == 0) logical = (int64_t)(blockIdx.x % 8) * (nb / 8) + blockIdx.x / 8;
  const int64_t bm = logical % tiles_m, bn = logical / tiles_m;
  const int wm = wave % Gm::wm, wn = wave / Gm::wm;
  const int64_t a_tr0 = bm * Gm::at, w_tr0 = n_off / 32 + bn * Gm::wt;
  const int64_t m0 = bm * Gm::bm + wm * 32 * TM;
  const int64_t n0 = n_off + bn * Gm::bn + wn * 32 * TN;
  const int KTi = (int)KT;

  // Direct loads: code tiles t = wave + waves*u (A tiles first, then W);
  // scale instruction `wave` covers 4 tiles (16 lanes each).  Tiles past the
  // end of an operand read its last row tile (in bounds): they only feed
  // output rows / columns that are never stored.
  const int chunk = 2 * (lane & 31) + (lane >> 5);
  constexpr int CPW = Gm::code_loads / Gm::waves;
  const uint8_t* c_src[CPW];
  int c_dst[CPW];
#pragma unroll
  for (int u = 0; u < CPW; ++u) {
    const int t = wave + Gm::waves * u;
    const bool is_a = t < Gm::at;
    const int b = is_a ? t : t - Gm::at;
    const int64_t tr = min((is_a ? a_tr0 : w_tr0) + b, (is_a ? a_tiles_r : w_tiles_r) - 1);
    c_src[u] = (is_a ? a_codes : w_codes) + tr * KT * 1024 + chunk * 16;
    c_dst[u] = (is_a ? Gm::a_codes : Gm::w_codes) + b * 1024;
  }
  const int st = min(wave, Gm::scale_loads - 1) * 4 + (lane >> 4);   // scale tile of this lane
  const bool s_is_a = st < Gm::at;
  const int sb = s_is_a ? st : st - Gm::at;
  const int64_t s_tr = min((s_is_a ? a_tr0 : w_tr0) + sb, (s_is_a ? a_tiles_r : w_tiles_r) - 1);
  const uint8_t* s_src = (s_is_a ? a_scales : w_scales) + s_tr * KT * 64 + (lane & 15) * 4;
  // waves past the scale instructions repeat the last one (same bytes, same place)
  const int s_dst = (Gm::a_scales + (min(wave, Gm::scale_loads - 1) * 4) * 64);
  auto issue = [&](int kt) {
    uint8_t* stage = smem + (kt % S) * Gm::bytes;
#pragma unroll
    for (int u = 0; u < CPW; ++u)
      __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(c_src[u] + (size_t)kt * 1024),
                                       reinterpret_cast<void*>(stage + c_dst[u]), 16, 0, 0);
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(s_src + (size_t)kt * 64),
                                     reinterpret_cast<void*>(stage + s_dst), 4, 0, 0);
  };

  float16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = float16_t{};

  struct Ops {
    uint4_t a[TM], w[TN];
    uint32_t sa[TM], sw[TN];
  };
  const int a_rd = Gm::a_codes + wm * TM * 1024 + lane * 16;
  const int w_rd = Gm::w_codes + wn * TN * 1024 + lane * 16;
  const int as_rd = Gm::a_scales + wm * TM * 64 + lane;
  const int ws_rd = Gm::w_scales + wn * TN * 64 + lane;
  auto read_ops = [&](int kt, Ops& o) {
    const uint8_t* stg = smem + (kt % S) * Gm::bytes;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      o.a[i] = *reinterpret_cast<const uint4_t*>(stg + a_rd + i * 1024);
      o.sa[i] = stg[as_rd + i * 64];
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      o.w[j] = *reinterpret_cast<const uint4_t*>(stg + w_rd + j * 1024);
      o.sw[j] = stg[ws_rd + j * 64];
    }
  };
  auto mfmas = [&](const Ops& o) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int8v_t av = {(int)o.a[i][0], (int)o.a[i][1], (int)o.a[i][2], (int)o.a[i][3], 0, 0, 0, 0};
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int8v_t wv = {(int)o.w[j][0], (int)o.w[j][1], (int)o.w[j][2], (int)o.w[j][3], 0, 0, 0, 0};
        // A and W in E2M1 (format 4), scales in byte 0 of the scale operands
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, wv, acc[i][j], 4, 4, 0, (int)o.sa[i], 0,
                                                                   (int)o.sw[j]);
      }
    }
  };
  // this wavefront's loads of stage `need` have landed, with stages up to
  // `last` issued
  auto wait_stage = [&](int need, int last) {
    const int ahead = max(0, min(last, KTi - 1) - need);
    static_assert(S - 2 <= 4 && 4 * L <= 63, "wait table");
    if (ahead >= 4) mx_wait_vm<4 * L>();
    else if (ahead == 3) mx_wait_vm<3 * L>();
    else if (ahead == 2) mx_wait_vm<2 * L>();
    else if (ahead == 1) mx_wait_vm<L>();
    else mx_wait_vm<0>();
  };

  // prologue: stages 0 .. S-1 in flight, stage 0 landed everywhere
#pragma unroll
  for (int s = 0; s < S; ++s)
    if (s < KTi) issue(s);
  wait_stage(0, S - 1);
  mx_barrier();
  Ops o0, o1;
  read_ops(0, o0);
  // Step kt (operands of stage kt in `cur`, read during the previous step):
  // wait for this wavefront's loads of stage kt+1 and for this wavefront's
  // reads of stage kt, then the barrier: stage kt+1 has landed everywhere and
  // every wavefront is done with stage kt's slot, which is refilled with
  // stage kt+S.  Stage kt+1's operands are read while step kt's MFMAs run.
  // The sched_barriers keep the compiler from sinking the MFMAs past the
  // next step's waits and barrier (the matrix cores would idle through them).
  auto step = [&](int kt, Ops& cur, Ops& nxt) {
    const bool more = kt + 1 < KTi;
    if (more) wait_stage(kt + 1, kt + S - 1);
    __builtin_amdgcn_s_waitcnt((0x3F & 0xF) | (0x7 << 4) | (0x0 << 8) | ((0x3F >> 4) << 14));   // lgkmcnt(0)
    mx_barrier();
    if (kt + S < KTi) issue(kt + S);
    if (more) read_ops(kt + 1, nxt);
    __builtin_amdgcn_sched_barrier(0);
    mfmas(cur);
    __builtin_amdgcn_sched_barrier(0);
  };
  int kt = 0;
  for (; kt + 1 < KTi; kt += 2) {
    step(kt, o0, o1);
    step(kt + 1, o1, o0);
  }
  if (kt < KTi) step(kt, o0, o1);

  const int col_in = lane & 31;
  const int row_off = 4 * (lane >> 5);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int64_t col = n0 + j * 32 + col_in;
      if (col >= N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + i * 32 + 8 * (r >> 2) + row_off + (r & 3);
        if (row < M) {
          if (OUT == 0)
            reinterpret_cast<float*>(Y)[row * N + col] = acc[i][j][r];
          else
            reinterpret_cast<uint16_t*>(Y)[row * N + col] = (uint16_t)f32_to_bf16_rne(acc[i][j][r]);
        }
      }
    }
  }
}

template <class Gm>
hipError_t launch_mx_geo(const MxGemmArgs& a, int64_t n_off, int64_t n_end, hipStream_t s) {
  const int64_t a_tiles_r = round_up(a.M, 32) / 32;
  const int64_t w_tiles_r = round_up(a.N, 32) / 32;
  const int64_t KT = round_up(a.K, 64) / 64;
  const int64_t tiles_m = (a.M + Gm::bm - 1) / Gm::bm, tiles_n = (n_end - n_off + Gm::bn - 1) / Gm::bn;
  const size_t lds = (size_t)Gm::stages * Gm::bytes;
  typedef void (*kern_t)(const uint8_t*, const uint8_t*, const uint8_t*, const uint8_t*, int64_t, int64_t, int64_t,
                         int64_t, int64_t, void*, int64_t, int64_t, int64_t);
  const kern_t kern = a.out_kind == 0 ? mxfp4_gemm_kernel<Gm, 0> : mxfp4_gemm_kernel<Gm, 1>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)(tiles_m * tiles_n)), dim3(Gm::threads), lds, s, a.A.codes, a.A.scales,
                     a.W.codes, a.W.scales, a.M, a.N, a_tiles_r, w_tiles_r, KT, a.Y, tiles_m, tiles_n, n_off);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_mx_quantize(const void* x, bool is_bf16, int64_t rows, int64_t cols, const MxView& out,
                              hipStream_t s) {
  const int64_t tiles_r = round_up(rows, 32) / 32, tiles_c = round_up(cols, 64) / 64;
  const int64_t tiles = tiles_r * tiles_c;
  if (tiles == 0) return hipSuccess;
  const unsigned grid = (unsigned)((tiles + 3) / 4);
  if (is_bf16)
    hipLaunchKernelGGL(mx_quantize_kernel<uint16_t>, dim3(grid), dim3(256), 0, s, static_cast<const uint16_t*>(x),
                       rows, cols, tiles_r, tiles_c, out.codes, out.scales);
  else
    hipLaunchKernelGGL(mx_quantize_kernel<float>, dim3(grid), dim3(256), 0, s, static_cast<const float*>(x), rows,
                       cols, tiles_r, tiles_c, out.codes, out.scales);
  return hipGetLastError();
}

hipError_t launch_mx_gemm(const MxGemmArgs& a, hipStream_t s) {
  if (a.M == 0 || a.N == 0) return hipSuccess;
  // 256x256 workgroup tiles: four wavefronts of 128x128, one per SIMD
  using Full = MxGeo<4, 4, 2, 2>;
  return launch_mx_geo<Full>(a, 0, a.N, s);
}

}  // namespace dq
