// MXFP4 W4A4 prefill on gfx950: the quantizer (weights and bf16
// activations) and the block-scaled GEMM.
//
// The paper runs MXFP4 in place of NVFP4 for a model released natively in
// that format (Sec. 3.2, the accuracy table of large LLMs, and its quantized
// arms).  The
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
//  * output tiles are handed out in bands of row panels, with each XCD taking
//    a compact sub-block of the tiles in flight (see gemm_tile_of).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <climits>
#include <type_traits>

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
// One workgroup per 4-tile scale group: wavefront q quantizes the 32x64 tile
// (4g + q, tc) in four passes of eight rows, eight lanes per row (8 elements
// each, so that a load instruction reads 128 contiguous bytes of each of 8
// bf16 rows); an MX block is the 4 lanes of a row that share its 32 columns,
// which exchange their maxima.  Codes: row-major 32 bytes per row of the
// tile, a lane's 4 bytes at 32 r + 4 (l % 8).  Scales: byte 4(r + 32h) + q of
// the group's 256 for row r and column half h, so that one dword per lane
// carries the scales of 4 row tiles (the GEMM's operand).  Rows past `rows`
// and columns past `cols` produce zero codes and scale code 0; tiles past the
// last row tile (group padding) get scale 0 only.
// Eight consecutive elements as fp32 (one 16-byte load for bf16, two for fp32).
template <typename T>
__device__ inline void load8(const T* __restrict__ src, float (&v)[8]);

template <>
__device__ inline void load8<uint16_t>(const uint16_t* __restrict__ src, float (&v)[8]) {
  const uint4_t w = *reinterpret_cast<const uint4_t*>(src);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = bf16_lo(w[i]);
    v[2 * i + 1] = bf16_hi(w[i]);
  }
}

template <>
__device__ inline void load8<float>(const float* __restrict__ src, float (&v)[8]) {
  const float4_t w0 = *reinterpret_cast<const float4_t*>(src);
  const float4_t w1 = *reinterpret_cast<const float4_t*>(src + 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[i] = w0[i];
    v[4 + i] = w1[i];
  }
}

template <typename T>
__global__ __launch_bounds__(256) void mx_quantize_kernel(const T* __restrict__ x, int64_t rows, int64_t cols,
                                                          int64_t tiles_r, int64_t tiles_c,
                                                          uint8_t* __restrict__ codes, uint8_t* __restrict__ scales) {
  __shared__ uint32_t s_grp[64];
  const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int64_t g = blockIdx.x / tiles_c, tc = blockIdx.x - g * tiles_c;
  const int64_t tr = 4 * g + q;
  // eight lanes per row (8 elements each: 128 contiguous bytes of bf16 per
  // row and load), eight rows per pass, four passes; an MX block is the
  // 4 lanes c & ~3 .. c | 3 of a row
  const int c = lane & 7, rr = lane >> 3;
  const int64_t col = tc * 64 + c * 8;
  const int64_t cc = min(col, cols - 8);   // cols % 32 == 0
  float v[4][8];
  bool ok[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t row = tr * 32 + 8 * i + rr;
    ok[i] = row < rows && col < cols;
    load8<T>(x + min(row, rows - 1) * cols + cc, v[i]);
  }
  uint8_t* sg = reinterpret_cast<uint8_t*>(s_grp);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float a = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      v[i][k] = ok[i] ? v[i][k] : 0.0f;
      a = fmaxf(a, fabsf(v[i][k]));
    }
    a = fmaxf(a, __shfl_xor(a, 1, 64));
    a = fmaxf(a, __shfl_xor(a, 2, 64));
    int e = a > 0.0f ? floor_log2(a) - 2 : -127;
    e = e < -127 ? -127 : (e > 127 ? 127 : e);
    const float p = __uint_as_float((uint32_t)(127 - e) << 23);
    const int r = 8 * i + rr;
    if (tr < tiles_r) {
      uint32_t w = 0u;
      w = cvt_pk_fp4<0>(w, v[i][0] * p, v[i][1] * p);
      w = cvt_pk_fp4<1>(w, v[i][2] * p, v[i][3] * p);
      w = cvt_pk_fp4<2>(w, v[i][4] * p, v[i][5] * p);
      w = cvt_pk_fp4<3>(w, v[i][6] * p, v[i][7] * p);
      *reinterpret_cast<uint32_t*>(codes + (tr * tiles_c + tc) * 1024 + r * 32 + c * 4) = fp4_canonical_zero(w);
    }
    if ((c & 3) == 0) sg[4 * (r + 32 * (c >> 2)) + q] = (uint8_t)(e + 127);
  }
  __syncthreads();
  if (q == 0) reinterpret_cast<uint32_t*>(scales + (g * tiles_c + tc) * 256)[lane] = s_grp[lane];
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
  static constexpr int a_scales = w_codes + wt * 1024;   // 4-tile scale groups of 256 bytes
  static constexpr int w_scales = a_scales + at * 64;
  static constexpr int bytes = w_scales + wt * 64;
  static constexpr int stages_fit = kMxLdsBudget / bytes;
  static constexpr int stages = stages_fit < 6 ? stages_fit : 6;
  // direct loads per stage: one per code tile; one dword load per 4-tile scale group
  static constexpr int code_loads = at + wt;
  static constexpr int scale_loads = (at + wt) / 4;
  static_assert(wt % 4 == 0 && at % 4 == 0, "scale groups of 4 tiles");
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

// Workgroup tiles of one geometry: tiles_m x tiles_n tiles over the output
// columns from n_off on.
struct MxPanels {
  int64_t tiles_m, tiles_n, n_off;
};

// Workgroup tile blk (0 .. P.tiles_m * P.tiles_n - 1) of geometry Gm.
template <class Gm, int OUT>
__device__ __forceinline__ void mx_gemm_tile(int64_t blk, const MxPanels& P, const uint8_t* __restrict__ a_codes,
                                             const uint8_t* __restrict__ a_scales,
                                             const uint8_t* __restrict__ w_codes,
                                             const uint8_t* __restrict__ w_scales, int64_t M, int64_t N,
                                             int64_t a_tiles_r, int64_t w_tiles_r, int64_t KT, void* __restrict__ Y) {
  const int64_t tiles_m = P.tiles_m, tiles_n = P.tiles_n, n_off = P.n_off;
  constexpr int S = Gm::stages;
  constexpr int TM = Gm::tm, TN = Gm::tn;
  constexpr int L = Gm::loads_per_wave;
  extern __shared__ __align__(16) uint8_t smem[];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int64_t bm, bn;
  gemm_tile_of(blk, tiles_m, tiles_n, bm, bn);
  const int wm = wave % Gm::wm, wn = wave / Gm::wm;
  const int64_t a_tr0 = bm * Gm::at, w_tr0 = n_off / 32 + bn * Gm::wt;
  const int64_t m0 = bm * Gm::bm + wm * 32 * TM;
  const int64_t n0 = n_off + bn * Gm::bn + wn * 32 * TN;
  const int KTi = (int)KT;

  // Direct loads: wavefront w loads code tiles w*CPW + u (A tiles first,
  // then W, contiguous in LDS) with one M0 and the LDS placement in the
  // instruction offset (which the hardware adds to both addresses; the lane
  // offsets subtract it back out); scale instruction `wave` covers one 4-tile
  // group (256 bytes), waves past the last group repeating it.  Each operand
  // row panel is one buffer resource (per load a fixed lane offset, per K
  // step one scalar offset), based kBias bytes low so that the lane offsets
  // stay non-negative.  Tiles past the end of an operand read its last row
  // tile (in bounds): they only feed output rows / columns that are never
  // stored.  K steps past the end reload the last one into a slot that is no
  // longer read, so that every step issues the same loads (no branches in
  // the main loop).
  const int chunk = 2 * (lane & 31) + (lane >> 5);
  constexpr int CPW = Gm::code_loads / Gm::waves;
  constexpr int kBias = 4096;
  static_assert(CPW * 1024 <= kBias, "instruction offsets within the bias");
  auto rsrc = [](const uint8_t* base, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base) - kBias, 0, (int)(bytes + kBias), 0x00020000);
  };
  const __amdgpu_buffer_rsrc_t rac = rsrc(a_codes + a_tr0 * KT * 1024, (int64_t)Gm::at * KT * 1024);
  const __amdgpu_buffer_rsrc_t rwc = rsrc(w_codes + w_tr0 * KT * 1024, (int64_t)Gm::wt * KT * 1024);
  const __amdgpu_buffer_rsrc_t ras = rsrc(a_scales + (a_tr0 / 4) * KT * 256, (int64_t)(Gm::at / 4) * KT * 256);
  const __amdgpu_buffer_rsrc_t rws = rsrc(w_scales + (w_tr0 / 4) * KT * 256, (int64_t)(Gm::wt / 4) * KT * 256);
  uint32_t c_off[CPW];
  bool c_a[CPW];
#pragma unroll
  for (int u = 0; u < CPW; ++u) {
    const int t = wave * CPW + u;
    const bool is_a = t < Gm::at;
    const int b = is_a ? t : t - Gm::at;
    const int64_t tr0 = is_a ? a_tr0 : w_tr0;
    const int64_t tr = min(tr0 + b, (is_a ? a_tiles_r : w_tiles_r) - 1) - tr0;
    c_a[u] = is_a;
    c_off[u] = (uint32_t)(tr * KT * 1024 + chunk * 16 + kBias - u * 1024);
  }
  const int c_m0 = wave * CPW * 1024;
  const int si = min(wave, Gm::scale_loads - 1);   // waves past the last scale group repeat it
  const bool s_is_a = si < Gm::at / 4;
  const int64_t a_groups = (a_tiles_r + 3) / 4, w_groups = (w_tiles_r + 3) / 4;
  const int64_t g0 = (s_is_a ? a_tr0 : w_tr0) / 4;
  const int64_t sg = min(g0 + (s_is_a ? si : si - Gm::at / 4), (s_is_a ? a_groups : w_groups) - 1) - g0;
  const uint32_t s_off = (uint32_t)(sg * KT * 256 + lane * 4 + kBias);
  const int s_dst = Gm::a_scales + si * 256;
  // stage kt into the ring slot at byte offset `off` (kt past the end: the last one again)
  // load r (0 .. L-1) of stage kt into the ring slot at byte offset `off`
  auto issue_one = [&](int kt, int off, auto rc) {
    constexpr int r = decltype(rc)::value;
    uint8_t* stage = smem + off;
    const int ktc = kt < KTi ? kt : KTi - 1;
    if constexpr (r < CPW) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(c_a[r] ? rac : rwc,
                                               (__attribute__((address_space(3))) void*)(stage + c_m0), 16,
                                               c_off[r], ktc * 1024, r * 1024, 0);
    } else {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(s_is_a ? ras : rws,
                                               (__attribute__((address_space(3))) void*)(stage + s_dst), 4, s_off,
                                               ktc * 256, 0, 0);
    }
  };
  auto issue = [&](int kt, int off) {
    uint8_t* stage = smem + off;
    const int ktc = kt < KTi ? kt : KTi - 1;
    static_for<0, CPW>([&](auto ic) {
      constexpr int u = decltype(ic)::value;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(c_a[u] ? rac : rwc,
                                               (__attribute__((address_space(3))) void*)(stage + c_m0), 16,
                                               c_off[u], ktc * 1024, u * 1024, 0);
    });
    __builtin_amdgcn_raw_ptr_buffer_load_lds(s_is_a ? ras : rws,
                                             (__attribute__((address_space(3))) void*)(stage + s_dst), 4, s_off,
                                             ktc * 256, 0, 0);
  };

  float16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = float16_t{};

  // Operands of one K step: code tiles, and the scale bytes of the
  // wavefront's A tiles (byte i = tile i) and W tiles (byte j = tile j) in
  // one dword each.
  struct Ops {
    uint4_t a[TM], w[TN];
    uint32_t sa, sw;
  };
  static_assert(TM == 4 && (TN == 4 || TN == 2), "scale dwords hold 4 tiles");
  const int a_rd = Gm::a_codes + wm * TM * 1024 + lane * 16;
  const int w_rd = Gm::w_codes + wn * TN * 1024 + lane * 16;
  const int as_rd = Gm::a_scales + wm * 256 + lane * 4;
  const int ws_rd = Gm::w_scales + (wn * TN / 4) * 256 + lane * 4;
  const int ws_shift = 8 * ((wn * TN) % 4);
  // read r (0 .. TM+TN+1) of a step's operands
  auto read_one = [&](const uint8_t* stg, Ops& o, int r) {
    if (r < TM) o.a[r] = *reinterpret_cast<const uint4_t*>(stg + a_rd + r * 1024);
    else if (r < TM + TN) o.w[r - TM] = *reinterpret_cast<const uint4_t*>(stg + w_rd + (r - TM) * 1024);
    else if (r == TM + TN) o.sa = *reinterpret_cast<const uint32_t*>(stg + as_rd);
    else o.sw = *reinterpret_cast<const uint32_t*>(stg + ws_rd) >> ws_shift;
  };
  constexpr int kReads = TM + TN + 2;
  auto mfma_one = [&](const Ops& o, int q) {
    const int i = q / TN, j = q % TN;
    const int8v_t av = {(int)o.a[i][0], (int)o.a[i][1], (int)o.a[i][2], (int)o.a[i][3], 0, 0, 0, 0};
    const int8v_t wv = {(int)o.w[j][0], (int)o.w[j][1], (int)o.w[j][2], (int)o.w[j][3], 0, 0, 0, 0};
    // W as the first operand: the accumulator block is the transposed output
    // tile, so each lane ends up with 4 consecutive output columns.  E2M1 is
    // format 4 for both operands; op_sel picks the tile's scale byte.
    switch (i * 4 + j) {
#define DQ_MX_MFMA(I, J)                                                                                     \
  case I * 4 + J:                                                                                            \
    if constexpr (J < TN)                                                                                    \
      acc[I][J] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(wv, av, acc[I][J], 4, 4, J, (int)o.sw, I,    \
                                                                 (int)o.sa);                                 \
    break;
      DQ_MX_MFMA(0, 0) DQ_MX_MFMA(0, 1) DQ_MX_MFMA(0, 2) DQ_MX_MFMA(0, 3)
      DQ_MX_MFMA(1, 0) DQ_MX_MFMA(1, 1) DQ_MX_MFMA(1, 2) DQ_MX_MFMA(1, 3)
      DQ_MX_MFMA(2, 0) DQ_MX_MFMA(2, 1) DQ_MX_MFMA(2, 2) DQ_MX_MFMA(2, 3)
      DQ_MX_MFMA(3, 0) DQ_MX_MFMA(3, 1) DQ_MX_MFMA(3, 2) DQ_MX_MFMA(3, 3)
#undef DQ_MX_MFMA
      default: break;
    }
  };
  constexpr int kMfmas = TM * TN;
  constexpr int kSlots = kMfmas > kReads + 3 ? kMfmas : kReads + 3;
  static_assert(3 + L <= kSlots, "every refill load has a slot in the step");

  if (KTi > 0) {
    // prologue: stages 0 .. S-1 in flight, stage 0 landed everywhere
#pragma unroll
    for (int st = 0; st < S; ++st) issue(st, st * Gm::bytes);
    mx_wait_vm<(S - 1) * L>();
    mx_barrier();
    Ops o0, o1;
    // One step (cur = stage kt's operands, read during the previous step):
    // two MFMAs are issued before the wait for stage kt+1 and the barrier so
    // that the matrix cores stay busy through them; after the barrier the
    // slot of stage kt (read by everyone) is refilled with stage kt+S, one
    // load after each MFMA (issued in a burst they held back the MFMAs that
    // followed), and the reads of stage kt+1 are interleaved with the
    // remaining MFMAs.  The
    // sched_barriers keep this order; the empty asm statements pin the
    // accumulators at the end of the step (otherwise the compiler sinks the
    // MFMAs, pure register operations, into the next step).
    // off: byte offset of stage kt's ring slot (refilled with stage kt+S),
    // noff: that of stage kt+1
    auto step = [&](int kt, Ops& cur, Ops& nxt, int off, int noff) {
      __builtin_amdgcn_s_waitcnt((0x3F & 0xF) | (0x7 << 4) | (0x0 << 8) | ((0x3F >> 4) << 14));   // lgkmcnt(0)
      mfma_one(cur, 0);
      mfma_one(cur, 1);
      __builtin_amdgcn_sched_barrier(0);
      mx_wait_vm<(S - 2) * L>();
      mx_barrier();
      mfma_one(cur, 2);
      __builtin_amdgcn_sched_barrier(0);
      const uint8_t* stg = smem + noff;
#pragma unroll
      for (int q = 3; q < kSlots; ++q) {
        __builtin_amdgcn_sched_barrier(0);
        static_for<0, L>([&](auto rc) {
          if (q == 3 + decltype(rc)::value) issue_one(kt + S, off, rc);
        });
        if (q - 3 < kReads) read_one(stg, nxt, q - 3);
        __builtin_amdgcn_sched_barrier(0);
        if (q < kMfmas) mfma_one(cur, q);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) asm volatile("" : "+a"(acc[i][j]));
    };
    // Full steps 0 .. KT-2 alternate o0 -> o1 and o1 -> o0; the first one is
    // peeled when their number is odd, so that the last step always consumes o0.
    const int full = KTi - 1;
    int kt = 0, off = 0, noff = Gm::bytes;
    auto adv = [&](int o) { return o + Gm::bytes == S * Gm::bytes ? 0 : o + Gm::bytes; };
    if (full & 1) {
#pragma unroll
      for (int r = 0; r < kReads; ++r) read_one(smem, o1, r);
      step(0, o1, o0, off, noff);
      kt = 1;
      off = noff;
      noff = adv(noff);
    } else {
#pragma unroll
      for (int r = 0; r < kReads; ++r) read_one(smem, o0, r);
    }
    for (; kt < full; kt += 2) {
      step(kt, o0, o1, off, noff);
      off = noff;
      noff = adv(noff);
      step(kt + 1, o1, o0, off, noff);
      off = noff;
      noff = adv(noff);
    }
    __builtin_amdgcn_s_waitcnt((0x3F & 0xF) | (0x7 << 4) | (0x0 << 8) | ((0x3F >> 4) << 14));   // lgkmcnt(0)
#pragma unroll
    for (int q = 0; q < kMfmas; ++q) mfma_one(o0, q);
    // drain the redundant reloads of the last steps before the workgroup ends
    mx_wait_vm<0>();
  }

  // Block (i, j) holds, in lane l, output row m0 + 32i + l%32 and columns
  // n0 + 32j + 8g + 4(l/32) + t in register 4g + t (g, t = 0..3): four
  // consecutive columns.
  //
  // bf16 output of a wavefront tile inside Y (N % 8 == 0): each 32-row block
  // goes through LDS (8-byte writes in the accumulator layout, 16-byte reads
  // along the rows) so that every store instruction writes whole 128-byte
  // lines; written straight from the accumulators, each instruction touches
  // 32 lines with 16 bytes each and the stores of a tile (issued by all
  // workgroups at about the same time) took ~7 % of the kernel at M = 32768.
  // The LDS ring is free once every wavefront has drained its loads.
  if constexpr (OUT == 1) {
    __syncthreads();
    constexpr int RS = 64 * TN + 16;                  // LDS bytes per staged row (pad staggers banks)
    constexpr int LPR = 4 * TN;                       // lanes per row in the read-back (16 bytes each)
    if (m0 + 32 * TM <= M && n0 + 32 * TN <= N && (N & 7) == 0) {
      uint8_t* ep = smem + (size_t)wave * 32 * RS;
      const int rl = lane & 31, h = lane >> 5;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const uint32_t b0 = f32_to_bf16_rne(acc[i][j][4 * g]), b1 = f32_to_bf16_rne(acc[i][j][4 * g + 1]);
            const uint32_t b2 = f32_to_bf16_rne(acc[i][j][4 * g + 2]), b3 = f32_to_bf16_rne(acc[i][j][4 * g + 3]);
            *reinterpret_cast<uint2_t*>(ep + rl * RS + (32 * j + 8 * g + 4 * h) * 2) =
                uint2_t{b0 | (b1 << 16), b2 | (b3 << 16)};
          }
#pragma unroll
        for (int r0 = 0; r0 < 32; r0 += 64 / LPR) {
          const int rr = r0 + lane / LPR, seg = lane % LPR;
          const uint4_t v = *reinterpret_cast<const uint4_t*>(ep + rr * RS + seg * 16);
          *reinterpret_cast<uint4_t*>(reinterpret_cast<uint16_t*>(Y) + (m0 + 32 * i + rr) * N + n0 + seg * 8) = v;
        }
      }
      return;
    }
  }
  const bool vec = (N & 3) == 0;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int64_t row = m0 + i * 32 + (lane & 31);
    if (row >= M) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t col = n0 + j * 32 + g * 8 + 4 * (lane >> 5);
        const float v0 = acc[i][j][4 * g], v1 = acc[i][j][4 * g + 1], v2 = acc[i][j][4 * g + 2],
                    v3 = acc[i][j][4 * g + 3];
        if (OUT == 0) {
          float* y = reinterpret_cast<float*>(Y) + row * N + col;
          if (vec && col + 3 < N) {
            *reinterpret_cast<float4_t*>(y) = float4_t{v0, v1, v2, v3};
          } else {
            if (col < N) y[0] = v0;
            if (col + 1 < N) y[1] = v1;
            if (col + 2 < N) y[2] = v2;
            if (col + 3 < N) y[3] = v3;
          }
        } else {
          const uint32_t b0 = f32_to_bf16_rne(v0), b1 = f32_to_bf16_rne(v1), b2 = f32_to_bf16_rne(v2),
                         b3 = f32_to_bf16_rne(v3);
          uint16_t* y = reinterpret_cast<uint16_t*>(Y) + row * N + col;
          if (vec && col + 3 < N) {
            *reinterpret_cast<uint2_t*>(y) = uint2_t{b0 | (b1 << 16), b2 | (b3 << 16)};
          } else {
            if (col < N) y[0] = (uint16_t)b0;
            if (col + 1 < N) y[1] = (uint16_t)b1;
            if (col + 2 < N) y[2] = (uint16_t)b2;
            if (col + 3 < N) y[3] = (uint16_t)b3;
          }
        }
      }
    }
  }
}

// One launch, two geometries: workgroups 0 .. full tiles - 1 take the tiles
// of Gf (columns 0 .. split - 1), the rest those of Gh (columns split ..).
template <class Gf, class Gh, int OUT>
__global__ __launch_bounds__(Gf::threads, 1) void mxfp4_gemm_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales, const uint8_t* __restrict__ w_codes,
    const uint8_t* __restrict__ w_scales, int64_t M, int64_t N, int64_t a_tiles_r, int64_t w_tiles_r, int64_t KT,
    void* __restrict__ Y, MxPanels full, MxPanels half) {
  static_assert(Gf::threads == Gh::threads, "one launch shape");
  const int64_t nf = full.tiles_m * full.tiles_n;
  const int64_t b = blockIdx.x;
  if (b < nf)
    mx_gemm_tile<Gf, OUT>(b, full, a_codes, a_scales, w_codes, w_scales, M, N, a_tiles_r, w_tiles_r, KT, Y);
  else
    mx_gemm_tile<Gh, OUT>(b - nf, half, a_codes, a_scales, w_codes, w_scales, M, N, a_tiles_r, w_tiles_r, KT, Y);
}

// Output columns 0 .. split-1 in Gf tiles, split .. N-1 in Gh tiles (split a
// multiple of Gf::bn, or N), one launch.
template <class Gf, class Gh>
hipError_t launch_mx_geo(const MxGemmArgs& a, int64_t split, hipStream_t s) {
  const int64_t a_tiles_r = round_up(a.M, 32) / 32;
  const int64_t w_tiles_r = round_up(a.N, 32) / 32;
  const int64_t KT = round_up(a.K, 64) / 64;
  // the loaders address one workgroup's row panel of an operand with 32-bit
  // buffer offsets (at most 8 code tiles of KT KiB, plus the bias)
  if ((int64_t)std::max(std::max(Gf::at, Gf::wt), std::max(Gh::at, Gh::wt)) * KT * 1024 + 4096 > INT32_MAX)
    return hipErrorNotSupported;
  const MxPanels full{(a.M + Gf::bm - 1) / Gf::bm, (split + Gf::bn - 1) / Gf::bn, 0};
  const MxPanels half{split < a.N ? (a.M + Gh::bm - 1) / Gh::bm : 0, (a.N - split + Gh::bn - 1) / Gh::bn, split};
  const int64_t blocks = full.tiles_m * full.tiles_n + half.tiles_m * half.tiles_n;
  const size_t lds = std::max((size_t)Gf::stages * Gf::bytes, (size_t)Gh::stages * Gh::bytes);
  typedef void (*kern_t)(const uint8_t*, const uint8_t*, const uint8_t*, const uint8_t*, int64_t, int64_t, int64_t,
                         int64_t, int64_t, void*, MxPanels, MxPanels);
  const kern_t kern = a.out_kind == 0 ? mxfp4_gemm_kernel<Gf, Gh, 0> : mxfp4_gemm_kernel<Gf, Gh, 1>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(Gf::threads), lds, s, a.A.codes, a.A.scales, a.W.codes,
                     a.W.scales, a.M, a.N, a_tiles_r, w_tiles_r, KT, a.Y, full, half);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_mx_quantize(const void* x, bool is_bf16, int64_t rows, int64_t cols, const MxView& out,
                              hipStream_t s) {
  const int64_t tiles_r = round_up(rows, 32) / 32, tiles_c = round_up(cols, 64) / 64;
  const int64_t groups = (tiles_r + 3) / 4 * tiles_c;
  if (groups == 0) return hipSuccess;
  const unsigned grid = (unsigned)groups;
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
  // 256x256 workgroup tiles (four wavefronts of 128x128, one per SIMD); one
  // workgroup fills a compute unit, so a last round that would leave compute
  // units idle runs instead as 256x128 tiles over the remaining column
  // panels, in the same launch.
  using Full = MxGeo<4, 4, 2, 2>;
  using Half = MxGeo<4, 2, 2, 2>;
  const int64_t n_split = gemm_column_split(a.M, a.N, Full::bm, Full::bn, Full::bm, Half::bn, num_cus(), kHalfRound);
  return launch_mx_geo<Full, Half>(a, n_split, s);
}

}  // namespace dq
