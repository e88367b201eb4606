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
// Structure
//  * a workgroup of WM x WN wavefronts covers a (32*TM*WM) x (32*TN*WN)
//    output tile; each wavefront owns 32*TM x 32*TN (TM x TN accumulator
//    blocks of 32x32).  The default is four wavefronts of 128 x 128 on a
//    256 x 256 tile, one wavefront per SIMD: each operand tile is dequantized
//    by two wavefronts (not four), and 64 MFMAs per K step give the
//    dequantization of the next sub-step room to run between them;
//  * operands stay compressed (4.5 bits/element) until they reach registers:
//    a ring of LDS stages, each holding the raw code and scale tiles of KS
//    64-column K steps, is filled by direct global->LDS loads
//    (global_load_lds_dwordx4 / _dword) stages-1 ahead, so the HBM and L2
//    latency is hidden without spending VGPRs on prefetch; one workgroup
//    barrier per stage;
//  * within a stage, a 32x64 code tile is one contiguous KiB; the loading
//    lane i fetches 16-byte chunk 2*(i%32) + i/32 so that the consuming lane
//    l (row l%32, columns 32*(l/32)..+31) reads LDS bytes 16l..16l+15
//    (conflict-free ds_read_b128);
//  * MFMA sub-step s of a K step consumes columns 32*(l/32) + 8s .. +7 on both
//    operands (a permutation of K shared by A and W);
//  * workgroups are numbered so that the 8 XCDs each own a contiguous range
//    of output-column panels (W panels stay in one XCD's L2).
#include <type_traits>

#include "dq_device.hpp"
#include "dq_internal.hpp"

namespace dq {

namespace {

constexpr int kLdsBudget = 150 * 1024;   // of gfx950's 160 KiB

// Workgroup geometry: WM x WN wavefronts, each owning 32*TM rows x 32*TN
// columns; KS 64-column K steps per LDS stage.
template <int TM, int TN, int WM, int WN, int KS>
struct Geo {
  static constexpr int tm = TM, tn = TN, wm = WM, wn = WN;
  static constexpr int waves = WM * WN;
  static constexpr int threads = 64 * waves;
  static constexpr int bm = 32 * TM * WM;      // workgroup tile rows
  static constexpr int bn = 32 * TN * WN;      // workgroup tile columns
  static constexpr int at = bm / 32;           // A code tiles per K step
  static constexpr int wt = bn / 32;           // W code tiles per K step
  static constexpr int ks = KS;                // 64-column K steps per stage (one barrier each)
  // LDS byte layout of one stage, per K step u: A codes, W codes, A scales, W scales
  static constexpr int step_bytes = at * 1024 + wt * 1024 + at * 128 + wt * 128;
  static constexpr int a_codes = 0;
  static constexpr int w_codes = at * 1024;
  static constexpr int a_scales = w_codes + wt * 1024;
  static constexpr int w_scales = a_scales + at * 128;
  static constexpr int bytes = KS * step_bytes;
  // fp16 copy of the workgroup's A tiles for one K step (dequantized once,
  // read by every wavefront of the row); double-buffered after the ring
  static constexpr int a16_tile = 32 * 64 * 2;
  static constexpr int a16_bytes = at * a16_tile;
  static constexpr int stages_fit = (kLdsBudget - 2 * a16_bytes) / bytes;
  static constexpr int stages = stages_fit < 4 ? stages_fit : 4;   // ring depth
  static constexpr int a16_base = stages * bytes;
  // direct-to-LDS instructions per K step: one per code tile, one per pair of scale tiles
  static constexpr int code_loads = at + wt;
  static constexpr int scale_loads = (at + wt) / 2;
  static_assert(at % 2 == 0 && wt % 2 == 0, "scale tiles are loaded in pairs");
  static_assert(stages >= 3, "LDS ring needs three stages");
  static_assert(waves == at, "each wavefront dequantizes one A tile per K step");
  static_assert(wt <= waves && (at + wt) / 2 <= waves, "at most one W tile and one scale pair per wavefront");
  static_assert(KS == 1, "one K step per stage");
};

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

// Number of direct-to-LDS load instructions wavefront `wave` issues per stage
// (code tiles round-robin over the wavefronts, then scale instructions).
template <class Gm>
__host__ __device__ constexpr int loads_per_stage(int wave) {
  return Gm::ks * ((Gm::code_loads - wave + Gm::waves - 1) / Gm::waves +
                   (Gm::scale_loads - wave + Gm::waves - 1) / Gm::waves);
}

// Issue the direct-to-LDS loads of one K step into `stage`.  Code tiles are
// distributed round-robin over the wavefronts; scale tiles are 128 bytes and
// one dword instruction covers two of them (lanes 0..31, 32..63).  Tiles past
// the end of an operand read a clamped, in-bounds address so that every
// wavefront issues a fixed number of loads (the data is zeroed on use).
template <class Gm>
__device__ inline void issue_stage(uint8_t* stage, const uint8_t* __restrict__ a_codes,
                                   const uint8_t* __restrict__ a_scales, const uint8_t* __restrict__ w_codes,
                                   const uint8_t* __restrict__ w_scales, int64_t a_tr0, int64_t a_tiles_r,
                                   int64_t w_tr0, int64_t w_tiles_r, int64_t kt, int64_t KT, int wave, int lane) {
  const int chunk = 2 * (lane & 31) + (lane >> 5);      // global 16-byte chunk fetched by this lane
  for (int u = 0; u < Gm::ks; ++u, ++kt, stage += Gm::step_bytes) {
  const int64_t ktc = kt < KT ? kt : KT - 1;             // past the end of K: reload the last step
  for (int t = wave; t < Gm::code_loads; t += Gm::waves) {
    const bool is_a = t < Gm::at;
    const int b = is_a ? t : t - Gm::at;
    const int64_t lim = is_a ? a_tiles_r : w_tiles_r;
    int64_t tr = (is_a ? a_tr0 : w_tr0) + b;
    tr = tr < lim ? tr : lim - 1;
    const uint8_t* src = (is_a ? a_codes : w_codes) + (tr * KT + ktc) * 1024 + chunk * 16;
    uint8_t* dst = stage + (is_a ? Gm::a_codes : Gm::w_codes) + b * 1024;
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(src), reinterpret_cast<void*>(dst), 16, 0, 0);
  }
  for (int t = wave; t < Gm::scale_loads; t += Gm::waves) {
    const bool is_a = t < Gm::at / 2;
    const int b = 2 * (is_a ? t : t - Gm::at / 2) + (lane >> 5);
    const int64_t lim = is_a ? a_tiles_r : w_tiles_r;
    int64_t tr = (is_a ? a_tr0 : w_tr0) + b;
    tr = tr < lim ? tr : lim - 1;
    const uint8_t* src = (is_a ? a_scales : w_scales) + (tr * KT + ktc) * 128 + (lane & 31) * 4;
    uint8_t* dst = stage + (is_a ? Gm::a_scales : Gm::w_scales) + (b & ~1) * 128;
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(src), reinterpret_cast<void*>(dst), 4, 0, 0);
  }
  }
}

// s_waitcnt vmcnt(n) (n < 64) with expcnt / lgkmcnt left at their maximum.
// gfx9 encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at [15:14].
template <int n>
__device__ inline void wait_vm() {
  __builtin_amdgcn_s_waitcnt((n & 0xF) | (0x7 << 4) | (0xF << 8) | ((n >> 4) << 14));
}

// Workgroup barrier without the release/acquire fences of __syncthreads (which
// would also wait for every outstanding prefetch); the empty asm statements
// keep the compiler from moving LDS accesses across it.
__device__ inline void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Output side of the GEMM: the plain result (fp32 / bf16, [M, Nout]) or its
// NVFP4 requantization (the next layer's input) in the tiled layout of dq.h.
struct GemmOut {
  void* Y;                 // OUT_F32 / OUT_BF16
  const float* G_out;      // OUT_NVFP4: static scale of the next layer's input
  uint8_t* codes;          // OUT_NVFP4
  uint8_t* scales;
  float* G;                // receives *G_out (may alias it)
  int64_t Nout;            // N, or N / 2 with SwiGLU
  int64_t tiles_r, tiles_c;   // NVFP4 tiles of [M, Nout]
};

enum { kOutF32 = 0, kOutBF16 = 1, kOutNvfp4 = 2 };

// silu(g) * u in fp32 (SwiGLU, the MLP non-linearity between gate/up and down)
__device__ inline float swiglu(float g, float u) { return g / (1.0f + expf(-g)) * u; }

// One E2M1 code (low nibble) of v for the block scale S != 0: the same
// arithmetic as the activation quantizer (correctly rounded v / S, hardware
// round-to-nearest-even with saturation, +0 for magnitude zero).
__device__ inline uint32_t e2m1_code(float v, float S) {
  const float rcp = 1.0f / S;
  return fp4_canonical_zero(cvt_pk_fp4<0>(0u, div_by_scale(v, S, rcp), 0.0f)) & 0xFu;
}

template <class Gm, int OUT, bool SW>
__global__ __launch_bounds__(Gm::threads, 1) void nvfp4_gemm_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales, const float* __restrict__ Ga,
    const uint8_t* __restrict__ w_codes, const uint8_t* __restrict__ w_scales, const float* __restrict__ Gw,
    int64_t M, int64_t N, int64_t a_tiles_r, int64_t w_tiles_r, int64_t KT, GemmOut out,
    int64_t tiles_m, int64_t tiles_n, int64_t n_off) {
  constexpr int kStages = Gm::stages;
  constexpr int TM = Gm::tm, TN = Gm::tn, KS = Gm::ks;
  extern __shared__ __align__(16) uint8_t smem[];

  const int lane = threadIdx.x & 63;
  // wavefront index as a uniform (scalar) value: the LDS destination of the
  // direct loads lives in M0 and must not look divergent to the compiler
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // XCD-aware numbering: workgroup b runs on XCD b % 8; give each XCD a
  // contiguous range of tiles, ordered column-panel-major.
  const int64_t nb = tiles_m * tiles_n;
  int64_t logical = blockIdx.x;
  if (nb % 8 == 0) logical = (int64_t)(blockIdx.x % 8) * (nb / 8) + blockIdx.x / 8;
  const int64_t bm = logical % tiles_m, bn = logical / tiles_m;
  const int wm = wave % Gm::wm, wn = wave / Gm::wm;
  // this launch covers tiles_n column panels from output column n_off on
  const int64_t a_tr0 = bm * Gm::at, w_tr0 = n_off / 32 + bn * Gm::wt;
  const int64_t m0 = bm * Gm::bm + wm * 32 * TM;
  const int64_t n0 = n_off + bn * Gm::bn + wn * 32 * TN;

  float16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = float16_t{};

  constexpr int S = kStages;
  const int KTi = (int)KT;
  // Direct loads of one stage (= K step): this wavefront fetches A code tile
  // `wave`, W code tile `wave` (if there is one) and one pair of scale tiles
  // (A pairs first, then W pairs, one per wavefront while they last).  Rows
  // past the end of an operand read the last row tile (in bounds; zeroed on
  // use).
  const int chunk = 2 * (lane & 31) + (lane >> 5);      // 16-byte chunk of the tile fetched by this lane
  const uint8_t* a_src = a_codes + (min(a_tr0 + wave, a_tiles_r - 1) * KT) * 1024 + chunk * 16;
  const bool has_w = wave < Gm::wt;
  const uint8_t* w_src = w_codes + (min(w_tr0 + (has_w ? wave : 0), w_tiles_r - 1) * KT) * 1024 + chunk * 16;
  constexpr int a_pairs = Gm::at / 2, pairs = (Gm::at + Gm::wt) / 2;
  const bool has_s = wave < pairs;
  const bool s_is_a = wave < a_pairs;
  const int s_pair = !has_s ? 0 : s_is_a ? wave : wave - a_pairs;
  const int64_t s_tr = min((s_is_a ? a_tr0 : w_tr0) + 2 * s_pair + (lane >> 5), (s_is_a ? a_tiles_r : w_tiles_r) - 1);
  const uint8_t* s_src = (s_is_a ? a_scales : w_scales) + (s_tr * KT) * 128 + (lane & 31) * 4;
  const int s_dst = (s_is_a ? Gm::a_scales : Gm::w_scales) + 2 * s_pair * 128;
  auto issue = [&](int kt) {
    uint8_t* stage = smem + (kt % S) * Gm::bytes;
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(a_src + (size_t)kt * 1024),
                                     reinterpret_cast<void*>(stage + Gm::a_codes + wave * 1024), 16, 0, 0);
    if (has_w)
      __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(w_src + (size_t)kt * 1024),
                                       reinterpret_cast<void*>(stage + Gm::w_codes + wave * 1024), 16, 0, 0);
    if (has_s)
      __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(s_src + (size_t)kt * 128),
                                       reinterpret_cast<void*>(stage + s_dst), 4, 0, 0);
  };
  // direct loads of this wavefront per stage (3 for every wavefront when
  // there are as many W tiles and scale pairs as wavefronts)
  constexpr bool kUniformL = Gm::wt == Gm::waves && pairs == Gm::waves;
  const int L = 1 + (has_w ? 1 : 0) + (has_s ? 1 : 0);
  // prologue: stages (= K steps) 0 .. S-1
#pragma unroll
  for (int st = 0; st < S; ++st)
    if (st < KTi) issue(st);
  // this wavefront's loads of stage `need` have landed, given stages up to
  // `last` issued (the later ones, at most S - 2, may stay in flight)
  auto wait_stage = [&](int need, int last) {
    const int ahead = max(0, min(last, KTi - 1) - need);
    if constexpr (kUniformL) {
      if (ahead >= 2) wait_vm<6>();
      else if (ahead == 1) wait_vm<3>();
      else wait_vm<0>();
    } else {
      switch (ahead * L) {   // loads allowed to stay in flight: 0 .. 2 L, L <= 3
        case 0: wait_vm<0>(); break;
        case 1: wait_vm<1>(); break;
        case 2: wait_vm<2>(); break;
        case 3: wait_vm<3>(); break;
        case 4: wait_vm<4>(); break;
        default: wait_vm<6>(); break;
      }
    }
  };
  static_assert(S - 2 <= 2, "wait_stage covers at most two stages in flight");

  // rows / columns of this wavefront that exist (zero inputs elsewhere)
  bool w_ok[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) w_ok[j] = (n0 / 32 + j) < w_tiles_r;
  const int lane_scale = (lane & 31) * 4 + (lane >> 5) * 2;
  const int row = lane & 31, half = lane >> 5;
  // Swizzle of the fp16 A tiles: 16-byte chunk c of row r is stored at chunk
  // c ^ g(r), g(r) = (r % 8) ^ (r / 8 % 2), so that any 8 or 16 consecutive
  // lanes of the producer's writes and of the MFMA operand reads touch
  // distinct banks (for 32 or 64 four-byte banks).
  const int gsw = (row & 7) ^ ((row >> 3) & 1);
  int a_rd[4], a_wr[4];   // per-lane byte offsets of the read / written chunks
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    a_rd[k] = Gm::a16_base + wm * TM * Gm::a16_tile + row * 128 + (((4 * half + k) ^ gsw) * 16);
    a_wr[k] = Gm::a16_base + wave * Gm::a16_tile + row * 128 + (((4 * half + k) ^ gsw) * 16);
  }
  const int w_rd = Gm::w_codes + wn * TN * 1024 + lane * 16;
  const int ws_rd = Gm::w_scales + wn * TN * 128 + lane_scale;
  const int a_prd = Gm::a_codes + wave * 1024 + lane * 16;
  const int as_prd = Gm::a_scales + wave * 128 + lane_scale;

  // Producer: A tile `wave` of K step kt, dequantized to fp16 into buffer BUF
  // (the raw tile is read first, so that the reads of a step can be issued
  // together).
  const bool p_ok = (a_tr0 + wave) < a_tiles_r;
  struct Raw {
    uint4_t c;
    uint32_t sc;
  };
  auto produce_read = [&](int kt) -> Raw {
    const uint8_t* stg = smem + (kt % S) * Gm::bytes;
    Raw r;
    r.c = *reinterpret_cast<const uint4_t*>(stg + a_prd);
    r.sc = *reinterpret_cast<const uint16_t*>(stg + as_prd);
    return r;
  };
  auto produce_write = [&](const Raw& r, auto buf) {
    half2_t s_lo, s_hi;
    scale_pairs(p_ok ? r.sc : 0u, s_lo, s_hi);   // a zero scale zeroes the (finite) codes of a missing tile
#pragma unroll
    for (int k = 0; k < 4; ++k)
      *reinterpret_cast<half8_t*>(smem + a_wr[k] + decltype(buf)::value * Gm::a16_bytes) =
          dequant8(r.c[k], k < 2 ? s_lo : s_hi);
  };
  auto lgkm0 = [] {
    __builtin_amdgcn_s_waitcnt((0x3F & 0xF) | (0x7 << 4) | (0x0 << 8) | ((0x3F >> 4) << 14));   // lgkmcnt(0)
  };
  // MFMA operands of two sub-steps (double buffer): sub-step s of a K step
  // uses slot s % 2.  The MFMAs of a step's last sub-step are deferred past the
  // step's barrier: their operands are already in registers, so they keep the
  // matrix cores busy while the next step's first LDS reads are in flight.
  half8_t af[2][TM], wf[2][TN];
  auto mfmas = [&](int slot) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[slot][i], wf[slot][j], acc[i][j], 0, 0, 0);
  };
  // One K step on A buffer BUF: read this step's operands and the next
  // step's raw A tile, finish the previous step (deferred MFMAs), produce the
  // next step's A into the other buffer, run sub-steps 0..2 (sub-step s+1's
  // operands are prepared while sub-step s's MFMAs run) and leave sub-step 3
  // pending; then the step's barrier (A of step kt+1 written, stage kt+2
  // landed, stage kt's slot and buffer BUF free) and the refill of stage kt's
  // slot.
  auto step = [&](int kt, auto buf, auto deferred) {
    using other = std::integral_constant<int, 1 - decltype(buf)::value>;
    const bool more = kt + 1 < KTi;
    Raw raw{};
    if (more) raw = produce_read(kt + 1);
    const uint8_t* stg = smem + (kt % S) * Gm::bytes;
    uint4_t wc[TN];
    uint32_t wsc[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      wc[j] = *reinterpret_cast<const uint4_t*>(stg + w_rd + j * 1024);
      wsc[j] = *reinterpret_cast<const uint16_t*>(stg + ws_rd + j * 128);
    }
    auto a_frag = [&](int i, int s) -> half8_t {
      return *reinterpret_cast<const half8_t*>(smem + a_rd[s] + decltype(buf)::value * Gm::a16_bytes +
                                               i * Gm::a16_tile);
    };
#pragma unroll
    for (int i = 0; i < TM; ++i) af[0][i] = a_frag(i, 0);
    if constexpr (decltype(deferred)::value) mfmas(1);
    if (more) produce_write(raw, other{});
    half2_t ws_[TN][2];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      scale_pairs(w_ok[j] ? wsc[j] : 0u, ws_[j][0], ws_[j][1]);
      wf[0][j] = dequant8(wc[j][0], ws_[j][0]);
    }
#pragma unroll
    for (int s = 0; s < 3; ++s) {
#pragma unroll
      for (int i = 0; i < TM; ++i) af[(s + 1) & 1][i] = a_frag(i, s + 1);
#pragma unroll
      for (int j = 0; j < TN; ++j) wf[(s + 1) & 1][j] = dequant8(wc[j][s + 1], ws_[j][(s + 1) >> 1]);
      mfmas(s & 1);
    }
    lgkm0();
    if (kt + 2 < KTi) wait_stage(kt + 2, kt + S - 1);
    lds_barrier();
    if (kt + S < KTi) issue(kt + S);
  };

  wait_stage(KTi > 1 ? 1 : 0, S - 1);
  lds_barrier();
  produce_write(produce_read(0), std::integral_constant<int, 0>{});
  lgkm0();
  lds_barrier();
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  using Yes = std::true_type;
  step(0, B0{}, std::false_type{});
  int kt = 1;
  for (; kt + 1 < KTi; kt += 2) {   // A buffers alternate: 0 on even steps, 1 on odd steps
    step(kt, B1{}, Yes{});
    step(kt + 1, B0{}, Yes{});
  }
  if (kt < KTi) step(kt, B1{}, Yes{});
  mfmas(1);   // the last step's deferred sub-step

  const float g = (*Ga) * (*Gw);
  const int col_in = lane & 31;
  const int row_off = 4 * (lane >> 5);
  // Accumulator block (i, j): rows m0 + 32i + 8(r/4) + row_off + r%4 (r =
  // register 0..15), GEMM column n0 + 32j + col_in.  With SwiGLU the weight
  // rows come in gate/up groups of 16, so the gate lanes (col_in < 16) pair
  // with the up lanes col_in + 16 and produce output feature
  // (n0 + 32j) / 2 + col_in.
  if constexpr (OUT != kOutNvfp4) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int64_t gcol = n0 + j * 32 + col_in;
        const int64_t col = SW ? (n0 + j * 32) / 2 + col_in : gcol;
        const bool col_ok = SW ? (col_in < 16 && col < out.Nout) : gcol < N;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = m0 + i * 32 + 8 * (r >> 2) + row_off + (r & 3);
          float v = acc[i][j][r] * g;
          if (SW) v = swiglu(v, __shfl_xor(v, 16, 64));
          if (col_ok && row < M) {
            if (OUT == kOutF32)
              reinterpret_cast<float*>(out.Y)[row * out.Nout + col] = v;
            else
              reinterpret_cast<uint16_t*>(out.Y)[row * out.Nout + col] = (uint16_t)f32_to_bf16_rne(v);
          }
        }
      }
    }
  } else {
    // NVFP4 requantization along the output columns (the next layer's K):
    // a 16-lane group holds one 16-block of one row, so the block maximum is
    // four cross-lane steps; 8 lanes pack their codes into one dword.
    const float Go = *out.G_out;
    const float den = 6.0f * Go;
    if (blockIdx.x == 0 && threadIdx.x == 0 && out.G != out.G_out) *out.G = Go;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int64_t tr = (m0 + i * 32) / 32;
      if (tr >= out.tiles_r) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int64_t gcol = n0 + j * 32 + col_in;
        const int64_t cbase = SW ? (n0 + j * 32) / 2 : n0 + j * 32;   // first output column of the block
        const int64_t tc = cbase / 64;
        if (tc >= out.tiles_c) continue;
        const int64_t col = cbase + col_in;
        const bool writer = SW ? col_in < 16 : true;
        const bool col_ok = writer && col < out.Nout && gcol < N;
        const int cc = (int)(col & 63);
        uint8_t* tcodes = out.codes + (tr * out.tiles_c + tc) * 1024;
        uint8_t* tscales = out.scales + (tr * out.tiles_c + tc) * 128;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rr = 8 * (r >> 2) + row_off + (r & 3);
          const int64_t row = tr * 32 + rr;
          float v = acc[i][j][r] * g;
          if (SW) v = swiglu(v, __shfl_xor(v, 16, 64));
          if (!(col_ok && row < M)) v = 0.0f;    // padding of the tile: zero codes and scales
          float a = fabsf(v);
          a = fmaxf(a, __shfl_xor(a, 1, 64));
          a = fmaxf(a, __shfl_xor(a, 2, 64));
          a = fmaxf(a, __shfl_xor(a, 4, 64));
          a = fmaxf(a, __shfl_xor(a, 8, 64));
          const uint32_t c = e4m3_encode_rne_sat(a / den);
          const float S = e4m3_decode(c) * Go;
          uint32_t w = (S == 0.0f ? 0u : e2m1_code(v, S)) << (4 * (lane & 7));
          w |= __shfl_xor(w, 1, 64);
          w |= __shfl_xor(w, 2, 64);
          w |= __shfl_xor(w, 4, 64);
          if (writer && (lane & 7) == 0) *reinterpret_cast<uint32_t*>(tcodes + rr * 32 + cc / 2) = w;
          if (writer && (lane & 15) == 0) tscales[rr * 4 + cc / 16] = (uint8_t)c;
        }
      }
    }
  }
}

// Launch geometry Gm over output columns n_off .. n_end-1 (n_off a multiple
// of 256; n_end a multiple of Gm::bn, or N).
template <class Gm>
hipError_t launch_geo(const GemmArgs& a, int64_t n_off, int64_t n_end, hipStream_t s) {
  const int64_t a_tiles_r = round_up(a.M, 32) / 32;
  const int64_t w_tiles_r = round_up(a.N, 32) / 32;
  const int64_t KT = round_up(a.K, 64) / 64;
  const int64_t tiles_m = (a.M + Gm::bm - 1) / Gm::bm, tiles_n = (n_end - n_off + Gm::bn - 1) / Gm::bn;
  const size_t lds = (size_t)Gm::a16_base + 2 * (size_t)Gm::a16_bytes;   // fp4 ring + fp16 A buffers
  static_assert(Gm::a16_base + 2 * Gm::a16_bytes <= kLdsBudget, "LDS budget");
  const bool sw = (a.flags & 1) != 0;
  GemmOut o{};
  o.Y = a.Y;
  o.Nout = sw ? a.N / 2 : a.N;
  if (a.out_kind == kOutNvfp4) {
    o.G_out = a.G_out;
    o.codes = a.Yq.codes;
    o.scales = a.Yq.scales;
    o.G = a.Yq.G;
    o.tiles_r = round_up(a.M, 32) / 32;
    o.tiles_c = round_up(o.Nout, 64) / 64;
  }
  typedef void (*kern_t)(const uint8_t*, const uint8_t*, const float*, const uint8_t*, const uint8_t*, const float*,
                         int64_t, int64_t, int64_t, int64_t, int64_t, GemmOut, int64_t, int64_t, int64_t);
  static const kern_t kerns[3][2] = {
      {nvfp4_gemm_kernel<Gm, kOutF32, false>, nvfp4_gemm_kernel<Gm, kOutF32, true>},
      {nvfp4_gemm_kernel<Gm, kOutBF16, false>, nvfp4_gemm_kernel<Gm, kOutBF16, true>},
      {nvfp4_gemm_kernel<Gm, kOutNvfp4, false>, nvfp4_gemm_kernel<Gm, kOutNvfp4, true>}};
  const kern_t kern = kerns[a.out_kind][sw ? 1 : 0];
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)(tiles_m * tiles_n)), dim3(Gm::threads), lds, s, a.A.codes, a.A.scales,
                     a.A.G, a.W.codes, a.W.scales, a.W.G, a.M, a.N, a_tiles_r, w_tiles_r, KT, o, tiles_m, tiles_n,
                     n_off);
  return hipGetLastError();
}

}  // namespace

__global__ void publish_scale_kernel(const float* src, float* dst) { *dst = *src; }

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s) {
  if (a.M == 0 || a.N == 0) {
    // empty result: an NVFP4 output still carries its scale
    if (a.out_kind == kOutNvfp4 && a.Yq.G != a.G_out)
      hipLaunchKernelGGL(publish_scale_kernel, dim3(1), dim3(1), 0, s, a.G_out, a.Yq.G);
    return hipGetLastError();
  }
  // 256x256 workgroup tiles as 2x4 wavefronts of 128x64, two per SIMD.  One
  // workgroup fills a CU, so a last round that would leave CUs idle is run
  // instead as a second launch of half-width (256x128) tiles over the
  // remaining column panels.
  using Full = Geo<4, 2, 2, 4, 1>;
  using Half = Geo<4, 1, 2, 4, 1>;
  const int64_t n_split = gemm_column_split(a.M, a.N, Full::bm, Full::bn, Half::bn, num_cus());
  hipError_t e = hipSuccess;
  if (n_split > 0) e = launch_geo<Full>(a, 0, n_split, s);
  if (e == hipSuccess && n_split < a.N) e = launch_geo<Half>(a, n_split, a.N, s);
  return e;
}

}  // namespace dq
