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
// block scale: the conversion's own scale operand only takes a power of two)
// and accumulates v_mfma_f32_32x32x16_f16 products in fp32.  The global
// scales are applied once in the epilogue.
//
// Structure
//  * a workgroup of WM x WN wavefronts covers a (32*TM*WM) x (32*TN*WN)
//    output tile; each wavefront owns 32*TM x 32*TN (TM x TN accumulator
//    blocks of 32x32).  The launch uses four wavefronts of 128 x 64 on a
//    256 x 128 tile and two workgroups per compute unit;
//  * operands stay compressed (4.5 bits/element) until they reach registers:
//    an LDS ring of up to six stages (one 64-column K step each: raw code tiles of
//    1 KiB and E4M3 scale tiles of 128 bytes) is filled by direct
//    global->LDS buffer loads as many steps ahead (a buffer resource per
//    operand row panel: per load a fixed lane offset, per step one scalar
//    offset, no address arithmetic in the loop); one workgroup barrier per step;
//  * within a stage, a 32x64 code tile is one contiguous KiB; the loading
//    lane i fetches 16-byte chunk 2*(i%32) + i/32 so that the consuming lane
//    l (row l%32, columns 32*(l/32)..+31) reads LDS bytes 16l..16l+15
//    (conflict-free ds_read_b128);
//  * MFMA sub-step s of a K step consumes columns 32*(l/32) + 8s .. +7 on both
//    operands (a permutation of K shared by A and W).  Each wavefront
//    dequantizes its own A and W tiles one sub-step ahead, interleaved with
//    the MFMAs of the current sub-step, and reads the next step's raw tiles
//    from LDS during the second sub-step;
//  * W is the MFMA's first operand, so an accumulator block is the transposed
//    output tile: each lane holds 4 consecutive output columns;
//  * output tiles are handed out in bands of row panels, each XCD taking a
//    compact sub-block of the tiles in flight (gemm_tile_of).
#include <algorithm>
#include <climits>
#include <type_traits>

#include "dq_device.hpp"
#include "dq_internal.hpp"

namespace dq {

namespace {

constexpr int kLdsBudget = 150 * 1024;   // of gfx950's 160 KiB
// Workgroup geometry: WM x WN wavefronts, each owning 32*TM rows x 32*TN
// columns; one 64-column K step per LDS stage; OCC workgroups per compute
// unit (registers and LDS sized for them).
template <int TM, int TN, int WM, int WN, int OCC>
struct Geo {
  static constexpr int tm = TM, tn = TN, wm = WM, wn = WN, occ = OCC;
  static constexpr int waves = WM * WN;
  static constexpr int threads = 64 * waves;
  static constexpr int bm = 32 * TM * WM;      // workgroup tile rows
  static constexpr int bn = 32 * TN * WN;      // workgroup tile columns
  static constexpr int at = bm / 32;           // A code tiles per K step
  static constexpr int wt = bn / 32;           // W code tiles per K step
  // LDS byte layout of one stage: A codes, W codes, A scales, W scales
  static constexpr int a_codes = 0;
  static constexpr int w_codes = at * 1024;
  static constexpr int a_scales = w_codes + wt * 1024;
  static constexpr int w_scales = a_scales + at * 128;
  // direct loads per stage: one per code tile, one dword load per pair of scale tiles
  static constexpr int code_loads = at + wt;
  static constexpr int scale_loads = (at + wt) / 2;
  static constexpr int cpw = code_loads / waves;
  static constexpr int spw = (scale_loads + waves - 1) / waves;
  // scale loads past the last pair land in padding after the W scales
  static constexpr int spad = (waves * spw - scale_loads) * 256;
  static constexpr int bytes = w_scales + wt * 128 + spad;
  static constexpr int stages_fit = kLdsBudget / OCC / bytes;
  static constexpr int stages = stages_fit < 6 ? stages_fit : 6;
  static constexpr int loads_per_wave = cpw + spw;
  static_assert(code_loads % waves == 0 && at % 2 == 0 && wt % 2 == 0, "uniform load distribution");
  static_assert(stages >= 4 && (stages - 1) * loads_per_wave <= 63, "LDS ring of four to six stages");
};

// 8 E2M1 codes (one dword) times an fp16 block scale -> 8 exact fp16 values.
__device__ inline half8_t dequant8(uint32_t w, half2_t s) {
  half2_t p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 0) * s;
  half2_t p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 1) * s;
  half2_t p2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 2) * s;
  half2_t p3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 3) * s;
  return half8_t{p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

// Half of dequant8: values 4*HF .. 4*HF+3 of the dword into v
template <int HF>
__device__ inline void dequant4(uint32_t w, half2_t s, half8_t& v) {
  const half2_t p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 2 * HF) * s;
  const half2_t p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 2 * HF + 1) * s;
  v[4 * HF] = p0[0];
  v[4 * HF + 1] = p0[1];
  v[4 * HF + 2] = p1[0];
  v[4 * HF + 3] = p1[1];
}

// One of the two E4M3 scale bytes in sc (byte `hi`) -> fp16 broadcast pair
__device__ inline half2_t scale_pair(uint32_t sc, int hi) {
  const half2_t s = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sc, 1.0f, false);
  return hi ? half2_t{s[1], s[1]} : half2_t{s[0], s[0]};
}

// s_waitcnt vmcnt(n) (n < 64) with expcnt / lgkmcnt left at their maximum.
// gfx9 encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at [15:14].
template <int n>
__device__ inline void wait_vm() {
  __builtin_amdgcn_s_waitcnt((n & 0xF) | (0x7 << 4) | (0xF << 8) | ((n >> 4) << 14));
}

// s_waitcnt lgkmcnt(0)
__device__ inline void wait_lgkm0() {
  __builtin_amdgcn_s_waitcnt((0x3F & 0xF) | (0x7 << 4) | (0x0 << 8) | ((0x3F >> 4) << 14));
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

// Workgroup tiles of one geometry: tiles_m x tiles_n tiles over the output
// columns from n_off on.
struct Panels {
  int64_t tiles_m, tiles_n, n_off;
};

// Workgroup tile blk (0 .. P.tiles_m * P.tiles_n - 1) of geometry Gm.
template <class Gm, int OUT, bool SW>
__device__ __forceinline__ void gemm_tile(
    int64_t blk, const Panels& P, const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const float* __restrict__ Ga, const uint8_t* __restrict__ w_codes, const uint8_t* __restrict__ w_scales,
    const float* __restrict__ Gw, int64_t M, int64_t N, int64_t a_tiles_r, int64_t w_tiles_r, int64_t KT,
    const GemmOut& out) {
  const int64_t n_off = P.n_off;
  constexpr int S = Gm::stages;
  constexpr int TM = Gm::tm, TN = Gm::tn;
  constexpr int L = Gm::loads_per_wave;
  constexpr int CPW = Gm::cpw, SPW = Gm::spw;
  extern __shared__ __align__(16) uint8_t smem[];

  const int lane = threadIdx.x & 63;
  // wavefront index as a uniform (scalar) value: the LDS destination of the
  // direct loads lives in M0 and must not look divergent to the compiler
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int64_t bm, bn;
  gemm_tile_of(blk, P.tiles_m, P.tiles_n, bm, bn);
  const int wm = wave % Gm::wm, wn = wave / Gm::wm;
  // this launch covers tiles_n column panels from output column n_off on
  const int64_t a_tr0 = bm * Gm::at, w_tr0 = n_off / 32 + bn * Gm::wt;
  const int64_t m0 = bm * Gm::bm + wm * 32 * TM;
  const int64_t n0 = n_off + bn * Gm::bn + wn * 32 * TN;
  const int KTi = (int)KT;

  // Direct loads of one stage: code tiles t = wave*CPW + u (A tiles first,
  // then W, contiguous in LDS); scale instruction idx covers tiles 2 idx
  // (lanes 0..31) and 2 idx + 1 (lanes 32..63).  Tiles
  // past the end of an operand read its last row tile (in bounds): they only
  // feed output rows / columns that are never stored.  K steps past the end
  // reload the last one into a slot that is no longer read, so every step
  // issues the same loads (no branches in the main loop).
  const int chunk = 2 * (lane & 31) + (lane >> 5);
  // Buffer resources based at this workgroup's first row tile of each
  // operand (offsets stay below at * KT * 1024 bytes, far inside 31 bits);
  // per load a fixed lane offset, per K step one scalar offset.  The bases
  // sit kBias bytes lower, so that the lane offsets, from which the
  // instruction offsets are taken back out, stay non-negative.
  constexpr int kBias = 4096;
  auto rsrc = [](const uint8_t* base, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base) - kBias, 0, (int)(bytes + kBias), 0x00020000);
  };
  const __amdgpu_buffer_rsrc_t rac = rsrc(a_codes + a_tr0 * KT * 1024, (int64_t)Gm::at * KT * 1024);
  const __amdgpu_buffer_rsrc_t rwc = rsrc(w_codes + w_tr0 * KT * 1024, (int64_t)Gm::wt * KT * 1024);
  const __amdgpu_buffer_rsrc_t ras = rsrc(a_scales + a_tr0 * KT * 128, (int64_t)Gm::at * KT * 128);
  const __amdgpu_buffer_rsrc_t rws = rsrc(w_scales + w_tr0 * KT * 128, (int64_t)Gm::wt * KT * 128);
  // wavefront w loads code tiles w*CPW + u (LDS: one M0 for all of them, the
  // instruction offset u KiB, which the hardware adds to both addresses, is
  // taken back out of the lane offset) and scale pairs w*SPW + u
  uint32_t c_off[CPW];
  bool c_a[CPW];
#pragma unroll
  for (int u = 0; u < CPW; ++u) {
    const int t = wave * CPW + u;
    const bool is_a = t < Gm::at;
    const int b = is_a ? t : t - Gm::at;
    const int64_t tr = min((is_a ? a_tr0 : w_tr0) + b, (is_a ? a_tiles_r : w_tiles_r) - 1) - (is_a ? a_tr0 : w_tr0);
    c_a[u] = is_a;
    c_off[u] = (uint32_t)(tr * KT * 1024 + chunk * 16 + kBias - u * 1024);
  }
  const int c_m0 = wave * CPW * 1024;
  uint32_t s_off[SPW];
  bool s_a[SPW];
#pragma unroll
  for (int u = 0; u < SPW; ++u) {
    const int idx = min(wave * SPW + u, Gm::scale_loads - 1);   // past the last pair: its data, into the padding
    const int t = 2 * idx + (lane >> 5);
    const bool is_a = 2 * idx < Gm::at;   // both tiles of a pair belong to one operand (at is even)
    const int b = is_a ? t : t - Gm::at;
    const int64_t tr = min((is_a ? a_tr0 : w_tr0) + b, (is_a ? a_tiles_r : w_tiles_r) - 1) - (is_a ? a_tr0 : w_tr0);
    s_a[u] = is_a;
    s_off[u] = (uint32_t)(tr * KT * 128 + (lane & 31) * 4 + kBias - u * 256);
  }
  const int s_m0 = Gm::a_scales + wave * SPW * 256;
  // stage kt into ring slot `slot` (kt past the end: the last one again)
  // load r (0 .. CPW + SPW - 1) of stage kt into ring slot `slot`
  auto issue_one = [&](int kt, int slot, auto rc) {
    constexpr int r = decltype(rc)::value;
    uint8_t* stage = smem + slot * Gm::bytes;
    const int ktc = kt < KTi ? kt : KTi - 1;
    if constexpr (r < CPW) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(c_a[r] ? rac : rwc,
                                               (__attribute__((address_space(3))) void*)(stage + c_m0), 16,
                                               c_off[r], ktc * 1024, r * 1024, 0);
    } else {
      constexpr int u = r - CPW;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(s_a[u] ? ras : rws,
                                               (__attribute__((address_space(3))) void*)(stage + s_m0), 4,
                                               s_off[u], ktc * 128, u * 256, 0);
    }
  };
  auto issue = [&](int kt, int slot) {
    uint8_t* stage = smem + slot * Gm::bytes;
    const int ktc = kt < KTi ? kt : KTi - 1;
    static_for<0, CPW>([&](auto ic) {
      constexpr int u = decltype(ic)::value;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(c_a[u] ? rac : rwc,
                                               (__attribute__((address_space(3))) void*)(stage + c_m0), 16,
                                               c_off[u], ktc * 1024, u * 1024, 0);
    });
    static_for<0, SPW>([&](auto ic) {
      constexpr int u = decltype(ic)::value;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(s_a[u] ? ras : rws,
                                               (__attribute__((address_space(3))) void*)(stage + s_m0), 4,
                                               s_off[u], ktc * 128, u * 256, 0);
    });
  };

  float16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = float16_t{};

  // Raw operands of one K step (codes, and the two E4M3 scales of the lane's
  // 32 columns) and dequantized fp16 operands of one sub-step.
  struct Raw {
    uint4_t a[TM], w[TN];
    uint32_t sa[TM], sw[TN];
  };
  struct Ops {
    half8_t a[TM], w[TN];
  };
  const int a_rd = Gm::a_codes + wm * TM * 1024 + lane * 16;
  const int w_rd = Gm::w_codes + wn * TN * 1024 + lane * 16;
  const int sl = (lane & 31) * 4 + (lane >> 5) * 2;
  const int as_rd = Gm::a_scales + wm * TM * 128 + sl;
  const int ws_rd = Gm::w_scales + wn * TN * 128 + sl;
  constexpr int kTiles = TM + TN;
  constexpr int kReads = 2 * kTiles;
  constexpr int kMfmas = TM * TN;
  auto read_one = [&](const uint8_t* stg, Raw& R, int r) {
    if (r < TM) R.a[r] = *reinterpret_cast<const uint4_t*>(stg + a_rd + r * 1024);
    else if (r < kTiles) R.w[r - TM] = *reinterpret_cast<const uint4_t*>(stg + w_rd + (r - TM) * 1024);
    else if (r < kTiles + TM) R.sa[r - kTiles] = *reinterpret_cast<const uint16_t*>(stg + as_rd + (r - kTiles) * 128);
    else R.sw[r - kTiles - TM] = *reinterpret_cast<const uint16_t*>(stg + ws_rd + (r - kTiles - TM) * 128);
  };
  // sub-step s of tile u (A tiles first): dword s of the codes, scale byte s/2
  auto dequant_one = [&](const Raw& R, int s, Ops& D, int u) {
    if (u < TM) D.a[u] = dequant8(R.a[u][s], scale_pair(R.sa[u], s >> 1));
    else D.w[u - TM] = dequant8(R.w[u - TM][s], scale_pair(R.sw[u - TM], s >> 1));
  };
  // the same in two halves, issued after different MFMAs (tile u's scale
  // pair kept in sp[u] between them)
  half2_t sp[kTiles];
  auto dequant_half = [&](const Raw& R, int s, Ops& D, int v) {
    const int u = v >> 1;
    if (v & 1) {
      if (u < TM) dequant4<1>(R.a[u][s], sp[u], D.a[u]);
      else dequant4<1>(R.w[u - TM][s], sp[u], D.w[u - TM]);
    } else if (u < TM) {
      sp[u] = scale_pair(R.sa[u], s >> 1);
      dequant4<0>(R.a[u][s], sp[u], D.a[u]);
    } else {
      sp[u] = scale_pair(R.sw[u - TM], s >> 1);
      dequant4<0>(R.w[u - TM][s], sp[u], D.w[u - TM]);
    }
  };
  // W as the first operand: the accumulator block is the transposed output tile
  auto mfma_one = [&](const Ops& D, int q) {
    const int i = q / TN, j = q % TN;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(D.w[j], D.a[i], acc[i][j], 0, 0, 0);
  };

  if (KTi > 0) {
    // prologue: stages 0 .. S-1 in flight, stage 0 landed everywhere
#pragma unroll
    for (int st = 0; st < S; ++st) issue(st, st);
    wait_vm<(S - 1) * L>();
    lds_barrier();
    Raw R0, R1;
    Ops D0, D1;
    // One K step, its raw operands in Rc and sub-step 0 already dequantized
    // in D0.  Sub-step s runs its MFMAs on D[s % 2] while the next sub-step
    // is dequantized into the other buffer, half a tile (four conversions
    // and four multiplies) after each MFMA or so, evenly spread: a lone
    // wavefront per SIMD issues its MFMAs on time only when no MFMA is
    // followed by a whole tile's conversions.  After the first two MFMAs: the wait for
    // stage kt+1 and the barrier (stage kt+1 landed everywhere, everyone done
    // reading stage kt's slot, which is refilled with stage kt+S, one load
    // per MFMA from the third on).  During
    // sub-step 1 the raw tiles of stage kt+1 are read into Rn; sub-step 3
    // dequantizes sub-step 0 of the next step from them.  The sched_barrier
    // fences keep this order; the empty asm statements pin the accumulators
    // at the end of the step (the compiler would otherwise sink the MFMAs,
    // pure register operations, behind the next step's barrier).
    auto step = [&](int kt, Raw& Rc, Raw& Rn, int slot) {
      const int nslot = slot + 1 == S ? 0 : slot + 1;
      const uint8_t* stg_next = smem + nslot * Gm::bytes;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        Ops& Dc = (s & 1) ? D1 : D0;
        Ops& Dn = (s & 1) ? D0 : D1;
        if (s == 3) wait_lgkm0();
#pragma unroll
        for (int q = 0; q < kMfmas; ++q) {
          __builtin_amdgcn_sched_barrier(0);
          mfma_one(Dc, q);
          __builtin_amdgcn_sched_barrier(0);
          if (s == 0 && q == 1) {
            wait_vm<(S - 2) * L>();
            lds_barrier();
            if (2 + L > kMfmas) issue(kt + S, slot);
            __builtin_amdgcn_sched_barrier(0);
          }
          // the refill of stage kt's slot, one load after each of the next
          // MFMAs (all at once when the sub-step has too few of them)
          if (2 + L <= kMfmas && s == 0 && q >= 2 && q < 2 + L) {
            static_for<0, L>([&](auto rc) {
              if (q == 2 + decltype(rc)::value) issue_one(kt + S, slot, rc);
            });
            __builtin_amdgcn_sched_barrier(0);
          }
          if (s == 1) {
#pragma unroll
            for (int r = 0; r < kReads; ++r)
              if ((r * kMfmas) / kReads == q) read_one(stg_next, Rn, r);
            __builtin_amdgcn_sched_barrier(0);
          }
#pragma unroll
          for (int v = 0; v < 2 * kTiles; ++v)
            if ((v * kMfmas) / (2 * kTiles) == q) {
              if (s < 3) dequant_half(Rc, s + 1, Dn, v);
              else dequant_half(Rn, 0, Dn, v);
            }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) asm volatile("" : "+a"(acc[i][j]));
    };
    // steps alternate Rc / Rn between R0 and R1; the first step is peeled
    // when their number is odd
    auto first = [&](Raw& R) {
#pragma unroll
      for (int r = 0; r < kReads; ++r) read_one(smem, R, r);
      wait_lgkm0();
#pragma unroll
      for (int u = 0; u < kTiles; ++u) dequant_one(R, 0, D0, u);
    };
    int kt = 0, slot = 0;
    auto adv = [&](int sl) { return sl + 1 == S ? 0 : sl + 1; };
    if (KTi & 1) {
      first(R1);
      step(0, R1, R0, 0);
      kt = 1;
      slot = 1;
    } else {
      first(R0);
    }
    for (; kt < KTi; kt += 2) {
      step(kt, R0, R1, slot);
      slot = adv(slot);
      step(kt + 1, R1, R0, slot);
      slot = adv(slot);
    }
    // drain the redundant reloads of the last steps before the workgroup ends
    wait_vm<0>();
  }

  // Block (i, j) holds, in lane l, output row m0 + 32i + l%32 and GEMM
  // columns n0 + 32j + 8g + 4h + t in register 4g + t (g, t = 0..3,
  // h = l/32).  With SwiGLU the weight rows come in gate/up groups of 16, so
  // registers 4g + t (g < 2, gate) and 4(g + 2) + t (up) of the same lane
  // meet, producing output feature (n0 + 32j)/2 + 8g + 4h + t.
  const float gs = (*Ga) * (*Gw);
  const int h = lane >> 5;
  if constexpr (OUT == kOutBF16 && !SW) {
    // A full wave tile leaves through LDS: each store instruction then writes
    // whole 128-byte rows instead of 16 bytes of each of 32 rows.  The barrier
    // covers the other waves' last LDS reads and direct loads into the ring.
    __syncthreads();
    constexpr int RS = 64 * TN + 16;   // LDS bytes per staged row (the pad staggers banks)
    constexpr int LPR = 4 * TN;        // lanes per row in the read-back (16 bytes each)
    if (m0 + 32 * TM <= M && n0 + 32 * TN <= out.Nout && (out.Nout & 7) == 0) {
      uint8_t* ep = smem + (size_t)wave * 32 * RS;
      const int rl = lane & 31;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            uint32_t b[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) b[t] = f32_to_bf16_rne(acc[i][j][4 * g + t] * gs);
            *reinterpret_cast<uint2_t*>(ep + rl * RS + (32 * j + 8 * g + 4 * h) * 2) =
                uint2_t{b[0] | (b[1] << 16), b[2] | (b[3] << 16)};
          }
#pragma unroll
        for (int r0 = 0; r0 < 32; r0 += 64 / LPR) {
          const int rr = r0 + lane / LPR, seg = lane % LPR;
          const uint4_t v = *reinterpret_cast<const uint4_t*>(ep + rr * RS + seg * 16);
          *reinterpret_cast<uint4_t*>(reinterpret_cast<uint16_t*>(out.Y) + (m0 + 32 * i + rr) * out.Nout + n0 +
                                      seg * 8) = v;
        }
      }
      return;
    }
  }
  if constexpr (OUT != kOutNvfp4) {
    const bool vec = (out.Nout & 3) == 0;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int64_t row = m0 + i * 32 + (lane & 31);
      if (row >= M) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
#pragma unroll
        for (int g = 0; g < (SW ? 2 : 4); ++g) {
          float v[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            v[t] = acc[i][j][4 * g + t] * gs;
            if (SW) v[t] = swiglu(v[t], acc[i][j][4 * (g + 2) + t] * gs);
          }
          const int64_t col = (SW ? (n0 + j * 32) / 2 : n0 + j * 32) + 8 * g + 4 * h;
          if (OUT == kOutF32) {
            float* y = reinterpret_cast<float*>(out.Y) + row * out.Nout + col;
            if (vec && col + 3 < out.Nout) {
              *reinterpret_cast<float4_t*>(y) = float4_t{v[0], v[1], v[2], v[3]};
            } else {
#pragma unroll
              for (int t = 0; t < 4; ++t)
                if (col + t < out.Nout) y[t] = v[t];
            }
          } else {
            uint32_t b[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) b[t] = f32_to_bf16_rne(v[t]);
            uint16_t* y = reinterpret_cast<uint16_t*>(out.Y) + row * out.Nout + col;
            if (vec && col + 3 < out.Nout) {
              *reinterpret_cast<uint2_t*>(y) = uint2_t{b[0] | (b[1] << 16), b[2] | (b[3] << 16)};
            } else {
#pragma unroll
              for (int t = 0; t < 4; ++t)
                if (col + t < out.Nout) y[t] = (uint16_t)b[t];
            }
          }
        }
      }
    }
  } else {
    // NVFP4 requantization along the output columns (the next layer's K):
    // a 16-column block of a row is held by lanes l and l ^ 32 (8 values
    // each), so the block maximum is one cross-lane step; each of the two
    // lanes stores one dword of 8 codes.
    const float Go = *out.G_out;
    const float den = 6.0f * Go;
    if (blockIdx.x == 0 && threadIdx.x == 0 && out.G != out.G_out) *out.G = Go;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int64_t tr = (m0 + i * 32) / 32;
      if (tr >= out.tiles_r) continue;
      const int rr = lane & 31;
      const int64_t row = tr * 32 + rr;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
#pragma unroll
        for (int q = 0; q < (SW ? 1 : 2); ++q) {
          const int64_t cbase = SW ? (n0 + j * 32) / 2 : n0 + j * 32 + 16 * q;   // first column of the block
          const int64_t tc = cbase / 64;
          if (tc >= out.tiles_c) continue;
          float v[8];
          float a = 0.0f;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int g = (SW ? 0 : 2 * q) + e / 4, t = e % 4;
            float x = acc[i][j][4 * g + t] * gs;
            if (SW) x = swiglu(x, acc[i][j][4 * (g + 2) + t] * gs);
            const int64_t col = cbase + 8 * (e / 4) + 4 * h + t;
            if (!(row < M && col < out.Nout)) x = 0.0f;   // padding of the tile: zero codes and scales
            v[e] = x;
            a = fmaxf(a, fabsf(x));
          }
          a = fmaxf(a, __shfl_xor(a, 32, 64));
          const uint32_t c = e4m3_encode_rne_sat(a / den);
          const float Sc = e4m3_decode(c) * Go;
          // the 8 codes as one dword (value e in nibble e): the activation
          // quantizer's arithmetic, two conversions per instruction
          const float rcp = 1.0f / Sc;   // Sc == 0: the codes are forced to 0 below
          float yq[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) yq[e] = div_by_scale(v[e], Sc, rcp);
          uint32_t cw = cvt_pk_fp4<0>(0u, yq[0], yq[1]);
          cw = cvt_pk_fp4<1>(cw, yq[2], yq[3]);
          cw = cvt_pk_fp4<2>(cw, yq[4], yq[5]);
          cw = cvt_pk_fp4<3>(cw, yq[6], yq[7]);
          cw = Sc == 0.0f ? 0u : fp4_canonical_zero(cw);
          const uint32_t P0 = cw & 0xFFFFu, P1 = cw >> 16;
          // dword 0 = columns cbase..+7 (h = 0's P0, h = 1's P0); dword 1 =
          // columns cbase+8..+15 (h = 0's P1, h = 1's P1)
          const uint32_t recv = (uint32_t)__shfl_xor((int)(h == 0 ? P1 : P0), 32, 64);
          const uint32_t word = h == 0 ? (P0 | (recv << 16)) : (recv | (P1 << 16));
          const int cc = (int)(cbase & 63);
          uint8_t* tcodes = out.codes + (tr * out.tiles_c + tc) * 1024;
          *reinterpret_cast<uint32_t*>(tcodes + rr * 32 + cc / 2 + 4 * h) = word;
          if (h == 0) out.scales[(tr * out.tiles_c + tc) * 128 + rr * 4 + cc / 16] = (uint8_t)c;
        }
      }
    }
  }
}

// One launch, two geometries: workgroups 0 .. big tiles - 1 take the tiles
// of Gm (columns 0 .. split - 1), the rest those of Gh (columns split ..).
template <class Gm, class Gh, int OUT, bool SW>
__global__ __launch_bounds__(Gm::threads, Gm::occ) void nvfp4_gemm_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales, const float* __restrict__ Ga,
    const uint8_t* __restrict__ w_codes, const uint8_t* __restrict__ w_scales, const float* __restrict__ Gw,
    int64_t M, int64_t N, int64_t a_tiles_r, int64_t w_tiles_r, int64_t KT, GemmOut out, Panels big, Panels small) {
  static_assert(Gm::threads == Gh::threads && Gm::occ == Gh::occ, "one launch shape");
  const int64_t nb = big.tiles_m * big.tiles_n;
  const int64_t b = blockIdx.x;
  if (b < nb)
    gemm_tile<Gm, OUT, SW>(b, big, a_codes, a_scales, Ga, w_codes, w_scales, Gw, M, N, a_tiles_r, w_tiles_r, KT, out);
  else
    gemm_tile<Gh, OUT, SW>(b - nb, small, a_codes, a_scales, Ga, w_codes, w_scales, Gw, M, N, a_tiles_r, w_tiles_r, KT,
                           out);
}

// One launch: output columns 0 .. split-1 in Gm tiles, split .. N-1 in Gh
// tiles (split a multiple of Gm::bn and of 128, so that an NVFP4 output tile
// of the SwiGLU half-width result never straddles the two; or N).
template <class Gm, class Gh, bool kBf16Only = false>
hipError_t launch_geo(const GemmArgs& a, int64_t split, hipStream_t s) {
  const int64_t a_tiles_r = round_up(a.M, 32) / 32;
  const int64_t w_tiles_r = round_up(a.N, 32) / 32;
  const int64_t KT = round_up(a.K, 64) / 64;
  // the loaders address one workgroup's row panel of an operand with 32-bit
  // buffer offsets (at most 8 code tiles of KT KiB)
  if ((int64_t)std::max(std::max(Gm::at, Gm::wt), std::max(Gh::at, Gh::wt)) * KT * 1024 + 4096 > INT32_MAX)
    return hipErrorNotSupported;
  const Panels big{(a.M + Gm::bm - 1) / Gm::bm, (split + Gm::bn - 1) / Gm::bn, 0};
  const Panels small{split < a.N ? (a.M + Gh::bm - 1) / Gh::bm : 0, (a.N - split + Gh::bn - 1) / Gh::bn, split};
  const int64_t blocks = big.tiles_m * big.tiles_n + small.tiles_m * small.tiles_n;
  const size_t lds = std::max((size_t)Gm::stages * Gm::bytes, (size_t)Gh::stages * Gh::bytes);
  static_assert(Gm::stages * Gm::bytes <= kLdsBudget && Gh::stages * Gh::bytes <= kLdsBudget, "LDS budget");
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
                         int64_t, int64_t, int64_t, int64_t, int64_t, GemmOut, Panels, Panels);
  kern_t kern;
  if constexpr (kBf16Only) {
    kern = nvfp4_gemm_kernel<Gm, Gh, kOutBF16, false>;
  } else {
    static const kern_t kerns[3][2] = {
        {nvfp4_gemm_kernel<Gm, Gh, kOutF32, false>, nvfp4_gemm_kernel<Gm, Gh, kOutF32, true>},
        {nvfp4_gemm_kernel<Gm, Gh, kOutBF16, false>, nvfp4_gemm_kernel<Gm, Gh, kOutBF16, true>},
        {nvfp4_gemm_kernel<Gm, Gh, kOutNvfp4, false>, nvfp4_gemm_kernel<Gm, Gh, kOutNvfp4, true>}};
    kern = kerns[a.out_kind][sw ? 1 : 0];
  }
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(Gm::threads), lds, s, a.A.codes, a.A.scales, a.A.G,
                     a.W.codes, a.W.scales, a.W.G, a.M, a.N, a_tiles_r, w_tiles_r, KT, o, big, small);
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
  // bf16 output without SwiGLU on grids of at least two full rounds of
  // 256x256 tiles: one workgroup of four 128x128 wavefronts per compute unit
  // (one wavefront per SIMD, 256 accumulator registers).  A wavefront
  // dequantizes a third fewer operand elements per MFMA than a 128x64 one;
  // on such grids that outweighs the lost overlap between two workgroups
  // (27B down-projection at M = 32768 4-5 % faster, M = 8192 3 %, the 8B
  // down-projection at M = 8192 6 %, the 27B gate/up shape at M = 4096 2 %).
  // The NVFP4 and SwiGLU epilogues are longer and lose more than that when no
  // second workgroup runs its main loop meanwhile (2-7 % slower at
  // 4096 x 34816 x 5120).  A partial last round of at most half the compute
  // units takes the trailing columns as 256x128 tiles, one per compute unit.
  const int cus = num_cus();
  if (a.out_kind == kOutBF16 && (a.flags & 1) == 0) {
    using Gb = Geo<4, 4, 2, 2, 1>;
    using Gbh = Geo<4, 2, 2, 2, 1>;
    const int64_t tm = (a.M + Gb::bm - 1) / Gb::bm, panels = (a.N + Gb::bn - 1) / Gb::bn;
    const int64_t tiles = tm * panels, rounds = tiles / cus, rest = tiles % cus;
    if (rounds >= 2) {
      const int64_t split = rest > 0 && 2 * rest <= cus ? rounds * cus / tm * Gb::bn : a.N;
      return launch_geo<Gb, Gbh, true>(a, split, s);
    }
  }
  // Otherwise 256x128 workgroup tiles as 2x2 wavefronts of 128x64, two
  // workgroups per compute unit (two wavefronts per SIMD): one workgroup's
  // dequantization and barrier waits overlap the other's MFMAs, and a
  // workgroup's output stores overlap the other's main loop (on grids of one
  // or two rounds 9-17 % faster than the 256x256 tiles).  128x128 tiles (2x2
  // wavefronts of 64x64) dequantize a third more operand elements per MFMA,
  // so they only take the columns of a last round that would leave most
  // slots empty (at most a quarter full), or the whole grid when it is under
  // one round.  Measured on the paper's linears: the 27B o-projection (a
  // quarter-full last round) 10 % faster, shapes with a half-full last round
  // unchanged or 1-2 % slower, so those keep 256x128 tiles.
  using Gm = Geo<4, 2, 2, 2, 2>;
  using Gh = Geo<2, 2, 2, 2, 2>;
  const int64_t slots = (int64_t)cus * Gm::occ;
  const int64_t tm = (a.M + Gm::bm - 1) / Gm::bm, panels = (a.N + Gm::bn - 1) / Gm::bn;
  const int64_t tiles = tm * panels, rounds = tiles / slots, rest = tiles % slots;
  int64_t split = a.N;
  if (rounds == 0 && 2 * tiles <= slots)
    split = 0;
  else if (rounds > 0 && rest > 0 && 4 * rest <= slots)
    split = rounds * slots / tm * Gm::bn;
  return launch_geo<Gm, Gh>(a, split, s);
}

}  // namespace dq
