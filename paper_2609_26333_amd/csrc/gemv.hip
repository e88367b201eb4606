// Weight-only LUT GEMV for decode on gfx950 (paper Sec. 2.3 "format
// disaggregation": activations stay bf16 on decode; App. C "Kernel
// specification": time is set by the bytes of weight streamed per token).
//
//   y[b, n] = sum_k x[b, k] * w_hat[n, k],  w_hat = LUT_n[code]  (PER_ROW)
//                                           w_hat = grid[code] * d_blk * G  (PAPER_GRID)
//
// Design (MI355X: 8 TB/s HBM against ~39 T VALU lane-ops/s leaves under two
// VALU instructions per 3-bit weight):
//  * codes stream with one coalesced wavefront load per 16-row x 128-column
//    chunk of a row tile (64 lanes x 12 bytes for 3 bits, x 8 bytes for 2
//    bits), a ring of loads kept in flight ahead of use;
//  * each 32-code group is split into eight 4-code byte selectors with shifts
//    and masks (the bit layout in dq.h is chosen for this), and v_perm_b32
//    looks the 4 codes up in register-resident byte tables (low bytes and
//    high bytes of the row's fp16 entries), then interleaves them into fp16
//    pairs: about 1.6 VALU instructions per 3-bit weight;
//  * the multiply-accumulate runs on MFMA (v_mfma_f32_16x16x32_f16: 16 weight
//    rows x 32 k x 16 batch columns), so batch 1..16 costs the same VALU work;
//  * activations are staged into LDS as fp16, rescaled by a power of two
//    (exact products with the fp16 table); the wavefronts of a workgroup
//    split K and reduce through LDS in a fixed order, so results are
//    deterministic.
// Two kernels: a persistent one (resident workgroups looping over row tiles,
// whenever the activations fit in LDS) and a piecewise one for larger B*K.
#include <algorithm>
#include <atomic>
#include <cstdint>
#include <mutex>

#include "dq.h"
#include "dq_device.hpp"
#include "dq_internal.hpp"

namespace dq {

namespace {

constexpr int kStageVec = 4;    // register-staged 8-element activation vectors per thread and piece

// One lane's 32-code group: 12 bytes (3 bits) or 8 bytes (2 bits).  Plain
// structs, so that sizeof is exactly the group size (a 3-element vector type
// would be padded to 16 bytes).
struct Group3 {
  uint32_t w[3];
};
struct Group2 {
  uint32_t w[2];
};
static_assert(sizeof(Group3) == 12 && sizeof(Group2) == 8, "group sizes");

template <int BITS>
struct CodeVec;
template <>
struct CodeVec<3> {
  typedef Group3 type;
  static constexpr int bytes = 12;
};
template <>
struct CodeVec<2> {
  typedef Group2 type;
  static constexpr int bytes = 8;
};

// fp16 pair from the low-byte and high-byte lookups of four codes
__device__ inline void lookup4(uint32_t sel, uint32_t tl0, uint32_t tl1, uint32_t th0, uint32_t th1,
                               uint32_t& p0, uint32_t& p1) {
  const uint32_t lo = __builtin_amdgcn_perm(tl1, tl0, sel);
  const uint32_t hi = __builtin_amdgcn_perm(th1, th0, sel);
  p0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);
  p1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);
}

// 8 selectors (4 codes each, byte values 0..2^BITS-1) of one 32-code group
template <int BITS>
__device__ inline void selectors(const typename CodeVec<BITS>::type& w, uint32_t (&s)[8]);

template <>
__device__ inline void selectors<3>(const Group3& g, uint32_t (&s)[8]) {
  const uint32_t* w = g.w;
  s[0] = w[0] & 0x07070707u;
  s[1] = (w[0] >> 3) & 0x07070707u;
  s[2] = w[1] & 0x07070707u;
  s[3] = (w[1] >> 3) & 0x07070707u;
  s[4] = w[2] & 0x07070707u;
  s[5] = (w[2] >> 3) & 0x07070707u;
  s[6] = ((w[0] >> 6) & 0x03030303u) | ((w[2] >> 4) & 0x04040404u);
  s[7] = ((w[1] >> 6) & 0x03030303u) | ((w[2] >> 5) & 0x04040404u);
}

template <>
__device__ inline void selectors<2>(const Group2& g, uint32_t (&s)[8]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    s[j] = (g.w[0] >> (2 * j)) & 0x03030303u;
    s[4 + j] = (g.w[1] >> (2 * j)) & 0x03030303u;
  }
}

__device__ inline half8_t as_half8(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  uint4_t u{a, b, c, d};
  return __builtin_bit_cast(half8_t, u);
}

__device__ inline half8_t scale_half8(half8_t v, half2_t s) {
  half2_t a{v[0], v[1]}, b{v[2], v[3]}, c{v[4], v[5]}, d{v[6], v[7]};
  a *= s;
  b *= s;
  c *= s;
  d *= s;
  return half8_t{a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
}

// Table of one row (PER_ROW) or the grid (PAPER_GRID): the 2^BITS fp16
// entries as raw dwords (2 bits: the upper half is unused).
template <int BITS>
__device__ inline uint4_t load_table(const uint16_t* L) {
  if (BITS == 3) return *reinterpret_cast<const uint4_t*>(L);
  const uint2_t d = *reinterpret_cast<const uint2_t*>(L);
  return uint4_t{d[0], d[1], 0u, 0u};
}

// Low bytes and high bytes of the table entries, as v_perm_b32 pools.
template <int BITS>
__device__ inline void table_pools(const uint4_t& d, uint32_t& tl0, uint32_t& tl1, uint32_t& th0, uint32_t& th1) {
  tl0 = __builtin_amdgcn_perm(d[1], d[0], 0x06040200u);
  th0 = __builtin_amdgcn_perm(d[1], d[0], 0x07050301u);
  if (BITS == 3) {
    tl1 = __builtin_amdgcn_perm(d[3], d[2], 0x06040200u);
    th1 = __builtin_amdgcn_perm(d[3], d[2], 0x07050301u);
  } else {
    tl1 = tl0;
    th1 = th0;
  }
}

// Piecewise kernel: work decomposition.  A workgroup holds RT row tiles x
// KS K-splits (W = RT*KS wavefronts); wavefront (rt, ks) consumes chunks ks,
// ks+KS, ... of row tile rt.  Each wavefront walks a fixed sequence of CPW
// slots per activation piece (a multiple of its load ring) and keeps RING
// code loads in flight.  A slot past the end of the piece's chunks re-reads
// the piece's last chunk and multiplies it by a zero activation chunk instead
// of branching, so the slot loop has no data-dependent control flow.  The KS
// partial sums of a row tile are reduced through LDS in a fixed order.  Each
// activation piece is staged through registers, and the next piece's
// activations are loaded while the current one is consumed.
//
// Memory order.  The weight codes stream from HBM as long row-hit bursts that
// keep every channel busy; a scattered miss issued behind them (the
// activations, shared by all workgroups) waits until the streams drain.  So a
// workgroup stages its first activation piece before it issues any code load,
// and with several pieces the workgroups of each XCD first pull the whole
// activation matrix into that XCD's L2, which the later pieces then hit.
struct GemvPlan {
  int RT, KS, PK, CPW, npieces;
  int64_t tiles, KC;
};

// Raw buffer loads (LLVM AMDGPU intrinsics): a scalar resource (base, size),
// a per-lane VGPR offset and a uniform SGPR offset, so the address of a code
// load costs no VALU instruction; offsets past the resource size read zero.
typedef int32_t i32x2_t __attribute__((ext_vector_type(2)));
typedef int32_t i32x3_t __attribute__((ext_vector_type(3)));
typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));
__device__ i32x2_t raw_buffer_load_b64(i32x4_t rsrc, int32_t voff, int32_t soff,
                                       int32_t aux) __asm("llvm.amdgcn.raw.buffer.load.v2i32");
__device__ i32x3_t raw_buffer_load_b96(i32x4_t rsrc, int32_t voff, int32_t soff,
                                       int32_t aux) __asm("llvm.amdgcn.raw.buffer.load.v3i32");
__device__ int16_t raw_buffer_load_b16(i32x4_t rsrc, int32_t voff, int32_t soff,
                                       int32_t aux) __asm("llvm.amdgcn.raw.buffer.load.i16");
__device__ int32_t raw_buffer_load_b32(i32x4_t rsrc, int32_t voff, int32_t soff,
                                       int32_t aux) __asm("llvm.amdgcn.raw.buffer.load.i32");

// gfx9 buffer resource over [p, p + bytes): 48-bit base, stride 0, byte range,
// 32-bit data format (raw loads ignore the format)
__device__ inline i32x4_t buffer_resource(const void* p, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  return i32x4_t{(int32_t)(uint32_t)a, (int32_t)(uint32_t)((a >> 32) & 0xFFFFu), (int32_t)bytes, 0x00020000};
}

// One wavefront's code stream over its row tile: a ring of RING chunk loads
// (and, for PAPER_GRID, of the chunk's two block-scale bytes).
template <int BITS, int MODE, int RING>
struct CodeStream {
  typedef typename CodeVec<BITS>::type cvec;
  static constexpr int kChunkBytes = 64 * CodeVec<BITS>::bytes;
  i32x4_t rcodes;         // the tile's codes
  i32x4_t rscales;        // PAPER_GRID: the tile's block scales
  int32_t lane_code;      // this lane's group within a chunk: lane * group bytes
  int32_t lane_scale;     // this lane's scale pair within a chunk: lane * 2
  int PK, KS, ks, KC;
  cvec ring[RING];
  uint32_t sring[RING];

  __device__ void init(const uint8_t* tile_codes, const uint8_t* tile_scales, int lane, int PK_, int KS_, int ks_,
                       int KC_) {
    rcodes = buffer_resource(tile_codes, (uint32_t)KC_ * kChunkBytes);
    if (MODE == 1) rscales = buffer_resource(tile_scales, (uint32_t)KC_ * 128);
    lane_code = lane * CodeVec<BITS>::bytes;
    lane_scale = lane * 2;
    PK = PK_;
    KS = KS_;
    ks = ks_;
    KC = KC_;
  }
  // chunk of slot s in piece p, clamped to the piece's last chunk (in bounds)
  __device__ int chunk(int p, int s) const { return min(p * PK + s * KS + ks, min((p + 1) * PK, KC) - 1); }
  __device__ void load(int r, int c) {
    if constexpr (BITS == 3) {
      const i32x3_t v = raw_buffer_load_b96(rcodes, lane_code, c * kChunkBytes, 0);
      ring[r] = cvec{{(uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2]}};
    } else {
      const i32x2_t v = raw_buffer_load_b64(rcodes, lane_code, c * kChunkBytes, 0);
      ring[r] = cvec{{(uint32_t)v[0], (uint32_t)v[1]}};
    }
    if (MODE == 1) sring[r] = (uint16_t)raw_buffer_load_b16(rscales, lane_scale, c * 128, 0);
  }
};

// Consume the CPW slots of piece p (activation chunks of the staged piece
// start at xrow; chunk PK of every staged row is zero), prefetching RING slots
// ahead, into piece pn once the sequence wraps.  pacc[st] accumulates the
// st-th 32-column step of every chunk, so consecutive MFMAs are independent.
template <int BITS, int MODE, int RING>
__device__ __forceinline__ void consume(CodeStream<BITS, MODE, RING>& cs, int p, int pn, int CPW,
                                        const _Float16* xrow, int zero_shift, const uint4_t& tab,
                                        float4_t (&pacc)[4]) {
  uint32_t tl0, tl1, th0, th1;
  table_pools<BITS>(tab, tl0, tl1, th0, th1);
  // activation fragments of slot s (4 x 8 fp16 per lane); those of slot s+1
  // are read from LDS while slot s computes
  auto xfrag = [&](int s, half8_t (&f)[4]) {
    const half8_t* xp = reinterpret_cast<const half8_t*>(xrow + min(s * cs.KS + cs.ks + zero_shift, cs.PK) * 128);
#pragma unroll
    for (int st = 0; st < 4; ++st) f[st] = xp[st];
  };
  half8_t bf[4];
  xfrag(0, bf);
  for (int s0 = 0; s0 < CPW; s0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) {
      const int s = s0 + r;
      half8_t bn[4];
      xfrag(s + 1, bn);   // past CPW: a zero or in-range chunk, never used
      // keep these reads at the top of the slot (the scheduler would sink
      // them next to their MFMAs and expose the LDS latency)
      __builtin_amdgcn_sched_barrier(0);
      const uint32_t sv = cs.sring[r];
      uint32_t sel[8];
      selectors<BITS>(cs.ring[r], sel);
      // refill the ring slot once its codes are in the selectors
      const bool wrap = s + RING >= CPW;
      cs.load(r, wrap ? cs.chunk(pn, s + RING - CPW) : cs.chunk(p, s + RING));
      half2_t s_lo, s_hi;
      if (MODE == 1) {
        const half2_t sc2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sv, 1.0f, false);
        s_lo = half2_t{sc2[0], sc2[0]};
        s_hi = half2_t{sc2[1], sc2[1]};
      }
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        uint32_t a0, a1, a2, a3;
        lookup4(sel[2 * st], tl0, tl1, th0, th1, a0, a1);
        lookup4(sel[2 * st + 1], tl0, tl1, th0, th1, a2, a3);
        half8_t af = as_half8(a0, a1, a2, a3);
        if (MODE == 1) af = scale_half8(af, st < 2 ? s_lo : s_hi);
        pacc[st] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, bf[st], pacc[st], 0, 0, 0);
      }
#pragma unroll
      for (int st = 0; st < 4; ++st) bf[st] = bn[st];
    }
  }
}

// fp16 rescale exponent of a batch row whose maximum magnitude has bits mb:
// the maximum lands in [2^14, 2^15)
__device__ inline int stage_exponent(uint32_t mb) {
  return mb ? min(126, 14 - ((int)((mb >> 23) & 0xFF) - 127)) : 0;
}

__device__ inline half8_t to_half8_scaled(const uint4_t& raw, float sc) {
  half8_t h;
#pragma unroll
  for (int w4 = 0; w4 < 4; ++w4) {
    h[2 * w4] = (_Float16)(bf16_lo(raw[w4]) * sc);
    h[2 * w4 + 1] = (_Float16)(bf16_hi(raw[w4]) * sc);
  }
  return h;
}

__device__ inline float max_abs8(const uint4_t& raw) {
  float m = 0.0f;
#pragma unroll
  for (int w4 = 0; w4 < 4; ++w4) m = fmaxf(m, fmaxf(fabsf(bf16_lo(raw[w4])), fabsf(bf16_hi(raw[w4]))));
  return m;
}

// maximum over the 16-lane group (all 64 lanes must be active)
__device__ inline float group16_max(float m) {
  m = fmaxf(m, __shfl_xor(m, 1, 64));
  m = fmaxf(m, __shfl_xor(m, 2, 64));
  m = fmaxf(m, __shfl_xor(m, 4, 64));
  m = fmaxf(m, __shfl_xor(m, 8, 64));
  return m;
}

// maximum over the wavefront (all 64 lanes must be active)
__device__ inline float wave_max(float m) {
  m = group16_max(m);
  m = fmaxf(m, __shfl_xor(m, 16, 64));
  return fmaxf(m, __shfl_xor(m, 32, 64));
}

// Reduce the KS partial sums of each row tile in a fixed order and store
// (lane: batch column j = lane % 16, rows 4q..4q+3 of the tile).
__device__ inline void reduce_store(float4_t acc, float4_t* red, int wave, int lane, int ks, int KS, bool tile_ok,
                                    int64_t tile, int64_t N, int out_kind, void* __restrict__ y, bool xlane) {
  if (KS > 1) {
    red[wave * 64 + lane] = acc;
    __syncthreads();
  }
  if (ks == 0 && tile_ok && xlane) {
    for (int k2 = 1; k2 < KS; ++k2) {
      const float4_t o = red[(wave + k2) * 64 + lane];
      acc[0] += o[0];
      acc[1] += o[1];
      acc[2] += o[2];
      acc[3] += o[3];
    }
    const int q = lane >> 4, j = lane & 15;
#pragma unroll
    for (int r2 = 0; r2 < 4; ++r2) {
      const int64_t row = tile * 16 + 4 * q + r2;
      if (row < N) {
        const int64_t o = (int64_t)j * N + row;
        if (out_kind == 0)
          reinterpret_cast<float*>(y)[o] = acc[r2];
        else
          reinterpret_cast<uint16_t*>(y)[o] = (uint16_t)f32_to_bf16_rne(acc[r2]);
      }
    }
  }
}


// ---------------------------------------------------------------- persistent
// Resident workgroups that loop over row tiles (used whenever the staged
// activations fit in LDS).  Workgroup g owns the R consecutive row tiles
// g*R .. g*R + R - 1 ("rounds"; the last workgroup may have fewer); its W
// wavefronts split every tile's K: wavefront w consumes
// chunks w, w + W, ... of the tile (CPW = ceil(KC / W) slots per round).
// Each activation chunk is consumed by exactly one wavefront, which stages it
// itself: it loads its own raw bf16 chunks straight into LDS, rescales them by
// a power of two taken from their own maximum (so the fp16 copy is exact for
// every value within 2^31 of that maximum) and converts them in place; its
// partial sums are unscaled before the reduction.  Each wavefront also copies
// the tables of its rounds into a private LDS slot.  Nothing is shared before
// the reduction, so wavefronts start streaming without a barrier; the code
// stream is one ring across all rounds.  Partial sums are parked per round
// and wavefront in LDS; after the single barrier, wavefront r mod W adds the
// W partials of round r in a fixed order and stores the tile (deterministic).
struct PersistPlan {
  int CPW, rounds;
  int64_t tiles, KC;
};

// maximum over the 64 lanes (all active) via DPP and lane reads: uniform
__device__ inline float wave_max_dpp(float v) {
  int b = __float_as_int(v);
  b = __float_as_int(fmaxf(__int_as_float(b), __int_as_float(__builtin_amdgcn_mov_dpp(b, 0xB1, 0xF, 0xF, false))));
  b = __float_as_int(fmaxf(__int_as_float(b), __int_as_float(__builtin_amdgcn_mov_dpp(b, 0x4E, 0xF, 0xF, false))));
  b = __float_as_int(fmaxf(__int_as_float(b), __int_as_float(__builtin_amdgcn_mov_dpp(b, 0x141, 0xF, 0xF, false))));
  b = __float_as_int(fmaxf(__int_as_float(b), __int_as_float(__builtin_amdgcn_mov_dpp(b, 0x140, 0xF, 0xF, false))));
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(b, 0)), r1 = __int_as_float(__builtin_amdgcn_readlane(b, 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(b, 32)), r3 = __int_as_float(__builtin_amdgcn_readlane(b, 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

template <int BITS, int MODE, int RING, int XREG, int TI>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(6)))
void lut_gemv_persist_kernel(const uint16_t* __restrict__ x, int B, int64_t K, const uint8_t* __restrict__ codes,
                             const uint16_t* __restrict__ lut, const uint8_t* __restrict__ scales,
                             const float* __restrict__ Gp, int64_t N, PersistPlan plan, int out_kind,
                             void* __restrict__ y) {
  // Issue arbitration favours older wavefronts: without help the youngest
  // wavefront of every SIMD stages late and finishes last.  Staging runs at
  // the top priority, and in the slot loop the priority falls with progress
  // (3, 2, 1, 0 by quarters), so lagging wavefronts catch up.
  __builtin_amdgcn_s_setprio(3);
  typedef typename CodeVec<BITS>::type cvec;
  constexpr int kChunkBytes = 64 * CodeVec<BITS>::bytes;
  constexpr int kTabBytes = 16 * 2 * (1 << BITS);     // one row tile's tables
  extern __shared__ __align__(16) uint8_t smem[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int W = blockDim.x >> 6;
  const int KCi = (int)plan.KC, CPW = plan.CPW, R = plan.rounds;
  const int T = (int)plan.tiles;
  const int t0 = (int)blockIdx.x * R;              // this workgroup's tiles: t0 .. t0 + nr - 1
  const int nr = min(R, T - t0);                   // rounds of this workgroup (1 <= nr <= R)
  const int rowstride = (KCi + 1) * 128 + 8;       // fp16 per staged batch row (+ zero chunk, pad)
  // LDS: staged activations | partial sums [R][W][64] float4 | tables [W][TI KiB] (PER_ROW)
  _Float16* xs = reinterpret_cast<_Float16*>(smem);
  float4_t* part = reinterpret_cast<float4_t*>(smem + (size_t)B * rowstride * 2);
  uint8_t* tabs = reinterpret_cast<uint8_t*>(part + (size_t)R * W * 64) + (size_t)wave * TI * 1024;
  const int i = lane & 15, j = lane & 15, q = lane >> 4;
  auto tile_of = [&](int r) { return t0 + r; };

  // ---- 1. this wavefront's activation chunks (lane l: elements 2l, 2l+1 of
  // each chunk), and the tables of its rounds.  Batch 1 with at most XREG
  // chunks per wavefront: into registers through a range-checked buffer
  // resource (reads past K return zero).  Otherwise raw into LDS, with reads
  // past K clamped in bounds and zeroed at conversion.
  const int nxc = (KCi - wave + W - 1) / W;        // chunks of this wavefront
  constexpr bool xreg = XREG > 0;   // the host guarantees B == 1 and nxc <= XREG
  uint32_t xr[XREG > 0 ? XREG : 1];
  if constexpr (xreg) {
    const i32x4_t rx = buffer_resource(x, (uint32_t)(K * 2));
#pragma unroll
    for (int u = 0; u < (XREG > 0 ? XREG : 1); ++u)
      xr[u] = (uint32_t)raw_buffer_load_b32(rx, lane * 4 + ((u * W + wave) * 128) * 2, 0, 0);
  } else {
    for (int jj = 0; jj < B; ++jj)
      for (int c = wave; c < KCi; c += W) {
        const int64_t k = min((int64_t)c * 128 + 2 * lane, K - 2);
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(x + (int64_t)jj * K + k),
                                         reinterpret_cast<void*>(xs + jj * rowstride + c * 128), 4, 0, 0);
      }
  }
  if (MODE == 0) {
    // the tables of tiles t0 .. are contiguous: TI KiB per wavefront (a fixed
    // count of loads, so that the compiler's load counting stays exact);
    // reads past the table array return zero
    const __amdgpu_buffer_rsrc_t rl = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(lut), 0, (int)((int64_t)T * kTabBytes), 0x00020000);
#pragma unroll
    for (int ti = 0; ti < TI; ++ti)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, (__attribute__((address_space(3))) void*)(tabs + ti * 1024), 16,
                                               lane * 16 + t0 * kTabBytes + ti * 1024, 0, 0, 0);
  }
  uint4_t grid_tab{0u, 0u, 0u, 0u};
  if (MODE == 1) grid_tab = load_table<BITS>(lut);

  // ---- 2. the first RING code loads (and block-scale pairs).  Slot cursor
  // (round r, step s) -> chunk s*W + wave of tile g + r*G; past the last slot
  // the cursor stays on it (harmless re-reads keep the ring unconditional)
  const i32x4_t rcodes = buffer_resource(codes, (uint32_t)T * (uint32_t)KCi * kChunkBytes);
  i32x4_t rscales{};
  if (MODE == 1) rscales = buffer_resource(scales, (uint32_t)T * (uint32_t)KCi * 128);
  const int32_t lane_code = lane * CodeVec<BITS>::bytes, lane_scale = lane * 2;
  cvec ring[RING];
  uint32_t sring[RING];
  int lr = 0, ls = 0;   // load cursor
  auto load_next = [&](int slot) {
    const int cidx = tile_of(lr) * KCi + min(ls * W + wave, KCi - 1);
    if constexpr (BITS == 3) {
      const i32x3_t v = raw_buffer_load_b96(rcodes, lane_code, cidx * kChunkBytes, 0);
      ring[slot] = cvec{{(uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2]}};
    } else {
      const i32x2_t v = raw_buffer_load_b64(rcodes, lane_code, cidx * kChunkBytes, 0);
      ring[slot] = cvec{{(uint32_t)v[0], (uint32_t)v[1]}};
    }
    if (MODE == 1) sring[slot] = (uint16_t)raw_buffer_load_b16(rscales, lane_scale, cidx * 128, 0);
    if (++ls == CPW) {
      ls = 0;
      ++lr;
    }
    if (lr == nr) {   // stay on the last slot
      lr = nr - 1;
      ls = CPW - 1;
    }
  };
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int r = 0; r < RING; ++r) load_next(r);
  __builtin_amdgcn_sched_barrier(0);
  // the zero chunk of every staged row (each wavefront writes the same zeros)
  for (int jj = 0; jj < B; ++jj) reinterpret_cast<uint32_t*>(xs + jj * rowstride + KCi * 128)[lane] = 0u;

  // ---- 3. once its own loads have landed (vmcnt: the code loads may still
  // be in flight), the wavefront rescales and converts its chunks in place
  {
    constexpr int kv = RING * (MODE == 1 ? 2 : 1) + (MODE == 0 ? TI : 1);
    __builtin_amdgcn_s_waitcnt((kv & 0xF) | ((kv >> 4) << 14) | (0x7 << 4) | (0xF << 8));
  }
  __builtin_amdgcn_sched_barrier(0);
  float unscale = 1.0f;
  // the scaled values are exact in fp16 down to 2^-17 (at most 2^32 below the
  // maximum, which lands in [2^14, 2^15)); smaller ones become fp16 subnormals,
  // truncated toward zero by the conversion (an error below 2^-24, i.e. 2^-38
  // of the maximum)
  auto to_h2 = [](uint32_t v, float sc) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(bf16_lo(v) * sc, bf16_hi(v) * sc));
  };
  if constexpr (xreg) {
    float m = 0.0f;
#pragma unroll
    for (int u = 0; u < (XREG > 0 ? XREG : 1); ++u)
      if (u < nxc) m = fmaxf(m, fmaxf(fabsf(bf16_lo(xr[u])), fabsf(bf16_hi(xr[u]))));
    const int e = stage_exponent(__float_as_uint(wave_max_dpp(m)));
    const float sc = __builtin_ldexpf(1.0f, e);
    unscale = __builtin_ldexpf(1.0f, -e);
    uint32_t* row = reinterpret_cast<uint32_t*>(xs) + lane;
#pragma unroll
    for (int u = 0; u < (XREG > 0 ? XREG : 1); ++u)
      if (u < nxc) row[(u * W + wave) * 64] = to_h2(xr[u], sc);
  } else {
    // batches of 8 chunks, so that the LDS round trips overlap
    for (int jj = 0; jj < B; ++jj) {
      uint32_t* row = reinterpret_cast<uint32_t*>(xs + jj * rowstride) + lane;
      float m = 0.0f;
      for (int t0 = 0; t0 < nxc; t0 += 8) {
        uint32_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = t0 + u < nxc ? row[((t0 + u) * W + wave) * 64] : 0u;
#pragma unroll
        for (int u = 0; u < 8; ++u) m = fmaxf(m, fmaxf(fabsf(bf16_lo(v[u])), fabsf(bf16_hi(v[u]))));
      }
      const int e = stage_exponent(__float_as_uint(wave_max_dpp(m)));
      const float sc = __builtin_ldexpf(1.0f, e);
      if (j == jj) unscale = __builtin_ldexpf(1.0f, -e);
      for (int t0 = 0; t0 < nxc; t0 += 8) {
        uint32_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = t0 + u < nxc ? row[((t0 + u) * W + wave) * 64] : 0u;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int c = (t0 + u) * W + wave;
          if (t0 + u < nxc) row[c * 64] = (int64_t)c * 128 + 2 * lane < K ? to_h2(v[u], sc) : 0u;
        }
      }
    }
  }
  const bool xlane = j < B;
  if (MODE == 1) unscale *= *Gp;
  auto round_table = [&](int r) {
    if (MODE == 1) return grid_tab;
    const uint8_t* t = tabs + r * kTabBytes + i * 2 * (1 << BITS);   // r < TI KiB / kTabBytes
    if (BITS == 3) return *reinterpret_cast<const uint4_t*>(t);
    const uint2_t d = *reinterpret_cast<const uint2_t*>(t);
    return uint4_t{d[0], d[1], 0u, 0u};
  };

  // ---- 4. slots: RING loads in flight across rounds.  The table copies
  // were issued just before the ring: wait for them (the compiler does not
  // track loads into LDS); later rounds' tables have landed by the time the
  // round's first ring slot has
  if (MODE == 0) {
    __builtin_amdgcn_s_waitcnt((RING & 0xF) | ((RING >> 4) << 14) | (0x7 << 4) | (0xF << 8));
    __builtin_amdgcn_sched_barrier(0);
  }
  uint32_t tl0, tl1, th0, th1;
  table_pools<BITS>(round_table(0), tl0, tl1, th0, th1);
  float4_t pacc[4];
#pragma unroll
  for (int st = 0; st < 4; ++st) pacc[st] = float4_t{0.f, 0.f, 0.f, 0.f};
  // batch columns >= B read row 0: their MFMA output columns are never stored
  const _Float16* xrow = xs + (xlane ? j : 0) * rowstride + 32 * q;
  const int total = nr * CPW;
  int rd = 0, s = 0;   // consume cursor
  // slot r of the ring (r is a compile-time index once inlined)
  auto slot = [&](const int r) __attribute__((always_inline)) {
      const int c = s * W + wave;
      const int xc = (rd < nr && c < KCi) ? c : KCi;   // past the end: the zero chunk
      half8_t bf[4];
      const half8_t* xp = reinterpret_cast<const half8_t*>(xrow + xc * 128);
#pragma unroll
      for (int st = 0; st < 4; ++st) bf[st] = xp[st];
      const uint32_t sv = sring[r];
      uint32_t sel[8];
      selectors<BITS>(ring[r], sel);
      load_next(r);
      half2_t s_lo, s_hi;
      if (MODE == 1) {
        const half2_t sc2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sv, 1.0f, false);
        s_lo = half2_t{sc2[0], sc2[0]};
        s_hi = half2_t{sc2[1], sc2[1]};
      }
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        uint32_t a0, a1, a2, a3;
        lookup4(sel[2 * st], tl0, tl1, th0, th1, a0, a1);
        lookup4(sel[2 * st + 1], tl0, tl1, th0, th1, a2, a3);
        half8_t af = as_half8(a0, a1, a2, a3);
        if (MODE == 1) af = scale_half8(af, st < 2 ? s_lo : s_hi);
        pacc[st] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, bf[st], pacc[st], 0, 0, 0);
      }
      if (__builtin_expect(++s == CPW, 0)) {   // end of a round: rare
        s = 0;
        if (rd < nr) {   // end of round rd: park the partial sums
          float4_t acc;
#pragma unroll
          for (int r2 = 0; r2 < 4; ++r2)
            acc[r2] = ((pacc[0][r2] + pacc[1][r2]) + (pacc[2][r2] + pacc[3][r2])) * unscale;
#pragma unroll
          for (int st = 0; st < 4; ++st) pacc[st] = float4_t{0.f, 0.f, 0.f, 0.f};
          part[((size_t)rd * W + wave) * 64 + lane] = acc;
          if (rd + 1 < nr) table_pools<BITS>(round_table(rd + 1), tl0, tl1, th0, th1);
        }
        ++rd;
      }
  };
  // whole ring cycles without exits (an exit would make the compiler wait
  // for every load at the top of each cycle), then the remaining slots
  const int full = total / RING * RING;
  const int q1 = total / 4, q2 = total / 2, q3 = (3 * total) / 4;
  // one loop per priority level (s_setprio takes an immediate), so that the
  // cycles carry no branches for it
  int f0 = 0;
  for (; f0 < full && f0 < q1; f0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) slot(r);
  }
  __builtin_amdgcn_s_setprio(2);
  for (; f0 < full && f0 < q2; f0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) slot(r);
  }
  __builtin_amdgcn_s_setprio(1);
  for (; f0 < full && f0 < q3; f0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) slot(r);
  }
  __builtin_amdgcn_s_setprio(0);
  for (; f0 < full; f0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) slot(r);
  }
#pragma unroll
  for (int r = 0; r < RING - 1; ++r)
    if (full + r < total) slot(r);
  // ---- 5. reduce each round's W partials in order and store the tile
  __syncthreads();
  for (int r = wave; r < nr; r += W) {
    if (!xlane) continue;
    const float4_t* pr = part + (size_t)r * W * 64 + lane;
    float4_t o = pr[0];
    for (int w2 = 1; w2 < W; ++w2) {
      const float4_t t2 = pr[w2 * 64];
      o[0] += t2[0];
      o[1] += t2[1];
      o[2] += t2[2];
      o[3] += t2[3];
    }
    const int64_t tile = tile_of(r);
#pragma unroll
    for (int r2 = 0; r2 < 4; ++r2) {
      const int64_t row = tile * 16 + 4 * q + r2;
      if (row < N) {
        const int64_t o2 = (int64_t)j * N + row;
        if (out_kind == 0)
          reinterpret_cast<float*>(y)[o2] = o[r2];
        else
          reinterpret_cast<uint16_t*>(y)[o2] = (uint16_t)f32_to_bf16_rne(o[r2]);
      }
    }
  }
}

constexpr int kRingMulti = 8;

// ---------------------------------------------------------------- batched
// Batch B >= 2.  Each workgroup takes K group kg (KCR chunks) of a group of
// W * TPW row tiles.  It copies the bf16 slice of x (all B rows) into LDS,
// one wavefront per batch row rescales the row's slice by a power of two
// from the slice's own maximum and converts it to fp16 in place (exact for
// every value within 2^31 of that maximum), and each wavefront then owns TPW
// whole tiles over the K group: its code stream is contiguous per tile and
// it reduces nothing with other wavefronts.  The tile sums are unscaled per
// batch row.  With one K group they are y; otherwise they go to a per-K-group
// partial buffer that a reduction pass adds up in K-group order (results are
// deterministic).  A hand-off between workgroups inside the kernel would
// need a device-scope release per workgroup, which on this architecture
// writes back the XCD's whole L2.
struct SplitPlan {
  int KG, TPW, KCR;   // K groups, tiles per wavefront, chunks per K group
  int tiles, KC;
};

template <int BITS, int MODE, int RING, int TI>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(6)))
void lut_gemv_split_kernel(const uint16_t* __restrict__ x, int64_t K, int B, const uint8_t* __restrict__ codes, const uint16_t* __restrict__ lut,
                           const uint8_t* __restrict__ scales, const float* __restrict__ Gp, int64_t N,
                           SplitPlan plan, float* __restrict__ partials, int out_kind, void* __restrict__ y) {
  __builtin_amdgcn_s_setprio(3);
  typedef typename CodeVec<BITS>::type cvec;
  constexpr int kChunkBytes = 64 * CodeVec<BITS>::bytes;
  constexpr int kTabBytes = 16 * 2 * (1 << BITS);
  extern __shared__ __align__(16) uint8_t smem[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int W = blockDim.x >> 6;
  const int KG = plan.KG, TPW = plan.TPW, KCR = plan.KCR, KC = plan.KC, T = plan.tiles;
  const int kg = (int)blockIdx.x % KG, tg = (int)blockIdx.x / KG;
  const int tw = (tg * W + wave) * TPW;                    // this wavefront's first tile
  const int ntw = max(0, min(TPW, T - tw));                 // and its tile count
  const int c0 = kg * KCR, nc = min(KCR, KC - c0);         // the K group's chunks
  const int rowstride = nc * 128 + 8;                       // fp16 per staged batch row (pad staggers banks)
  // LDS: activations [B][rowstride] | tables [W][TI KiB]; static: unscale
  // factors and grid, copied by wavefront 0.  Tile sums go straight from the
  // accumulators to y or to the K group's partials, so LDS holds only what
  // the streaming reads and more workgroups fit on a compute unit.
  __shared__ __align__(16) uint32_t s_small[32];
  _Float16* xs = reinterpret_cast<_Float16*>(smem);
  uint8_t* tabs = smem + round_up((int64_t)B * rowstride * 2, 16) + (size_t)wave * TI * 1024;
  const int i = lane & 15, j = lane & 15, q = lane >> 4;
  const bool xlane = j < B;

  // ---- 1. the K group's slice of the raw bf16 activations, four chunks of
  // a row per 16-byte-per-lane copy (spread over the wavefronts; lanes past
  // the slice row stay idle, reads past K are clamped in bounds and zeroed at
  // conversion) and this wavefront's tables
  {
    const int nq = (nc + 3) / 4;
    for (int t = wave; t < B * nq; t += W) {
      const int b = t / nq, u = 4 * (t - b * nq);
      const int64_t k = min((int64_t)(c0 + u) * 128 + 8 * lane, K - 8);   // K % 32 == 0
      if (lane < (nc - u) * 16)
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(x + (int64_t)b * K + k),
                                         reinterpret_cast<void*>(xs + b * rowstride + u * 128), 16, 0, 0);
    }
  }
  if (MODE == 0) {   // tables of tiles tw .. tw + TPW - 1 (contiguous); reads past the array return zero
    const __amdgpu_buffer_rsrc_t rl = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(lut), 0, (int)((int64_t)T * kTabBytes), 0x00020000);
#pragma unroll
    for (int ti = 0; ti < TI; ++ti)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, (__attribute__((address_space(3))) void*)(tabs + ti * 1024), 16,
                                               lane * 16 + tw * kTabBytes + ti * 1024, 0, 0, 0);
  }
  // the grid into LDS as well: with only the ring's loads tracked by the
  // compiler, its waits in the loop stay exact
  if (MODE == 1 && wave == 0 && lane < (1 << BITS) / 2)
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(lut + 2 * lane),
                                     reinterpret_cast<void*>(s_small + 16), 4, 0, 0);

  // ---- 2. the code ring: slot (tile i, chunk u) -> chunk c0 + u of tile tw + i;
  // past the last slot the cursor stays on it
  const i32x4_t rcodes = buffer_resource(codes, (uint32_t)T * (uint32_t)KC * kChunkBytes);
  i32x4_t rscales{};
  if (MODE == 1) rscales = buffer_resource(scales, (uint32_t)T * (uint32_t)KC * 128);
  const int32_t lane_code = lane * CodeVec<BITS>::bytes, lane_scale = lane * 2;
  cvec ring[RING];
  uint32_t sring[RING];
  const int last = max(ntw, 1) - 1;   // a wavefront without tiles re-reads tile tw's range: in bounds
  const int twc = min(tw, T - 1);
  int li = 0, lu = 0;
  auto load_next = [&](int slot) {
    const int cidx = (twc + min(li, last)) * KC + c0 + lu;
    if constexpr (BITS == 3) {
      const i32x3_t v = raw_buffer_load_b96(rcodes, lane_code, cidx * kChunkBytes, 0);
      ring[slot] = cvec{{(uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2]}};
    } else {
      const i32x2_t v = raw_buffer_load_b64(rcodes, lane_code, cidx * kChunkBytes, 0);
      ring[slot] = cvec{{(uint32_t)v[0], (uint32_t)v[1]}};
    }
    if (MODE == 1) sring[slot] = (uint16_t)raw_buffer_load_b16(rscales, lane_scale, cidx * 128, 0);
    if (++lu == nc) {
      lu = 0;
      ++li;
    }
    if (li == ntw) {
      li = max(ntw, 1) - 1;
      lu = nc - 1;
    }
  };
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int r = 0; r < RING; ++r) load_next(r);
  __builtin_amdgcn_sched_barrier(0);
  // the slice and table copies were issued before the ring: wait for them
  // (the compiler does not track loads into LDS), then make every
  // wavefront's part of the slice visible (LDS-only barrier)
  {
    constexpr int kv = RING * (MODE == 1 ? 2 : 1);
    __builtin_amdgcn_s_waitcnt((kv & 0xF) | ((kv >> 4) << 14) | (0x7 << 4) | (0xF << 8));
  }
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  // ---- 2b. per batch row, the slice's maximum, then fp16 in place; the
  // row's unscale factor into LDS.  A row takes one wavefront (B <= W) or
  // half of one (B > W: rows wave and wave + W side by side), its lanes
  // striding over the row's dwords with eight reads in flight per round trip
  auto to_h2 = [](uint32_t v, float sc) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(bf16_lo(v) * sc, bf16_hi(v) * sc));
  };
  {
    const bool half = B > W;
    const int tpr = half ? 32 : 64;                        // lanes per row
    const int lr = half ? (lane & 31) : lane;
    const int b = wave + (half ? W * (lane >> 5) : 0);
    const bool live = b < B;                                // rows past B: reads only, of row 0
    uint32_t* row = reinterpret_cast<uint32_t*>(xs + (live ? b : 0) * rowstride);
    const int nd = nc * 64;   // dwords of the slice row
    float m = 0.0f;
    for (int d0 = lr; d0 < nd; d0 += 8 * tpr) {
      uint32_t v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = d0 + u * tpr < nd ? row[d0 + u * tpr] : 0u;
#pragma unroll
      for (int u = 0; u < 8; ++u) m = fmaxf(m, fmaxf(fabsf(bf16_lo(v[u])), fabsf(bf16_hi(v[u]))));
    }
    m = fmaxf(m, __shfl_xor(m, 1, 64));
    m = fmaxf(m, __shfl_xor(m, 2, 64));
    m = fmaxf(m, __shfl_xor(m, 4, 64));
    m = fmaxf(m, __shfl_xor(m, 8, 64));
    m = fmaxf(m, __shfl_xor(m, 16, 64));
    if (!half) m = fmaxf(m, __shfl_xor(m, 32, 64));
    const int e = stage_exponent(__float_as_uint(m));
    const float sc = __builtin_ldexpf(1.0f, e);
    if (live) {
      for (int d0 = lr; d0 < nd; d0 += 8 * tpr) {
        uint32_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = d0 + u * tpr < nd ? row[d0 + u * tpr] : 0u;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int d = d0 + u * tpr;
          if (d < nd) row[d] = (int64_t)c0 * 128 + 2 * d < K ? to_h2(v[u], sc) : 0u;
        }
      }
      if (lr == 0) s_small[b] = __float_as_uint(__builtin_ldexpf(1.0f, -e));
    }
  }
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  float unscale = xlane ? __uint_as_float(s_small[j]) : 1.0f;
  if (MODE == 1) unscale *= *Gp;
  uint4_t grid_tab{0u, 0u, 0u, 0u};
  if (MODE == 1) {
    if (BITS == 3)
      grid_tab = *reinterpret_cast<const uint4_t*>(s_small + 16);
    else
      grid_tab = uint4_t{s_small[16], s_small[17], 0u, 0u};
  }
  auto tile_table = [&](int t) {
    if (MODE == 1) return grid_tab;
    const uint8_t* tp = tabs + t * kTabBytes + i * 2 * (1 << BITS);   // t < TI KiB / kTabBytes
    if (BITS == 3) return *reinterpret_cast<const uint4_t*>(tp);
    const uint2_t d = *reinterpret_cast<const uint2_t*>(tp);
    return uint4_t{d[0], d[1], 0u, 0u};
  };

  // ---- 3. slots
  uint32_t tl0, tl1, th0, th1;
  table_pools<BITS>(tile_table(0), tl0, tl1, th0, th1);
  float4_t pacc[4];
#pragma unroll
  for (int st = 0; st < 4; ++st) pacc[st] = float4_t{0.f, 0.f, 0.f, 0.f};
  const _Float16* xrow = xs + (xlane ? j : 0) * rowstride + 32 * q;
  // read the slice once before the loop: the compiler then settles its wait
  // for the copies into LDS here, not at the top of every ring cycle
  {
    const uint32_t probe = *reinterpret_cast<const uint32_t*>(xrow);
    asm volatile("" ::"v"(probe));
  }
  const int total = ntw * nc;
  int ti_ = 0, u = 0;
  auto slot = [&](const int r) __attribute__((always_inline)) {
      half8_t bf[4];
      const half8_t* xp = reinterpret_cast<const half8_t*>(xrow + u * 128);
#pragma unroll
      for (int st = 0; st < 4; ++st) bf[st] = xp[st];
      const uint32_t sv = sring[r];
      uint32_t sel[8];
      selectors<BITS>(ring[r], sel);
      load_next(r);
      half2_t s_lo, s_hi;
      if (MODE == 1) {
        const half2_t sc2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sv, 1.0f, false);
        s_lo = half2_t{sc2[0], sc2[0]};
        s_hi = half2_t{sc2[1], sc2[1]};
      }
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        uint32_t a0, a1, a2, a3;
        lookup4(sel[2 * st], tl0, tl1, th0, th1, a0, a1);
        lookup4(sel[2 * st + 1], tl0, tl1, th0, th1, a2, a3);
        half8_t af = as_half8(a0, a1, a2, a3);
        if (MODE == 1) af = scale_half8(af, st < 2 ? s_lo : s_hi);
        pacc[st] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, bf[st], pacc[st], 0, 0, 0);
      }
      if (__builtin_expect(++u == nc, 0)) {   // end of tile ti_: lane (q, j) stores rows 4q..4q+3 of batch row j
        u = 0;
        float4_t acc;
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2)
          acc[r2] = ((pacc[0][r2] + pacc[1][r2]) + (pacc[2][r2] + pacc[3][r2])) * unscale;
#pragma unroll
        for (int st = 0; st < 4; ++st) pacc[st] = float4_t{0.f, 0.f, 0.f, 0.f};
        if (xlane) {
          const int64_t tile = tw + ti_;
          if (KG == 1) {
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2) {
              const int64_t row = tile * 16 + 4 * q + r2;
              if (row < N) {
                const int64_t o2 = (int64_t)j * N + row;
                if (out_kind == 0)
                  reinterpret_cast<float*>(y)[o2] = acc[r2];
                else
                  reinterpret_cast<uint16_t*>(y)[o2] = (uint16_t)f32_to_bf16_rne(acc[r2]);
              }
            }
          } else {
            *reinterpret_cast<float4_t*>(partials + (((int64_t)kg * T + tile) * B + j) * 16 + 4 * q) = acc;
          }
        }
        ++ti_;
        if (ti_ < ntw) table_pools<BITS>(tile_table(ti_), tl0, tl1, th0, th1);
      }
  };
  // whole ring cycles without exits, then the remaining slots (see the
  // batch-1 kernel); wave priority falls with progress
  const int full = total / RING * RING;
  const int q1 = total / 4, q2 = total / 2, q3 = (3 * total) / 4;
  // one loop per priority level (s_setprio takes an immediate), so that the
  // cycles carry no branches for it
  int f0 = 0;
  for (; f0 < full && f0 < q1; f0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) slot(r);
  }
  __builtin_amdgcn_s_setprio(2);
  for (; f0 < full && f0 < q2; f0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) slot(r);
  }
  __builtin_amdgcn_s_setprio(1);
  for (; f0 < full && f0 < q3; f0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) slot(r);
  }
  __builtin_amdgcn_s_setprio(0);
  for (; f0 < full; f0 += RING) {
#pragma unroll
    for (int r = 0; r < RING; ++r) slot(r);
  }
#pragma unroll
  for (int r = 0; r < RING - 1; ++r)
    if (full + r < total) slot(r);
}

// y[jj][row] = sum over the K groups, in order, of the split kernel's
// partials [KG][T][B][16]
__global__ __launch_bounds__(256) void reduce_partials_kernel(const float* __restrict__ partials, int KG, int T, int B,
                                                              int64_t N, int out_kind, void* __restrict__ y) {
  const int total = T * B * 16;
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x) {
    const int tile = t / (B * 16);
    const int rem = t - tile * B * 16, jj = rem >> 4, row16 = rem & 15;
    const int64_t row = (int64_t)tile * 16 + row16;
    if (row >= N) continue;
    // K groups summed in order; four loads in flight per step
    float v = 0.0f;
    int g = 0;
    for (; g + 4 <= KG; g += 4) {
      const float a0 = partials[(int64_t)g * total + t], a1 = partials[(int64_t)(g + 1) * total + t];
      const float a2 = partials[(int64_t)(g + 2) * total + t], a3 = partials[(int64_t)(g + 3) * total + t];
      v += a0;
      v += a1;
      v += a2;
      v += a3;
    }
    for (; g < KG; ++g) v += partials[(int64_t)g * total + t];
    const int64_t o = (int64_t)jj * N + row;
    if (out_kind == 0)
      reinterpret_cast<float*>(y)[o] = v;
    else
      reinterpret_cast<uint16_t*>(y)[o] = (uint16_t)f32_to_bf16_rne(v);
  }
}

// ---------------------------------------------------------------- several pieces
template <int BITS, int MODE>
__global__ __launch_bounds__(768) void lut_gemv_multi_kernel(const uint16_t* __restrict__ x, int B, int64_t K,
                                                             const uint8_t* __restrict__ codes,
                                                             const uint16_t* __restrict__ lut,
                                                             const uint8_t* __restrict__ scales,
                                                             const float* __restrict__ Gp, int64_t N,
                                                             GemvPlan plan, int out_kind, void* __restrict__ y) {
  constexpr int RING = kRingMulti;
  extern __shared__ __align__(16) uint8_t smem[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nthreads = blockDim.x;
  const int KS = plan.KS, rt = wave / KS, ks = wave % KS;
  const int64_t tile = (int64_t)blockIdx.x * plan.RT + rt;
  const bool tile_ok = tile < plan.tiles;
  const int64_t tile_c = tile_ok ? tile : plan.tiles - 1;
  const int PK = plan.PK, NP = plan.npieces;
  const int vpr = PK * 16;                         // 8-element vectors per staged piece row
  const int rowstride = (PK + 1) * 128 + 8;        // fp16 elements per staged batch row (+ zero chunk, pad)
  _Float16* xs = reinterpret_cast<_Float16*>(smem);
  float4_t* red = reinterpret_cast<float4_t*>(smem + (size_t)B * rowstride * 2);
  __shared__ uint32_t piece_max[2][16];            // double-buffered per-piece batch-row maxima

  // Staging assignment, fixed for the kernel: vector n of this thread is
  // elements [8*spos, 8*spos + 8) of batch row sj of every piece (valid when
  // sj < B); ((f + 0.5) / vpr in fp32 truncates to the exact quotient for
  // these small operands).
  int sj[kStageVec], spos[kStageVec];
  {
    const float rvpr = 1.0f / (float)vpr;
#pragma unroll
    for (int n = 0; n < kStageVec; ++n) {
      const int f = n * nthreads + (int)threadIdx.x;
      sj[n] = (int)(((float)f + 0.5f) * rvpr);
      spos[n] = f - sj[n] * vpr;
    }
  }
  uint4_t v[kStageVec];
  auto load_piece_x = [&](int p) {
    const int64_t k0 = (int64_t)p * PK * 128;
#pragma unroll
    for (int n = 0; n < kStageVec; ++n) {
      const bool ok = sj[n] < B;
      int64_t k = k0 + (int64_t)spos[n] * 8;
      const bool in_k = ok && k < K;
      k = in_k ? k : 0;
      const uint4_t t = *reinterpret_cast<const uint4_t*>(x + (int64_t)(ok ? sj[n] : 0) * K + k);   // in bounds
      v[n] = in_k ? t : uint4_t{0u, 0u, 0u, 0u};
    }
  };
  if ((int)threadIdx.x < 16) {
    piece_max[0][threadIdx.x] = 0u;
    piece_max[1][threadIdx.x] = 0u;
  }
  for (int t = threadIdx.x; t < B * 16; t += nthreads)   // zero chunk of every staged row
    reinterpret_cast<uint4_t*>(xs + (t >> 4) * rowstride + PK * 128)[t & 15] = uint4_t{0u, 0u, 0u, 0u};

  // ---- 1. lookup table, the first activation piece and this workgroup's
  // share of the L2 warm-up of the whole activation matrix (workgroup b runs
  // on XCD b % 8)
  const int i = lane & 15, q = lane >> 4, j = lane & 15;
  uint4_t tab{0u, 0u, 0u, 0u};
  if (tile_ok) tab = load_table<BITS>(MODE == 0 ? lut + (tile * 16 + i) * (1 << BITS) : lut);
  load_piece_x(0);
  uint32_t warm = 0;
  {
    const uint32_t V = (uint32_t)(B * K / 8);      // 16-byte vectors of x
    const uint32_t wgs_xcd = (gridDim.x + 7) / 8, share = (V + wgs_xcd - 1) / wgs_xcd;
    const uint32_t lo = (blockIdx.x / 8) * share, hi = min(V, lo + share);
    for (uint32_t f = lo + threadIdx.x; f < hi; f += nthreads) warm ^= reinterpret_cast<const uint4_t*>(x)[f][0];
  }

  CodeStream<BITS, MODE, RING> cs;
  cs.init(codes + tile_c * plan.KC * CodeStream<BITS, MODE, RING>::kChunkBytes,
          MODE == 1 ? scales + tile_c * plan.KC * 128 : nullptr, lane, PK, KS, ks, (int)plan.KC);
  const bool xlane = j < B;
  float4_t acc = {0.f, 0.f, 0.f, 0.f};

  for (int p = 0; p < NP; ++p) {
    // ---- 2. stage the activation piece: maxima, then fp16
    uint32_t* pm = piece_max[p & 1];
    // the 64 lanes of a wavefront hold consecutive vectors, so they span a
    // few consecutive batch rows: one wavefront reduction and one LDS atomic
    // per row
#pragma unroll
    for (int n = 0; n < kStageVec; ++n) {
      const float m = max_abs8(v[n]);
      const int r0 = __builtin_amdgcn_readfirstlane(sj[n]), r1 = __builtin_amdgcn_readlane(sj[n], 63);
      for (int r = r0; r <= r1 && r < B; ++r) {
        const float mr = wave_max(sj[n] == r ? m : 0.0f);
        if (lane == 0 && mr > 0.0f) atomicMax(&pm[r], __float_as_uint(mr));
      }
    }
    if (p == 0) asm volatile("" ::"v"(warm));      // the warm-up loads have landed
    __syncthreads();
#pragma unroll
    for (int n = 0; n < kStageVec; ++n)
      if (sj[n] < B)
        *reinterpret_cast<half8_t*>(xs + sj[n] * rowstride + spos[n] * 8) =
            to_half8_scaled(v[n], __builtin_ldexpf(1.0f, stage_exponent(pm[sj[n]])));
    if ((int)threadIdx.x < 16) piece_max[(p + 1) & 1][threadIdx.x] = 0u;   // last read in piece p-1
    __syncthreads();
    const float unscale = xlane ? __builtin_ldexpf(1.0f, -stage_exponent(pm[j])) : 1.0f;
    if (p == 0) {
      // ---- 3. the first RING code loads, once the first piece is staged (a
      // load issued while the weight streams start can stall on back-pressure)
#pragma unroll
      for (int r = 0; r < RING; ++r) cs.load(r, cs.chunk(0, r));
    }
    load_piece_x(min(p + 1, NP - 1));              // L2 hits (warmed above); the last piece re-reads itself

    // ---- 4. this wavefront's slots of the piece
    float4_t pacc[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) pacc[st] = float4_t{0.f, 0.f, 0.f, 0.f};
    const _Float16* xrow = xs + (xlane ? j : 0) * rowstride + 32 * q;
    consume<BITS, MODE, RING>(cs, p, min(p + 1, NP - 1), plan.CPW, xrow, tile_ok ? 0 : PK, tab, pacc);
#pragma unroll
    for (int r2 = 0; r2 < 4; ++r2) acc[r2] += ((pacc[0][r2] + pacc[1][r2]) + (pacc[2][r2] + pacc[3][r2])) * unscale;
    __syncthreads();   // the piece buffer is free again
  }
  if (MODE == 1) {
    const float g = *Gp;
#pragma unroll
    for (int r2 = 0; r2 < 4; ++r2) acc[r2] *= g;
  }
  // ---- 5. K-split reduction and store
  reduce_store(acc, red, wave, lane, ks, KS, tile_ok, tile, N, out_kind, y, xlane);
}

// n zero elements of 4 (fp32) or 2 (bf16) bytes
template <typename T>
__global__ void zero_fill_kernel(T* p, int64_t n) {
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n; t += (int64_t)gridDim.x * blockDim.x) p[t] = 0;
}

constexpr int64_t kLdsPerCu = 160 * 1024;
constexpr int kCUs = 256;

constexpr int kRingPersist = 4;
constexpr int64_t kPersistLdsMax = 150 * 1024;

// Workgroups of `waves` wavefronts that one compute unit holds at once: the
// waves of a workgroup are spread evenly over the 4 SIMDs, so each SIMD needs
// room for ceil(waves / 4) of them (a SIMD holds 512 / VGPRs-per-wave, at
// most 8), and the LDS must hold all of them.
inline int persist_wgs_per_cu(int vgprs, int waves, int64_t lds) {
  const int per_simd = std::min(8, 512 / (int)round_up(vgprs, 8));
  const int by_vgpr = per_simd / ((waves + 3) / 4);
  const int by_lds = (int)(kLdsPerCu / std::max<int64_t>(1, lds + 1024));
  return std::max(1, std::min(by_vgpr, by_lds));
}

// Wavefront tasks per compute unit for the batched kernel.  Fewer tasks mean
// fewer K groups: less partial-sum traffic and less activation staging per
// weight byte, but fewer wavefronts streaming.  Measured over the 27B block
// (q/k/v, o, gate/up, down), one call each in a captured graph: at batch 8,
// 12 tasks 5 % faster than 6 in total (gate/up and down gain, the small
// matrices lose); at batch 16, 6 tasks 12 % faster than 12 (the activation
// staging of a K group grows with the batch); 24 and 48 slower everywhere.
// (Timed alone, 64 calls of one matrix in a row, q/k/v and o at batch 8 run
// faster with 6 tasks; in the token's order of matrices they do not.)
inline int64_t gemv_tasks_per_cu(int64_t B) { return B >= 12 ? 6 : 12; }

// Plan of the batch B >= 2 split-K kernel (see lut_gemv_split_kernel).
struct BatchedPlan {
  bool ok;               // false: the codes exceed the kernel's 32-bit offsets
  int64_t KG, KCR, TPW;  // K groups, chunks per K group, tiles per wavefront
  int64_t TI, G, lds;    // table KiB per wavefront, workgroups, LDS bytes
  size_t partial_bytes;  // K-group partial sums (0 when KG == 1)
};

inline BatchedPlan plan_batched(int bits, int64_t B, int64_t T, int64_t KC) {
  constexpr int kW = 8;
  const int64_t tab_bytes = 32 << bits;
  BatchedPlan p{};
  p.ok = T * KC * 64 * (bits == 3 ? 12 : 8) < ((int64_t)1 << 31);
  // wavefront tasks (one tile over one K group) per compute unit; a K
  // group's slice of x stays within ~40 KiB of LDS
  const int64_t tasks = (int64_t)num_cus() * gemv_tasks_per_cu(B);
  const int64_t kcr_lds = std::max<int64_t>(1, (40 * 1024) / (B * 256));
  int64_t KG = std::max<int64_t>((KC + kcr_lds - 1) / kcr_lds, std::min<int64_t>(KC, (tasks + T - 1) / T));
  p.KCR = (KC + KG - 1) / KG;
  p.KG = (KC + p.KCR - 1) / p.KCR;
  p.TPW = std::min<int64_t>(16, std::max<int64_t>(1, T * p.KG / tasks));
  p.TI = (p.TPW * tab_bytes + 1023) / 1024;
  const int64_t TG = (T + kW * p.TPW - 1) / (kW * p.TPW);
  p.G = p.KG * TG;
  p.lds = round_up(B * (p.KCR * 128 + 8) * 2, 16) + kW * p.TI * 1024;
  p.partial_bytes = p.KG > 1 ? (size_t)(p.KG * T * B * 16 * 4) : 0;
  return p;
}

// Batch B >= 2: split-K kernel, and with more than one K group a reduction
// pass over the K-group partials, held in the caller's workspace `ws` (at
// least plan.partial_bytes) or, when ws is NULL, in stream-ordered staging
// from the library's pool.  Returns hipErrorNotSupported when the matrix is
// too large for the kernel's 32-bit offsets.
template <int BITS, int MODE>
hipError_t launch_gemv_batched(const uint16_t* x, int64_t B, const LutView& w, int out_kind, void* y, void* ws,
                               hipStream_t s, int64_t T, int64_t KC) {
  constexpr int kW = 8;
  const int64_t N = w.rows, K = w.cols;
  const BatchedPlan p = plan_batched(BITS, B, T, KC);
  if (!p.ok) return hipErrorNotSupported;
  typedef void (*kern_t)(const uint16_t*, int64_t, int, const uint8_t*, const uint16_t*, const uint8_t*,
                         const float*, int64_t, SplitPlan, float*, int, void*);
  kern_t kern;
  switch (MODE == 1 ? 1 : p.TI) {
    case 1: kern = lut_gemv_split_kernel<BITS, MODE, kRingPersist, 1>; break;
    case 2: kern = lut_gemv_split_kernel<BITS, MODE, kRingPersist, 2>; break;
    case 3: kern = lut_gemv_split_kernel<BITS, MODE, kRingPersist, 3>; break;
    default: kern = lut_gemv_split_kernel<BITS, MODE, kRingPersist, 4>; break;
  }
  float* partials = reinterpret_cast<float*>(ws);
  const bool pooled = p.KG > 1 && partials == nullptr;
  hipError_t e = hipSuccess;
  if (pooled) {
    e = pool_alloc_async(reinterpret_cast<void**>(&partials), p.partial_bytes, s);
    if (e != hipSuccess) return e;
  }
  SplitPlan sp{};
  sp.KG = (int)p.KG;
  sp.TPW = (int)p.TPW;
  sp.KCR = (int)p.KCR;
  sp.tiles = (int)T;
  sp.KC = (int)KC;
  hipLaunchKernelGGL(kern, dim3((unsigned)p.G), dim3(kW * 64), (size_t)p.lds, s, x, K, (int)B, w.codes, w.lut,
                     w.scales, w.G, N, sp, partials, out_kind, y);
  e = hipGetLastError();
  if (p.KG > 1 && e == hipSuccess) {
    const int64_t n = T * B * 16;
    hipLaunchKernelGGL(reduce_partials_kernel, dim3((unsigned)std::min<int64_t>(2048, (n + 255) / 256)), dim3(256), 0,
                       s, partials, (int)p.KG, (int)T, (int)B, N, out_kind, y);
    e = hipGetLastError();
  }
  if (pooled) {
    const hipError_t f = hipFreeAsync(partials, s);
    if (e == hipSuccess) e = f;
  }
  return e;
}

template <int BITS, int MODE>
hipError_t launch_gemv_t(const uint16_t* x, int64_t B, const LutView& w, int out_kind, void* y, void* ws,
                         hipStream_t s) {
  const int64_t N = w.rows, K = w.cols;
  GemvPlan pl{};
  pl.tiles = round_up(N, 16) / 16;
  pl.KC = round_up(K, 128) / 128;
  if (B >= 2) {
    const hipError_t e = launch_gemv_batched<BITS, MODE>(x, B, w, out_kind, y, ws, s, pl.tiles, pl.KC);
    if (e != hipErrorNotSupported) return e;
  }
  // Persistent kernel whenever the staged activations leave room for at
  // least one workgroup per compute unit and a workgroup needs at most 8
  // rounds (2 KiB of tables per wavefront).  Four wavefronts split a row
  // tile's K when each then streams at most 10 chunks, else eight (measured
  // at batch 1: 8B up-projection, 8 chunks each, 13 % faster with four; 27B
  // gate/up 5 %; the 27B down-projection, 34 chunks each, 49 % slower).
  if (B == 1) {
    const int kW = (pl.KC + 3) / 4 <= 10 ? 4 : 8;
    constexpr int kTabBytes = 32 << BITS;
    const int64_t code_bytes = pl.tiles * pl.KC * 64 * (BITS == 3 ? 12 : 8);
    const int64_t cpw = (pl.KC + kW - 1) / kW;
    const int xv = B == 1 && cpw <= 8 ? 0 : B == 1 && cpw <= 18 ? 1 : 2;   // activation staging variant
    auto table_kib = [&](int64_t rounds) { return (rounds * kTabBytes + 1023) / 1024; };
    // LDS: staged activations, per round W partial sums, W table copies
    auto lds_of = [&](int64_t rounds) {
      return B * ((pl.KC + 1) * 128 + 8) * 2 + rounds * kW * 1024 + (MODE == 0 ? kW * table_kib(rounds) * 1024 : 0);
    };
    typedef void (*kern_t)(const uint16_t*, int, int64_t, const uint8_t*, const uint16_t*, const uint8_t*,
                           const float*, int64_t, PersistPlan, int, void*);
    auto pick = [&](int ti) -> kern_t {
      if (ti <= 1)
        return xv == 0 ? lut_gemv_persist_kernel<BITS, MODE, kRingPersist, 8, 1>
               : xv == 1 ? lut_gemv_persist_kernel<BITS, MODE, kRingPersist, 18, 1>
                         : lut_gemv_persist_kernel<BITS, MODE, kRingPersist, 0, 1>;
      return xv == 0 ? lut_gemv_persist_kernel<BITS, MODE, kRingPersist, 8, 2>
             : xv == 1 ? lut_gemv_persist_kernel<BITS, MODE, kRingPersist, 18, 2>
                       : lut_gemv_persist_kernel<BITS, MODE, kRingPersist, 0, 2>;
    };
    if (lds_of(1) <= kPersistLdsMax && code_bytes < ((int64_t)1 << 31)) {
      // VGPRs of the kernels (the same for every table count), queried once
      static std::atomic<int> vgprs_of[3];
      std::atomic<int>& vgprs = vgprs_of[xv];
      if (vgprs.load(std::memory_order_relaxed) == 0) {
        hipFuncAttributes a{};
        vgprs.store(hipFuncGetAttributes(&a, reinterpret_cast<const void*>(pick(1))) == hipSuccess && a.numRegs > 0
                        ? a.numRegs : 128, std::memory_order_relaxed);
      }
      // rounds: one per resident workgroup slot, every workgroup running the
      // same number (a partial last round would leave few wavefronts
      // streaming at the end).  At most four workgroups per compute unit:
      // wavefronts start at about two per nanosecond over the whole chip, so
      // the 27B gate/up matrix (2176 row tiles) ran 3-4 % faster as 726
      // workgroups of three rounds than as 1088 of two; smaller matrices keep
      // one round either way.
      int64_t rounds = 1;
      for (int it = 0; it < 3; ++it) {
        const int per_cu =
            std::min(4, persist_wgs_per_cu(vgprs.load(std::memory_order_relaxed), kW, lds_of(rounds)));
        const int64_t gmax = std::max<int64_t>(1, (int64_t)num_cus() * per_cu);
        rounds = (pl.tiles + gmax - 1) / gmax;
      }
      const int ti = (int)table_kib(rounds);
      if (lds_of(rounds) <= kPersistLdsMax && (MODE == 1 || ti <= 2)) {
        PersistPlan pp{};
        pp.tiles = pl.tiles;
        pp.KC = pl.KC;
        pp.CPW = (int)cpw;
        pp.rounds = (int)rounds;
        const int64_t G = (pl.tiles + rounds - 1) / rounds;
        hipLaunchKernelGGL(pick(ti), dim3((unsigned)G), dim3(kW * 64), (size_t)lds_of(rounds), s, x, (int)B, K,
                           w.codes, w.lut, w.scales, w.G, N, pp, out_kind, y);
        return hipGetLastError();
      }
    }
  }
pieces:
  // Several pieces.  Row tiles per workgroup: the workgroups must spread
  // evenly over the compute units (cost = rounds x row tiles per workgroup);
  // ties go to more row tiles per workgroup, which amortizes the staging.  K
  // splits per row tile: about 8 chunks per wavefront, at most 12 wavefronts.
  const int64_t ks0 = std::max<int64_t>(1, (pl.KC + 7) / 8);
  int best_rt = 1;
  int64_t best_cost = INT64_MAX;
  for (int rt = 1; rt <= 12; ++rt) {
    const int64_t wgs = (pl.tiles + rt - 1) / rt;
    const int64_t cost = ((wgs + kCUs - 1) / kCUs) * rt;
    if (cost <= best_cost) {
      best_cost = cost;
      best_rt = rt;
    }
  }
  pl.RT = best_rt;
  pl.KS = (int)std::min<int64_t>(ks0, std::max(1, 12 / pl.RT));
  const int W = pl.RT * pl.KS;
  const int nthreads = W * 64;
  // piece: activations in LDS (<= 64 KiB with the zero chunk) and at most
  // kStageVec 8-vectors per thread
  auto lds_x = [&](int64_t pk) { return B * ((pk + 1) * 128 + 8) * 2; };
  int64_t pk = pl.KC;
  while (pk > 1 && (lds_x(pk) > 64 * 1024 || B * pk * 16 > (int64_t)kStageVec * nthreads)) pk = (pk + 1) / 2;
  pl.PK = (int)pk;
  pl.npieces = (int)((pl.KC + pk - 1) / pk);
  pl.CPW = (int)round_up((pk + pl.KS - 1) / pl.KS, kRingMulti);
  const size_t lds = (size_t)lds_x(pk) + (size_t)W * 1024;
  const int64_t blocks = (pl.tiles + pl.RT - 1) / pl.RT;
  hipLaunchKernelGGL((lut_gemv_multi_kernel<BITS, MODE>), dim3((unsigned)blocks), dim3(nthreads), lds, s, x, (int)B,
                     K, w.codes, w.lut, w.scales, w.G, N, pl, out_kind, y);
  return hipGetLastError();
}

}  // namespace

// Scratch of dq_decode_gemv_noalloc: the split-K partial sums of batch >= 2
// calls, for callers that cannot allocate.  Each GPU the library runs on
// holds its own copy until the process ends; its device address is looked up
// once per device (host code must never pass the array's name itself: that
// is a host-side stand-in).  Calls that overlap on one GPU share it and race.
// The partial sums are written in full by the split kernel before the
// reduction reads them, so nothing needs clearing between calls.
constexpr size_t kNoallocScratchBytes = DQ_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kNoallocScratchBytes];

size_t gemv_noalloc_scratch_bytes() { return kNoallocScratchBytes; }

hipError_t gemv_noalloc_scratch(void** ptr) {
  static std::mutex mu;
  static void* dev_ptr[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (dev_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    dev_ptr[dev] = p;
  }
  *ptr = dev_ptr[dev];
  return hipSuccess;
}

size_t gemv_workspace_bytes(int64_t B, const LutView& w) {
  if (B < 2 || w.rows == 0 || w.cols == 0) return 0;
  const BatchedPlan p = plan_batched(w.bits, B, round_up(w.rows, 16) / 16, round_up(w.cols, 128) / 128);
  return p.ok ? p.partial_bytes : 0;
}

hipError_t launch_gemv(const uint16_t* x, int64_t B, const LutView& w, int out_kind, void* y, void* ws,
                       hipStream_t s) {
  if (w.rows == 0 || B == 0) return hipSuccess;
  if (w.cols == 0) {   // empty sum: y = 0 (fp32 or bf16 zeros are all-zero bits)
    const int64_t n = B * w.rows;
    const dim3 grid((unsigned)std::min<int64_t>(1024, (n + 255) / 256));
    if (out_kind == 0)
      hipLaunchKernelGGL(zero_fill_kernel<uint32_t>, grid, dim3(256), 0, s, reinterpret_cast<uint32_t*>(y), n);
    else
      hipLaunchKernelGGL(zero_fill_kernel<uint16_t>, grid, dim3(256), 0, s, reinterpret_cast<uint16_t*>(y), n);
    return hipGetLastError();
  }
  if (w.bits == 3)
    return w.mode == 0 ? launch_gemv_t<3, 0>(x, B, w, out_kind, y, ws, s)
                       : launch_gemv_t<3, 1>(x, B, w, out_kind, y, ws, s);
  return w.mode == 0 ? launch_gemv_t<2, 0>(x, B, w, out_kind, y, ws, s)
                     : launch_gemv_t<2, 1>(x, B, w, out_kind, y, ws, s);
}

}  // namespace dq
