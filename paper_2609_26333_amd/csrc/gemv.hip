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
//    tile (64 lanes x 12 bytes for 3 bits, x 8 bytes for 2 bits); every
//    wavefront issues all of its code loads (up to a ring of 8 tiles) before
//    touching LDS, so the whole matrix is in flight early;
//  * each 32-code group is split into eight 4-code byte selectors with shifts
//    and masks (the bit layout in dq.h is chosen for this), and v_perm_b32
//    looks the 4 codes up in register-resident byte tables (low bytes and
//    high bytes of the row's fp16 entries), then interleaves them into fp16
//    pairs: about 1.5 VALU instructions per 3-bit weight;
//  * the multiply-accumulate runs on MFMA (v_mfma_f32_16x16x32_f16: 16 weight
//    rows x 32 k x 16 batch columns), so batch 1..16 costs the same VALU work;
//  * activations are staged once per workgroup and K-piece into LDS as fp16,
//    rescaled by a power of two per batch row (exact products with the fp16
//    table); the wavefronts of a workgroup split K and reduce through LDS in a
//    fixed order, so results are deterministic.
#include <algorithm>

#include "dq_device.hpp"
#include "dq_internal.hpp"

namespace dq {

namespace {

constexpr int kRing = 8;        // code loads in flight per wavefront
constexpr int kStageVec = 4;    // 8-element activation vectors staged per thread and piece

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

// Tables of one row (PER_ROW) or of the grid (PAPER_GRID): low bytes and high
// bytes of the 2^BITS fp16 entries, as v_perm_b32 pools.
template <int BITS>
__device__ inline void load_tables(const uint16_t* L, uint32_t& tl0, uint32_t& tl1, uint32_t& th0, uint32_t& th1) {
  if (BITS == 3) {
    const uint4_t d = *reinterpret_cast<const uint4_t*>(L);
    tl0 = __builtin_amdgcn_perm(d[1], d[0], 0x06040200u);
    th0 = __builtin_amdgcn_perm(d[1], d[0], 0x07050301u);
    tl1 = __builtin_amdgcn_perm(d[3], d[2], 0x06040200u);
    th1 = __builtin_amdgcn_perm(d[3], d[2], 0x07050301u);
  } else {
    const uint2_t d = *reinterpret_cast<const uint2_t*>(L);
    tl0 = tl1 = __builtin_amdgcn_perm(d[1], d[0], 0x06040200u);
    th0 = th1 = __builtin_amdgcn_perm(d[1], d[0], 0x07050301u);
  }
}

// Work decomposition.  A workgroup holds RT row tiles x KS K-splits
// (W = RT*KS <= 8 wavefronts).  K is processed in pieces of PK 128-column chunks;
// for each piece the workgroup stages the activations once (fp16, rescaled by
// a power of two so that the piece maximum of each batch row lands in
// [2^14, 2^15)), then wavefront (rt, ks) consumes chunks ks, ks+KS, ... of the
// piece for row tile rt.  Each wavefront walks a fixed sequence of CPW8 slots
// per piece (a multiple of 8) and keeps the code loads of the next 8 slots in
// flight across piece boundaries.  The KS partial sums of a row tile are
// reduced through LDS in a fixed order (deterministic).
struct GemvPlan {
  int RT, KS, PK, CPW8, npieces;
  int64_t tiles, KC;
};

template <int BITS, int MODE>
__global__ __launch_bounds__(512) void lut_gemv_kernel(const uint16_t* __restrict__ x, int B, int64_t K,
                                                       const uint8_t* __restrict__ codes,
                                                       const uint16_t* __restrict__ lut,
                                                       const uint8_t* __restrict__ scales,
                                                       const float* __restrict__ Gp, int64_t N, GemvPlan plan,
                                                       int out_kind, void* __restrict__ y) {
  typedef typename CodeVec<BITS>::type cvec;
  constexpr int GB = CodeVec<BITS>::bytes;
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ uint32_t piece_max[16];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nthreads = blockDim.x;
  const int rt = wave / plan.KS, ks = wave % plan.KS;
  const int64_t tile = (int64_t)blockIdx.x * plan.RT + rt;
  const bool tile_ok = tile < plan.tiles;
  const int64_t KC = plan.KC;
  const int PK = plan.PK, CPW8 = plan.CPW8, KS = plan.KS;

  // slot s of piece p -> chunk p*PK + s*KS + ks (valid when inside the piece and tile_ok)
  auto slot_chunk = [&](int p, int s, int64_t& c) -> bool {
    const int64_t local = (int64_t)s * KS + ks;
    const int64_t len = min((int64_t)PK, KC - (int64_t)p * PK);
    c = (int64_t)p * PK + local;
    return tile_ok && local < len;
  };
  const uint8_t* tile_codes = codes + (tile * KC * 64 + lane) * GB;

  // ---- 1. code loads of the first 8 slots
  cvec ring[kRing];
#pragma unroll
  for (int r = 0; r < kRing; ++r) {
    int64_t c;
    if (slot_chunk(0, r, c)) ring[r] = *reinterpret_cast<const cvec*>(tile_codes + c * 64 * GB);
  }

  // ---- 2. lookup tables (lane: row i = lane % 16 of the tile)
  const int i = lane & 15, q = lane >> 4, j = lane & 15;
  uint32_t tl0 = 0, tl1 = 0, th0 = 0, th1 = 0;
  if (tile_ok) load_tables<BITS>(MODE == 0 ? lut + (tile * 16 + i) * (1 << BITS) : lut, tl0, tl1, th0, th1);
  const uint16_t* sbase = nullptr;
  if (MODE == 1) sbase = reinterpret_cast<const uint16_t*>(scales + tile * KC * 128) + lane;

  const bool xlane = j < B;
  const int rowstride = PK * 128 + 8;              // fp16 elements per staged batch row
  _Float16* xs = reinterpret_cast<_Float16*>(smem);
  float4_t acc = {0.f, 0.f, 0.f, 0.f};

  for (int p = 0; p < plan.npieces; ++p) {
    // ---- 3. stage the activation piece (all wavefronts), one pass through registers
    const int64_t k0 = (int64_t)p * PK * 128;
    const int len = (int)min((int64_t)PK, KC - (int64_t)p * PK);
    const int vec_per_row = len * 16;              // 8-element vectors per batch row
    const int nvec = B * vec_per_row;
    if ((int)threadIdx.x < B) piece_max[threadIdx.x] = 0u;
    __syncthreads();
    uint4_t v[kStageVec];
#pragma unroll
    for (int n = 0; n < kStageVec; ++n) {
      const int f = n * nthreads + threadIdx.x;
      v[n] = uint4_t{0u, 0u, 0u, 0u};
      if (f < nvec) {
        const int jj = f / vec_per_row;
        const int64_t k = k0 + (int64_t)(f % vec_per_row) * 8;
        if (k < K) v[n] = *reinterpret_cast<const uint4_t*>(x + (int64_t)jj * K + k);
        float m = 0.0f;
#pragma unroll
        for (int w4 = 0; w4 < 4; ++w4) m = fmaxf(m, fmaxf(fabsf(bf16_lo(v[n][w4])), fabsf(bf16_hi(v[n][w4]))));
        if (m > 0.0f) atomicMax(&piece_max[jj], __float_as_uint(m));
      }
    }
    __syncthreads();
#pragma unroll
    for (int n = 0; n < kStageVec; ++n) {
      const int f = n * nthreads + threadIdx.x;
      if (f < nvec) {
        const int jj = f / vec_per_row;
        const uint32_t mb = piece_max[jj];
        const int e = mb ? min(126, 14 - ((int)((mb >> 23) & 0xFF) - 127)) : 0;
        const float sc = __builtin_ldexpf(1.0f, e);
        half8_t h;
#pragma unroll
        for (int w4 = 0; w4 < 4; ++w4) {
          h[2 * w4] = (_Float16)(bf16_lo(v[n][w4]) * sc);
          h[2 * w4 + 1] = (_Float16)(bf16_hi(v[n][w4]) * sc);
        }
        *reinterpret_cast<half8_t*>(xs + jj * rowstride + (f % vec_per_row) * 8) = h;
      }
    }
    __syncthreads();
    float unscale = 1.0f;
    if (xlane && piece_max[j]) unscale = __builtin_ldexpf(1.0f, -min(126, 14 - ((int)((piece_max[j] >> 23) & 0xFF) - 127)));

    // ---- 4. this wavefront's chunks of the piece: lookups + MFMA
    float4_t pacc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < CPW8; s0 += kRing) {
#pragma unroll
      for (int r = 0; r < kRing; ++r) {
        const int s = s0 + r;
        int64_t c;
        const bool ok = slot_chunk(p, s, c);
        cvec w;
        if (ok) w = ring[r];
        // prefetch the slot 8 ahead (possibly in the next piece)
        {
          int np = p, ns = s + kRing;
          if (ns >= CPW8) {
            ns -= CPW8;
            ++np;
          }
          int64_t nc;
          if (np < plan.npieces && slot_chunk(np, ns, nc))
            ring[r] = *reinterpret_cast<const cvec*>(tile_codes + nc * 64 * GB);
        }
        if (ok) {
          uint32_t sel[8];
          selectors<BITS>(w, sel);
          half2_t s_lo, s_hi;
          if (MODE == 1) {
            const half2_t sc2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sbase[c * 64], 1.0f, false);
            s_lo = half2_t{sc2[0], sc2[0]};
            s_hi = half2_t{sc2[1], sc2[1]};
          }
          const int cl = (int)(c - (int64_t)p * PK);
#pragma unroll
          for (int st = 0; st < 4; ++st) {
            uint32_t a0, a1, a2, a3;
            lookup4(sel[2 * st], tl0, tl1, th0, th1, a0, a1);
            lookup4(sel[2 * st + 1], tl0, tl1, th0, th1, a2, a3);
            half8_t af = as_half8(a0, a1, a2, a3);
            if (MODE == 1) af = scale_half8(af, st < 2 ? s_lo : s_hi);
            half8_t bf = half8_t{};
            if (xlane) bf = *reinterpret_cast<const half8_t*>(xs + j * rowstride + cl * 128 + 32 * q + 8 * st);
            pacc = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, bf, pacc, 0, 0, 0);
          }
        }
      }
    }
#pragma unroll
    for (int r2 = 0; r2 < 4; ++r2) acc[r2] += pacc[r2] * unscale;
    __syncthreads();   // the piece buffer is free again
  }

  // ---- 5. reduce the KS partial sums of each row tile (fixed order) and store
  if (MODE == 1) {
    const float g = *Gp;
#pragma unroll
    for (int r2 = 0; r2 < 4; ++r2) acc[r2] *= g;
  }
  float4_t* red = reinterpret_cast<float4_t*>(smem);
  red[wave * 64 + lane] = acc;
  __syncthreads();
  if (ks == 0 && tile_ok && xlane) {
    for (int k2 = 1; k2 < KS; ++k2) {
      const float4_t o = red[(wave + k2) * 64 + lane];
      acc[0] += o[0];
      acc[1] += o[1];
      acc[2] += o[2];
      acc[3] += o[3];
    }
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

template <int BITS, int MODE>
hipError_t launch_gemv_t(const uint16_t* x, int64_t B, const LutView& w, int out_kind, void* y, hipStream_t s) {
  const int64_t N = w.rows, K = w.cols;
  GemvPlan pl{};
  pl.tiles = round_up(N, 16) / 16;
  pl.KC = round_up(K, 128) / 128;
  // about 8 chunks per wavefront, at most 8 wavefronts per workgroup
  pl.KS = (int)std::min<int64_t>(8, std::max<int64_t>(1, (pl.KC + 7) / 8));
  int64_t rt = pl.tiles / 256;
  pl.RT = (int)std::max<int64_t>(1, std::min<int64_t>(rt, 8 / pl.KS));
  const int W = pl.RT * pl.KS;
  const int nthreads = W * 64;
  // piece: activations in LDS (<= 64 KiB) and at most kStageVec 8-vectors per thread
  int64_t pk = pl.KC;
  while (pk > 1 && ((int64_t)B * (pk * 128 + 8) * 2 > 64 * 1024 || B * pk * 16 > (int64_t)kStageVec * nthreads))
    pk = (pk + 1) / 2;
  pl.PK = (int)pk;
  pl.npieces = (int)((pl.KC + pk - 1) / pk);
  const int cpw = (int)((pk + pl.KS - 1) / pl.KS);
  pl.CPW8 = (cpw + kRing - 1) / kRing * kRing;
  size_t lds = (size_t)B * (pk * 128 + 8) * 2;
  const size_t red = (size_t)W * 64 * 16;
  if (lds < red) lds = red;
  auto kern = lut_gemv_kernel<BITS, MODE>;
  const int64_t blocks = (pl.tiles + pl.RT - 1) / pl.RT;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(nthreads), lds, s, x, (int)B, K, w.codes, w.lut, w.scales,
                     w.G, N, pl, out_kind, y);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemv(const uint16_t* x, int64_t B, const LutView& w, int out_kind, void* y,
                       hipStream_t s) {
  if (w.rows == 0 || B == 0) return hipSuccess;
  if (w.bits == 3)
    return w.mode == 0 ? launch_gemv_t<3, 0>(x, B, w, out_kind, y, s)
                       : launch_gemv_t<3, 1>(x, B, w, out_kind, y, s);
  return w.mode == 0 ? launch_gemv_t<2, 0>(x, B, w, out_kind, y, s)
                     : launch_gemv_t<2, 1>(x, B, w, out_kind, y, s);
}

}  // namespace dq
