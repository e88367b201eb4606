// NVFP4A16 decode GEMV on gfx950: the weight-only NVFP4 decode of format
// disaggregation (paper Sec. 2.3: decode keeps the activations in 16 bits
// and only the weights quantized; App. A "Quantization formats", "NVFP4").
//
//   y[b, n] = G * sum_k x[b, k] * e2m1(c[n, k]) * e4m3(s[n, k/16])
//
// Weights are the NVFP4 tensors of dq_pack_nvfp4 (32x64 tiles).  Lane l of a
// tile holds row l%32, columns 32(l/32)..+31: exactly the A operand of
// v_mfma_f32_32x32x16_f16 over four sub-steps (dword s = columns
// 32(l/32) + 8s .. +7, a permutation of K shared with the x operand).  Each
// dword becomes 8 exact fp16 values (hardware E2M1 -> fp16 conversion, one
// packed multiply by the E4M3 block scale: products of at most 6
// significant bits).  The activations are staged in LDS as fp16 after a
// power-of-two rescale per batch row and K group (the reading used by the
// LUT GEMV), so every product is exact and the sums are fp32.
//
// Work split: a workgroup takes one K group of a group of row tiles, stages
// that K slice of x once, and its wavefronts each stream whole tiles over the
// K group (no reduction between wavefronts).  With more than one K group the
// tile sums go to a workspace that a second pass adds up in K-group order
// (deterministic).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "dq_device.hpp"
#include "dq_internal.hpp"

namespace dq {

// Raw buffer loads (LLVM AMDGPU intrinsics): a scalar resource, a per-lane
// offset and a uniform offset; offsets past the resource size read zero.
typedef int32_t v4i_t __attribute__((ext_vector_type(4)));
__device__ v4i_t nv_buffer_load_b128(v4i_t rsrc, int32_t voff, int32_t soff,
                                     int32_t aux) __asm("llvm.amdgcn.raw.buffer.load.v4i32");
__device__ int16_t nv_buffer_load_b16(v4i_t rsrc, int32_t voff, int32_t soff,
                                      int32_t aux) __asm("llvm.amdgcn.raw.buffer.load.i16");

namespace {

// buffer resource over [p, p + bytes) (reads past the range return zero)
__device__ inline v4i_t nv_resource(const void* p, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  return v4i_t{(int32_t)(uint32_t)a, (int32_t)(uint32_t)((a >> 32) & 0xFFFFu), (int32_t)bytes, 0x00020000};
}

// 8 E2M1 codes times an fp16 block scale -> 8 exact fp16 values
__device__ inline half8_t nv_dequant8(uint32_t w, half2_t s) {
  const half2_t p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 0) * s;
  const half2_t p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 1) * s;
  const half2_t p2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 2) * s;
  const half2_t p3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 3) * s;
  return half8_t{p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

// fp16 rescale exponent of a batch row whose maximum magnitude has bits mb:
// the maximum lands in [2^14, 2^15)
__device__ inline int nv_stage_exponent(uint32_t mb) {
  return mb ? min(126, 14 - ((int)((mb >> 23) & 0xFF) - 127)) : 0;
}

constexpr int kNvWaves = 4;
constexpr int kCyc = 4;   // K steps per cycle of code loads

// maximum over the wavefront (all 64 lanes must be active)
__device__ inline float nv_wave_max(float m) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  return m;
}

// Workgroup (K group kg, tile group tg) of 4 wavefronts (four workgroups per
// compute unit).  The K group's
// slice of x (all B rows, KCR = 8 KC8 steps of 64 columns) is staged once in
// LDS as fp16; wavefront w then owns tiles (tg * 8 + w) * TPW + i, i < TPW,
// each over the whole K group, in cycles of kCyc steps: the code and scale loads
// of cycle q+1 are issued before cycle q is consumed (a fixed count, so the
// compiler's wait for them is exact); tiles and steps past the end read zeros
// through range-checked buffer loads, without touching memory.
template <int KC8>
__global__ __launch_bounds__(256) void nvfp4_gemv_kernel(const uint16_t* __restrict__ x, int B, int64_t K,
                                                         const uint8_t* __restrict__ codes,
                                                         const uint8_t* __restrict__ scales,
                                                         const float* __restrict__ Gp, int64_t N, int T, int KT,
                                                         int KG, int TPW, float* __restrict__ partials, int out_kind,
                                                         void* __restrict__ y) {
  constexpr int KCR = 8 * KC8;                        // K steps (64 columns) per K group
  constexpr int kRow = KCR * 64 + 8;                  // fp16 per staged batch row (+ pad)
  extern __shared__ __align__(16) uint8_t smem[];
  _Float16* xs = reinterpret_cast<_Float16*>(smem);   // [B + 1][kRow]: row B is zeros
  __shared__ uint32_t s_max[32];
  __shared__ float s_unscale[32];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int kg = (int)(blockIdx.x % (unsigned)KG), tg = (int)(blockIdx.x / (unsigned)KG);
  const int kt0 = kg * KCR;
  const int64_t k0 = (int64_t)kt0 * 64;
  const int valid = min(KCR, KT - kt0);               // valid steps of this K group
  const int r = lane & 31, h = lane >> 5;
  const int c_off = 16 * (2 * r + h);                 // row r, columns 32h..32h+31 of a tile
  const int s_off = 4 * r + 2 * h;                    // E4M3 scales of blocks 2h, 2h+1 of row r
  const int tile0 = (tg * kNvWaves + wave) * TPW;

  // loads of cycle q (tile tile0 + q / CPT, steps kCyc (q % CPT) .. +kCyc-1)
  // into one of two named buffers (they must stay in registers)
  struct Cycle {
    uint4_t c[kCyc];
    uint32_t s[kCyc];
  };
  constexpr int CPT = KCR / kCyc;                     // cycles per tile
  Cycle cb0, cb1;
  auto issue = [&](int q, Cycle& cb) {
    const int t = tile0 + q / CPT, st0 = kCyc * (q % CPT);
    const bool ok = t < T;
    const v4i_t rc = nv_resource(codes + ((int64_t)(ok ? t : 0) * KT + kt0) * 1024, ok ? (uint32_t)valid * 1024u : 0u);
    const v4i_t rs = nv_resource(scales + ((int64_t)(ok ? t : 0) * KT + kt0) * 128, ok ? (uint32_t)valid * 128u : 0u);
#pragma unroll
    for (int u = 0; u < kCyc; ++u) {
      const v4i_t v = nv_buffer_load_b128(rc, c_off, (st0 + u) * 1024, 0);
      cb.c[u] = uint4_t{(uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]};
      cb.s[u] = (uint16_t)nv_buffer_load_b16(rs, s_off, (st0 + u) * 128, 0);
    }
  };
  issue(0, cb0);

  // ---- stage x[:, k0 .. k0 + 64 KCR) as fp16: per batch row, the maximum
  // over the slice, a power-of-two scale, conversion in place
  if (threadIdx.x < 32) s_max[threadIdx.x] = 0u;
  for (int i = threadIdx.x; i < kRow / 2; i += blockDim.x) reinterpret_cast<uint32_t*>(xs + B * kRow)[i] = 0u;
  __syncthreads();
  // Eight loads in flight per thread before any is used (a load followed by
  // its use in every iteration would pay the memory latency per piece).  A
  // row holds a multiple of 64 pieces, so the 64 pieces of a wavefront's
  // load u all belong to one row: one LDS atomic per wavefront and load.
  const int per_row = KCR * 64 / 8;                   // 8-element pieces per batch row
  constexpr int kStageBatch = 8;
  for (int p0 = threadIdx.x; p0 < B * per_row; p0 += kStageBatch * (int)blockDim.x) {
    uint4_t v[kStageBatch];
#pragma unroll
    for (int u = 0; u < kStageBatch; ++u) {
      const int p = p0 + u * (int)blockDim.x;
      const int b = p / per_row, e = (p - b * per_row) * 8;
      v[u] = uint4_t{0u, 0u, 0u, 0u};
      if (p < B * per_row && k0 + e < K)
        v[u] = *reinterpret_cast<const uint4_t*>(x + (int64_t)b * K + k0 + e);   // K % 16 == 0
    }
#pragma unroll
    for (int u = 0; u < kStageBatch; ++u) {
      const int p = p0 + u * (int)blockDim.x;
      if (p - lane >= B * per_row) break;             // uniform: the wavefront's pieces are all past the end
      const int b = p / per_row, e = (p - b * per_row) * 8;
      float m = 0.0f;
#pragma unroll
      for (int w4 = 0; w4 < 4; ++w4) m = fmaxf(m, fmaxf(fabsf(bf16_lo(v[u][w4])), fabsf(bf16_hi(v[u][w4]))));
      m = nv_wave_max(m);
      if (lane == 0) atomicMax(&s_max[b], __float_as_uint(m));
      *reinterpret_cast<uint4_t*>(xs + b * kRow + e) = v[u];   // raw bf16 for now
    }
  }
  __syncthreads();
  if (threadIdx.x < (unsigned)B) {
    const int e = nv_stage_exponent(s_max[threadIdx.x]);
    s_max[threadIdx.x] = (uint32_t)(e + 127);           // the scale 2^e as a biased exponent
    s_unscale[threadIdx.x] = __builtin_ldexpf(1.0f, -e) * (*Gp);
  }
  __syncthreads();
  for (int p = threadIdx.x; p < B * per_row; p += blockDim.x) {
    const int b = p / per_row, e = (p - b * per_row) * 8;
    const float sc = __uint_as_float(s_max[b] << 23);
    const uint4_t v = *reinterpret_cast<const uint4_t*>(xs + b * kRow + e);
    uint4_t o;
#pragma unroll
    for (int w4 = 0; w4 < 4; ++w4)   // the scaled values are exact in fp16
      o[w4] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(bf16_lo(v[w4]) * sc, bf16_hi(v[w4]) * sc));
    *reinterpret_cast<uint4_t*>(xs + b * kRow + e) = o;
  }
  __syncthreads();

  // ---- cycles: lane l's x operand is batch row l%32 (the zero row past B);
  // the accumulator holds batch column l%32, tile rows 8(q/4) + 4h + q%4
  const int b_l = r < B ? r : B;
  const _Float16* xl = xs + b_l * kRow + 32 * h;
  const float us = s_unscale[r < B ? r : 0];
  // two accumulators (even and odd sub-steps) keep consecutive MFMAs
  // independent; the sched_barrier after every step keeps the compiler from
  // hoisting the LDS reads and dequantization of a whole cycle (and their
  // registers)
  float16_t acc[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) acc[s] = float16_t{};
  auto consume = [&](int q, const Cycle& cb) {
    const int st0 = kCyc * (q % CPT);
#pragma unroll
    for (int u = 0; u < kCyc; ++u) {
      const half2_t sp = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(cb.s[u], 1.0f, false);
      const half2_t s_lo = half2_t{sp[0], sp[0]}, s_hi = half2_t{sp[1], sp[1]};
      half8_t xb[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) xb[s] = *reinterpret_cast<const half8_t*>(xl + (st0 + u) * 64 + 8 * s);
#pragma unroll
      for (int s = 0; s < 4; ++s)
        acc[s & 1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(nv_dequant8(cb.c[u][s], s < 2 ? s_lo : s_hi), xb[s],
                                                            acc[s & 1], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (q % CPT == CPT - 1) {   // end of a tile: its sum over the K group
      const int t = tile0 + q / CPT;
      if (t < T && r < B) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int64_t row = (int64_t)t * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
          if (row >= N) continue;
          const float v = (acc[0][i] + acc[1][i]) * us;
          if (partials != nullptr) {
            partials[((int64_t)kg * B + r) * N + row] = v;
          } else if (out_kind == 0) {
            reinterpret_cast<float*>(y)[(int64_t)r * N + row] = v;
          } else {
            reinterpret_cast<uint16_t*>(y)[(int64_t)r * N + row] = (uint16_t)f32_to_bf16_rne(v);
          }
        }
      }
#pragma unroll
      for (int s = 0; s < 2; ++s) acc[s] = float16_t{};
    }
  };
  const int cycles = TPW * CPT;
  int q = 0;
  for (; q + 2 <= cycles; q += 2) {
    issue(q + 1, cb1);
    consume(q, cb0);
    issue(q + 2, cb0);   // past the last cycle: a tile past T, zeros without memory traffic
    consume(q + 1, cb1);
  }
  if (q < cycles) consume(q, cb0);
}

// One-launch kernel for small batches (B <= 8 with the staged slices within
// 48 KiB of LDS) and at most one resident round of row tiles (16 wavefronts
// per compute unit).  A workgroup of kKsWaves (4 or 8) wavefronts takes one
// row tile;
// wavefront w takes K steps [w SPW, (w + 1) SPW).  It copies its own slice of
// x straight into LDS (issued before its code loads, so the copy is not
// queued behind them), then per batch row takes the slice maximum, a
// power-of-two scale and converts in place (no barrier: nothing is shared),
// streams its codes in cycles of kCyc steps, and parks its unscaled partial
// sums in LDS.  After the one barrier, the kKsWaves partials of each (batch
// row, tile row) are added in wavefront order and stored (deterministic).


template <int kKsWaves>
__global__ __launch_bounds__(64 * kKsWaves) void nvfp4_gemv_ks_kernel(
    const uint16_t* __restrict__ x, int B, int64_t K, const uint8_t* __restrict__ codes,
    const uint8_t* __restrict__ scales, const float* __restrict__ Gp, int64_t N, int KT, int SPW, int xslots,
    int out_kind, void* __restrict__ y) {
  extern __shared__ __align__(16) uint8_t smem[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int t = blockIdx.x;
  const int row_len = SPW * 64;                       // staged fp16 per batch row
  const int pieces = B * SPW * 8;                     // 8-element pieces of the slice
  // LDS: per wavefront xslots * 64 pieces of 16 bytes | partials [kKsWaves][B][32]
  uint8_t* xw_raw = smem + (size_t)wave * xslots * 1024;
  _Float16* xw = reinterpret_cast<_Float16*>(xw_raw);
  float* part = reinterpret_cast<float*>(smem + (size_t)kKsWaves * xslots * 1024);
  const int kt0 = wave * SPW;
  const int nst = max(0, min(SPW, KT - kt0));         // valid steps of this wavefront
  const int64_t k0 = (int64_t)kt0 * 64;

  // ---- 1. the slice of x, raw, straight into LDS: piece p (batch row
  // p / (8 SPW), columns 8 (p % (8 SPW)) ..) lands at byte 16 p; addresses
  // past K are clamped in bounds and the pieces zeroed at conversion
  for (int j = 0; j < xslots; ++j) {
    const int p = min(j * 64 + lane, pieces - 1);
    const int b = p / (SPW * 8), e = p - b * (SPW * 8);
    const int64_t k = min(k0 + 8 * e, K - 8);
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(x + (int64_t)b * K + k),
                                     reinterpret_cast<void*>(xw_raw + j * 1024), 16, 0, 0);
  }

  // ---- 2. the first two cycles of code loads
  const int r = lane & 31, h = lane >> 5;
  const int c_off = 16 * (2 * r + h);
  const int s_off = 4 * r + 2 * h;
  const v4i_t rc = nv_resource(codes + ((int64_t)t * KT + kt0) * 1024, (uint32_t)nst * 1024u);
  const v4i_t rs = nv_resource(scales + ((int64_t)t * KT + kt0) * 128, (uint32_t)nst * 128u);
  struct Cycle {
    uint4_t c[kCyc];
    uint32_t s[kCyc];
  };
  Cycle cb0, cb1;
  auto issue = [&](int q, Cycle& cb) {
#pragma unroll
    for (int u = 0; u < kCyc; ++u) {
      const v4i_t v = nv_buffer_load_b128(rc, c_off, (kCyc * q + u) * 1024, 0);
      cb.c[u] = uint4_t{(uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]};
      cb.s[u] = (uint16_t)nv_buffer_load_b16(rs, s_off, (kCyc * q + u) * 128, 0);
    }
  };
  __builtin_amdgcn_sched_barrier(0);
  issue(0, cb0);
  issue(1, cb1);
  __builtin_amdgcn_sched_barrier(0);

  // ---- 3. once the copy has landed (vmcnt: the 4 kCyc code and scale loads
  // may still be in flight), per batch row: maximum, scale, conversion
  {
    constexpr int kv = 4 * kCyc;
    __builtin_amdgcn_s_waitcnt((kv & 0xF) | ((kv >> 4) << 14) | (0x7 << 4) | (0xF << 8));
  }
  __builtin_amdgcn_sched_barrier(0);
  const float G = *Gp;
  float us = 0.0f;
  for (int b = 0; b < B; ++b) {
    uint4_t* rowp = reinterpret_cast<uint4_t*>(xw + (size_t)b * row_len);
    float m = 0.0f;
    for (int e = lane; e < SPW * 8; e += 64) {
      const uint4_t v = rowp[e];
#pragma unroll
      for (int w4 = 0; w4 < 4; ++w4) m = fmaxf(m, fmaxf(fabsf(bf16_lo(v[w4])), fabsf(bf16_hi(v[w4]))));
    }
    const int ex = nv_stage_exponent(__float_as_uint(nv_wave_max(m)));
    const float sc = __builtin_ldexpf(1.0f, ex);
    if (r == b) us = __builtin_ldexpf(1.0f, -ex) * G;
    for (int e = lane; e < SPW * 8; e += 64) {
      const uint4_t v = rowp[e];
      uint4_t o{0u, 0u, 0u, 0u};
      if (k0 + 8 * e < K) {
#pragma unroll
        for (int w4 = 0; w4 < 4; ++w4)   // the scaled values are exact in fp16
          o[w4] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(bf16_lo(v[w4]) * sc, bf16_hi(v[w4]) * sc));
      }
      rowp[e] = o;
    }
  }

  // ---- 4. cycles: lane l's x operand is batch row l%32 (row 0 for l%32 >=
  // B: those MFMA output columns are never stored)
  const _Float16* xl = xw + (size_t)(r < B ? r : 0) * row_len + 32 * h;
  float16_t acc[2] = {float16_t{}, float16_t{}};
  auto consume = [&](int q, const Cycle& cb) {
#pragma unroll
    for (int u = 0; u < kCyc; ++u) {
      const int st = min(kCyc * q + u, SPW - 1);   // past SPW: zero codes, any in-range x
      const half2_t sp = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(cb.s[u], 1.0f, false);
      const half2_t s_lo = half2_t{sp[0], sp[0]}, s_hi = half2_t{sp[1], sp[1]};
      half8_t xb[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) xb[s] = *reinterpret_cast<const half8_t*>(xl + st * 64 + 8 * s);
#pragma unroll
      for (int s = 0; s < 4; ++s)
        acc[s & 1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(nv_dequant8(cb.c[u][s], s < 2 ? s_lo : s_hi), xb[s],
                                                            acc[s & 1], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  const int cycles = (SPW + kCyc - 1) / kCyc;
  int q = 0;
  for (; q + 2 <= cycles; q += 2) {
    consume(q, cb0);
    issue(q + 2, cb0);   // past the wavefront's steps: zeros without memory traffic
    consume(q + 1, cb1);
    issue(q + 3, cb1);
  }
  if (q < cycles) consume(q, cb0);
  // the last cycle's redundant loads (zero reads) drain before the wavefront ends
  __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8));

  // ---- 5. partials, one barrier, fixed-order sum over the wavefronts
  if (r < B) {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      part[(wave * B + r) * 32 + 8 * (i >> 2) + 4 * h + (i & 3)] = (acc[0][i] + acc[1][i]) * us;
  }
  __syncthreads();
  if ((int)threadIdx.x < B * 32) {
    const int b = threadIdx.x >> 5, rr = threadIdx.x & 31;
    float v = part[b * 32 + rr];
    for (int w = 1; w < kKsWaves; ++w) v += part[(w * B + b) * 32 + rr];
    const int64_t row = (int64_t)t * 32 + rr;
    if (row < N) {
      if (out_kind == 0)
        reinterpret_cast<float*>(y)[(int64_t)b * N + row] = v;
      else
        reinterpret_cast<uint16_t*>(y)[(int64_t)b * N + row] = (uint16_t)f32_to_bf16_rne(v);
    }
  }
}

// y[b, n] = sum over K groups, in order, of partials[g, b, n]
__global__ __launch_bounds__(256) void nvfp4_gemv_reduce_kernel(const float* __restrict__ partials, int KG,
                                                                int64_t BN, int out_kind, void* __restrict__ y) {
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < BN; t += (int64_t)gridDim.x * blockDim.x) {
    float v = 0.0f;
    for (int g = 0; g < KG; ++g) v += partials[(int64_t)g * BN + t];
    if (out_kind == 0)
      reinterpret_cast<float*>(y)[t] = v;
    else
      reinterpret_cast<uint16_t*>(y)[t] = (uint16_t)f32_to_bf16_rne(v);
  }
}

__global__ void nv_zero_kernel(uint32_t* __restrict__ p, int64_t words) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < words; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

struct NvGemvPlan {
  int KC8, KG, TPW, T, KT, G;
  size_t lds, partial_bytes;
};

// K groups of 8 KC8 steps (the staged x slice within ~48 KiB of LDS), then
// tiles per wavefront so that about 16 wavefronts per compute unit have work.
NvGemvPlan nv_plan(int64_t B, int64_t N, int64_t K) {
  NvGemvPlan p{};
  p.T = (int)((N + 31) / 32);
  p.KT = (int)((K + 63) / 64);
  const int64_t waves = 16 * (int64_t)num_cus();
  const int kc8_lds = std::max<int>(1, (int)((48 * 1024) / ((B + 1) * 8 * 64 * 2)));
  // K groups: enough for the wavefronts, at most what the LDS slice allows
  int kg = (int)std::max<int64_t>(1, std::min<int64_t>((waves + p.T - 1) / p.T, (p.KT + 7) / 8));
  int kc8 = std::max(1, ((p.KT + kg - 1) / kg + 7) / 8);
  kc8 = std::min(kc8, std::min(kc8_lds, 4));
  p.KC8 = kc8 >= 4 ? 4 : kc8 >= 2 ? 2 : 1;
  p.KG = (p.KT + 8 * p.KC8 - 1) / (8 * p.KC8);
  p.TPW = (int)std::max<int64_t>(1, (int64_t)p.T * p.KG / waves);
  const int tg = (p.T + kNvWaves * p.TPW - 1) / (kNvWaves * p.TPW);
  p.G = p.KG * tg;
  p.lds = (size_t)(B + 1) * (size_t)(8 * p.KC8 * 64 + 8) * 2;
  p.partial_bytes = p.KG > 1 ? (size_t)p.KG * (size_t)B * (size_t)N * 4 : 0;
  return p;
}

// The one-launch kernel: a workgroup per row tile when the tiles fit the
// resident workgroups (16 wavefronts per compute unit) and the staged slices
// fit in LDS.  Four wavefronts per workgroup when that leaves each at most 16
// K steps, else eight (measured: 8B up-projection at batch 1 8 % faster with
// four, 16 steps each; the 27B down-projection 20 % slower with four, 68
// steps each).
struct KsPlan {
  bool ok;
  int W, T, KT, SPW, xslots;
  size_t lds;
};

KsPlan ks_plan(int64_t B, int64_t N, int64_t K) {
  KsPlan p{};
  const int64_t T = (N + 31) / 32, KT = (K + 63) / 64;
  const int W = (KT + 3) / 4 <= 16 ? 4 : 8;
  const int64_t SPW = (KT + W - 1) / W;
  const int64_t xslots = (B * SPW * 8 + 63) / 64;
  p.lds = (size_t)W * (size_t)xslots * 1024 + (size_t)W * (size_t)B * 32 * 4;
  p.ok = B >= 1 && B <= 8 && T <= (16 / W) * (int64_t)num_cus() && p.lds <= 48 * 1024;
  p.W = W;
  p.T = (int)T;
  p.KT = (int)KT;
  p.SPW = (int)SPW;
  p.xslots = (int)xslots;
  return p;
}

}  // namespace

size_t gemv_nvfp4_workspace_bytes(int64_t B, int64_t N, int64_t K) {
  if (B < 1 || N == 0 || K == 0 || ks_plan(B, N, K).ok) return 0;
  return nv_plan(B, N, K).partial_bytes;
}

hipError_t launch_gemv_nvfp4(const uint16_t* x, int64_t B, const NvFp4View& w, int out_kind, void* y, void* ws,
                             hipStream_t s) {
  const int64_t N = w.rows, K = w.cols;
  if (N == 0 || B == 0) return hipSuccess;
  if (K == 0) {   // empty sum: y = 0 (fp32 or bf16 zeros are all-zero bits)
    const int64_t words = (B * N * (out_kind == 0 ? 4 : 2) + 3) / 4;
    hipLaunchKernelGGL(nv_zero_kernel, dim3((unsigned)std::min<int64_t>(1024, (words + 255) / 256)), dim3(256), 0, s,
                       reinterpret_cast<uint32_t*>(y), words);
    return hipGetLastError();
  }
  const KsPlan ks = ks_plan(B, N, K);
  if (ks.ok) {
    if (ks.W == 4)
      hipLaunchKernelGGL(nvfp4_gemv_ks_kernel<4>, dim3((unsigned)ks.T), dim3(256), ks.lds, s, x, (int)B, K, w.codes,
                         w.scales, w.G, N, ks.KT, ks.SPW, ks.xslots, out_kind, y);
    else
      hipLaunchKernelGGL(nvfp4_gemv_ks_kernel<8>, dim3((unsigned)ks.T), dim3(512), ks.lds, s, x, (int)B, K, w.codes,
                         w.scales, w.G, N, ks.KT, ks.SPW, ks.xslots, out_kind, y);
    return hipGetLastError();
  }
  const NvGemvPlan p = nv_plan(B, N, K);
  float* partials = reinterpret_cast<float*>(ws);
  const bool pooled = p.KG > 1 && partials == nullptr;
  hipError_t e = hipSuccess;
  if (pooled) {
    e = pool_alloc_async(reinterpret_cast<void**>(&partials), p.partial_bytes, s);
    if (e != hipSuccess) return e;
  }
  typedef void (*kern_t)(const uint16_t*, int, int64_t, const uint8_t*, const uint8_t*, const float*, int64_t, int,
                         int, int, int, float*, int, void*);
  const kern_t kern = p.KC8 == 4 ? nvfp4_gemv_kernel<4> : p.KC8 == 2 ? nvfp4_gemv_kernel<2> : nvfp4_gemv_kernel<1>;
  hipLaunchKernelGGL(kern, dim3((unsigned)p.G), dim3(64 * kNvWaves), p.lds, s, x, (int)B, K, w.codes, w.scales,
                     w.G, N, p.T, p.KT, p.KG, p.TPW, p.KG > 1 ? partials : nullptr, out_kind, y);
  e = hipGetLastError();
  if (p.KG > 1 && e == hipSuccess) {
    const int64_t BN = B * N;
    hipLaunchKernelGGL(nvfp4_gemv_reduce_kernel, dim3((unsigned)std::min<int64_t>(2048, (BN + 255) / 256)),
                       dim3(256), 0, s, partials, p.KG, BN, out_kind, y);
    e = hipGetLastError();
  }
  if (pooled) {
    const hipError_t f = hipFreeAsync(partials, s);
    if (e == hipSuccess) e = f;
  }
  return e;
}

}  // namespace dq
