// Device helpers shared by the gfx950 kernels: operand vector types, a
// compile-time loop, the E4M3 / E2M1 encoders used by the NVFP4 quantizers,
// exact fp32 division by a block scale, and the tiled NVFP4 / LUT layout
// offsets declared in dq.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace dq {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef float float16_t __attribute__((ext_vector_type(16)));
typedef uint32_t uint2_t __attribute__((ext_vector_type(2)));
typedef uint32_t uint3_t __attribute__((ext_vector_type(3)));
typedef uint32_t uint4_t __attribute__((ext_vector_type(4)));

constexpr float kGlobalDivisor = 2688.0f;  // 6 * 448: E2M1 max times E4M3 max

// f(integral_constant<int, U>) for U = B .. E - 1: unrolled loops whose
// index must be a compile-time constant (instruction offsets)
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// ---------------------------------------------------------------- layouts
// NVFP4 "32x64 tiles" (see dq.h).
__host__ __device__ inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// ---------------------------------------------------------------- E4M3
// Encode a non-negative fp32 value as OCP E4M3 (bias 7, max 448 = 0x7E):
// round to nearest, ties to even, saturating; values <= 2^-10 give 0.
__device__ inline uint32_t e4m3_encode_rne_sat(float t) {
  if (!(t > 0x1p-10f)) return 0u;
  if (t >= 448.0f) return 0x7Eu;
  if (t < 0x1p-6f) {
    // subnormal range: multiples of 2^-9; t * 512 is exact, rint is ties-to-even
    return (uint32_t)__builtin_rintf(t * 512.0f);
  }
  uint32_t b = __float_as_uint(t);
  // keep 3 mantissa bits, round the 20 dropped bits to nearest even
  uint32_t r = (b + 0x7FFFFu + ((b >> 20) & 1u)) >> 20;   // (exp << 3 | m3), carry ok
  return r - ((127u - 7u) << 3);
}

// Value of an E4M3 byte (sign in bit 7) as fp32 (exact).
__device__ inline float e4m3_decode(uint32_t c) {
  uint32_t e = (c >> 3) & 0xFu, m = c & 7u;
  float mag = (e == 0) ? (float)m * 0x1p-9f : __uint_as_float(((e + 120u) << 23) | (m << 20));
  return (c & 0x80u) ? -mag : mag;
}

// ---------------------------------------------------------------- division
// fp32 x / s, correctly rounded, given rcp = RN(1/s) (Markstein's correction:
// q0 = RN(x*rcp) is faithful, the residual x - q0*s is exact in one fma, and
// RN(q0 + r*rcp) is the correctly rounded quotient for normal s and x).
__device__ inline float div_by_scale(float x, float s, float rcp) {
  float q0 = x * rcp;
  float r = __builtin_fmaf(-q0, s, x);
  return __builtin_fmaf(r, rcp, q0);
}

// ---------------------------------------------------------------- E2M1
// Two fp32 values -> one byte of two E2M1 codes (lo = a, hi = b), nearest with
// ties to even and saturation at 6 (hardware conversion, unit scale), placed
// in byte `sel` of `old`.
template <int sel>
__device__ inline uint32_t cvt_pk_fp4(uint32_t old, float a, float b) {
  return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, 1.0f, sel);
}

// Clear the sign bit of every nibble whose magnitude is zero (canonical +0).
__device__ inline uint32_t fp4_canonical_zero(uint32_t w) {
  uint32_t m = w & 0x77777777u;
  uint32_t nz = (m + 0x77777777u) & 0x88888888u;   // bit 3 set where magnitude != 0
  return w & (nz | 0x77777777u);
}

// bf16 bits -> fp32 (exact)
__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16 bits, round to nearest even (finite inputs)
__device__ inline uint32_t f32_to_bf16_rne(float f) {
  uint32_t b = __float_as_uint(f);
  return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

// Atomic max of a non-negative float stored as its bit pattern.
__device__ inline void atomic_max_nonneg(float* p, float v) {
  atomicMax(reinterpret_cast<unsigned int*>(p), __float_as_uint(v));
}

// ---------------------------------------------------------------- GEMM tile order
// Output tile of workgroup b.  Tiles are ordered in bands of GM row panels,
// row panel fastest within a band, so that the ~256 workgroups in flight at
// once cover about GM x 256/GM tiles and share their A and W panels through
// the L2 and the MALL.  Workgroup b runs on XCD b % 8; within each complete
// group of 256 workgroups the 32 of one XCD take a 4 x 8 sub-block, so each
// XCD's L2 streams 12 panels instead of up to 33.
__device__ inline void gemm_tile_of(int64_t b, int64_t tiles_m, int64_t tiles_n, int64_t& bm, int64_t& bn) {
  const int64_t nb = tiles_m * tiles_n;
  const int GM = tiles_m >= 16 ? 16 : tiles_m >= 8 ? 8 : tiles_m >= 4 ? 4 : (int)tiles_m;
  int64_t L = b;
  if ((GM == 4 || GM == 8 || GM == 16) && (b | 255) < nb) {
    const int q = (int)(b & 255), xcd = q & 7, loc = q >> 3;
    const int xm = GM / 4;
    const int m_in = (xcd % xm) * 4 + (loc & 3), n_in = (xcd / xm) * 8 + (loc >> 2);
    L = b - q + m_in + GM * n_in;
  }
  const int64_t band = L / (GM * tiles_n);
  const int64_t first = band * GM;
  const int64_t gm = tiles_m - first < GM ? tiles_m - first : GM;
  const int64_t idx = L - band * GM * tiles_n;
  bm = first + idx % gm;
  bn = idx / gm;
}

// ---------------------------------------------------------------- wave ops
__device__ inline float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

}  // namespace dq
