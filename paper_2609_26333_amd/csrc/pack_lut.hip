// LUT weight packing on gfx950 (offline; the decode-side weight format).
//
// PER_ROW (benchmark decode format): one workgroup per output row sorts the
// row in LDS (bitonic sort of order-preserving integer keys), sums each of the
// 2^b equal-count bins in double-double arithmetic, divides by the count in
// fp64 and rounds once to fp16 (nearest even).  Codes are the nearest entry,
// ties to the lower index, decided by exact fp64 comparisons with the
// midpoints of adjacent entries.
//
// PAPER_GRID (paper App. A "LUT formats"): the NVFP4 two-level scaling with a
// signed E4M3 block scale that carries the sign of the block's
// largest-magnitude element (first on ties), codes = nearest grid level of
// fp32(w / S), ties to the lower level; zero-scale blocks take the zero level.
//
// Codes are written in the 16-row x 128-column tiled layout of dq.h.
#include "dq_device.hpp"
#include "dq_internal.hpp"

namespace dq {

namespace {

// ---------------------------------------------------------------- helpers
__device__ inline uint32_t sort_key(float f) {
  uint32_t b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ inline float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// Round-to-nearest-even right shift of a non-negative integer.
__device__ inline uint64_t rne_shift(uint64_t v, int s) {
  if (s <= 0) return v << (-s);
  if (s >= 64) return 0;
  const uint64_t q = v >> s;
  const uint64_t rem = v & ((1ull << s) - 1);
  const uint64_t half = 1ull << (s - 1);
  return q + ((rem > half || (rem == half && (q & 1))) ? 1 : 0);
}

// fp64 -> fp16 bits, one rounding to nearest even (finite input).
__device__ inline uint16_t f64_to_f16_rne(double d) {
  const uint64_t b = (uint64_t)__double_as_longlong(d);
  const uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
  const int exp = (int)((b >> 52) & 0x7FF);
  const uint64_t man = b & ((1ull << 52) - 1);
  if (exp == 0) return sign;                                   // zero or fp64 subnormal
  const int e = exp - 1023;
  const uint64_t full = man | (1ull << 52);
  if (e >= 16) return sign | 0x7C00u;                           // overflow
  if (e >= -14) {
    const uint64_t m = rne_shift(full, 42);                     // 11 bits, may carry to 2048
    const uint32_t h = ((uint32_t)(e + 15) << 10) + (uint32_t)(m - 1024);
    return sign | (uint16_t)(h >= 0x7C00u ? 0x7C00u : h);
  }
  // subnormal fp16: multiples of 2^-24; value = full * 2^(e - 52)
  const uint64_t m = rne_shift(full, (52 - 24) - e);
  return sign | (uint16_t)m;                                    // 1024 -> smallest normal
}

__device__ inline double f16_bits_to_f64(uint16_t h) {
  return (double)__builtin_bit_cast(_Float16, h);
}

// error-free sum
__device__ inline void two_sum(double a, double b, double& s, double& e) {
  s = a + b;
  const double bb = s - a;
  e = (a - (s - bb)) + (b - bb);
}

__device__ inline void dd_add(double& hi, double& lo, double x) {
  double s, e;
  two_sum(hi, x, s, e);
  hi = s;
  lo += e;
}

__device__ inline void dd_merge(double& h1, double& l1, double h2, double l2) {
  double s, e;
  two_sum(h1, h2, s, e);
  e += l1 + l2;
  const double t = s + e;          // fast two-sum normalization (|s| >= |e|)
  l1 = e - (t - s);
  h1 = t;
}

// code bits of 32 codes of one group into the dword layout of dq.h
template <int BITS>
__device__ inline void put_code(uint32_t (&w)[3], int t, uint32_t c) {
  const int s = t >> 2, b = t & 3;
  if (BITS == 3) {
    if (s < 6) {
      w[s >> 1] |= c << (8 * b + 3 * (s & 1));
    } else {
      w[s - 6] |= (c & 3u) << (8 * b + 6);
      w[2] |= (c >> 2) << (8 * b + 6 + (s - 6));
    }
  } else {
    w[s >> 2] |= c << (8 * b + 2 * (s & 3));
  }
}

template <int BITS>
__device__ inline void store_group(uint8_t* codes, int64_t row, int64_t group, int64_t KC, const uint32_t (&w)[3]) {
  constexpr int GB = BITS == 3 ? 12 : 8;
  const int64_t tile = row / 16, i = row % 16, c = group / 4, q = group % 4;
  uint32_t* p = reinterpret_cast<uint32_t*>(codes + ((tile * KC + c) * 64 + q * 16 + i) * GB);
  p[0] = w[0];
  p[1] = w[1];
  if (BITS == 3) p[2] = w[2];
}

// ---------------------------------------------------------------- PER_ROW
template <int BITS>
__global__ __launch_bounds__(1024) void pack_lut_per_row_kernel(const float* __restrict__ W, int64_t N, int64_t K,
                                                                int64_t P, int64_t KC, uint8_t* __restrict__ codes,
                                                                uint16_t* __restrict__ lut) {
  constexpr int NB = 1 << BITS;
  extern __shared__ __align__(16) uint8_t smem[];
  uint32_t* keys = reinterpret_cast<uint32_t*>(smem);
  __shared__ double part_hi[1024], part_lo[1024];
  __shared__ double mids[NB];

  const int64_t row = blockIdx.x;
  const int tid = threadIdx.x, T = blockDim.x;
  const int64_t groups = KC * 4;
  if (row >= N) {   // padding rows of the last 16-row tile: zero codes and entries
    const uint32_t z[3] = {0u, 0u, 0u};
    for (int64_t g = tid; g < groups; g += T) store_group<BITS>(codes, row, g, KC, z);
    if (tid < NB) lut[row * NB + tid] = 0;
    return;
  }
  const float* wr = W + row * K;
  for (int64_t k = tid; k < P; k += T) keys[k] = k < K ? sort_key(wr[k]) : 0xFFFFFFFFu;
  __syncthreads();
  // bitonic sort, ascending
  for (int64_t kk = 2; kk <= P; kk <<= 1) {
    for (int64_t jj = kk >> 1; jj > 0; jj >>= 1) {
      for (int64_t t = tid; t < P / 2; t += T) {
        const int64_t a = 2 * t - (t & (jj - 1));
        const int64_t b = a + jj;
        const uint32_t ka = keys[a], kb = keys[b];
        const bool up = (a & kk) == 0;
        if ((ka > kb) == up) {
          keys[a] = kb;
          keys[b] = ka;
        }
      }
      __syncthreads();
    }
  }
  // bin sums: T/NB threads per bin
  const int64_t cnt = K / NB;
  const int per = T / NB;
  const int bin = tid / per, sub = tid % per;
  double hi = 0.0, lo = 0.0;
  for (int64_t k = sub; k < cnt; k += per) dd_add(hi, lo, (double)key_value(keys[bin * cnt + k]));
  part_hi[tid] = hi;
  part_lo[tid] = lo;
  __syncthreads();
  for (int off = per / 2; off > 0; off >>= 1) {
    if (sub < off) {
      double h = part_hi[tid], l = part_lo[tid];
      dd_merge(h, l, part_hi[tid + off], part_lo[tid + off]);
      part_hi[tid] = h;
      part_lo[tid] = l;
    }
    __syncthreads();
  }
  __shared__ uint16_t entries[NB];
  if (tid < NB) {
    double h = part_hi[tid * per], l = part_lo[tid * per];
    const double sum = h + l;                 // already normalized: h == RN(h + l)
    const uint16_t e = f64_to_f16_rne(sum / (double)cnt);
    entries[tid] = e;
    lut[row * NB + tid] = e;
  }
  __syncthreads();
  if (tid < NB - 1) mids[tid] = (f16_bits_to_f64(entries[tid]) + f16_bits_to_f64(entries[tid + 1])) * 0.5;
  __syncthreads();
  // codes, one 32-column group per thread iteration
  for (int64_t g = tid; g < groups; g += T) {
    uint32_t w[3] = {0u, 0u, 0u};
    const int64_t kbase = g * 32;
    for (int t = 0; t < 32; ++t) {
      const int64_t k = kbase + t;
      if (k < K) {
        const double v = (double)wr[k];
        uint32_t c = 0;
#pragma unroll
        for (int m = 0; m < NB - 1; ++m) c += v > mids[m] ? 1u : 0u;
        put_code<BITS>(w, t, c);
      }
    }
    store_group<BITS>(codes, row, g, KC, w);
  }
}

// ---------------------------------------------------------------- PAPER_GRID
struct Grid {
  uint16_t v[8];
};

template <int BITS>
__global__ __launch_bounds__(256) void pack_lut_paper_kernel(const float* __restrict__ W, int64_t N, int64_t N16,
                                                             int64_t K, int64_t KC, const float* __restrict__ Gp,
                                                             Grid grid, int zero_level, uint8_t* __restrict__ codes,
                                                             uint8_t* __restrict__ scales, uint16_t* __restrict__ lut_out) {
  constexpr int NL = 1 << BITS;
  const int64_t groups = KC * 4;
  const int64_t gid = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (gid < NL) lut_out[gid] = grid.v[gid];
  if (gid >= N16 * groups) return;
  const int64_t row = gid / groups, g = gid % groups;
  double mid[NL - 1];
#pragma unroll
  for (int m = 0; m < NL - 1; ++m) mid[m] = (f16_bits_to_f64(grid.v[m]) + f16_bits_to_f64(grid.v[m + 1])) * 0.5;
  const float G = *Gp;
  uint32_t w[3] = {0u, 0u, 0u};
  uint32_t sb[2] = {0u, 0u};
  for (int h = 0; h < 2; ++h) {
    const int64_t k0 = g * 32 + h * 16;
    if (row >= N || k0 >= K) continue;           // padding: code 0, scale 0
    const float* wp = W + row * K + k0;
    float best = wp[0];
    float amax = fabsf(best);
    for (int t = 1; t < 16; ++t) {
      const float a = fabsf(wp[t]);
      if (a > amax) {
        amax = a;
        best = wp[t];
      }
    }
    const float t_ = amax / (6.0f * G);
    const uint32_t mag = e4m3_encode_rne_sat(t_);
    const uint32_t sbyte = mag | ((best < 0.0f && mag != 0u) ? 0x80u : 0u);
    const float S = e4m3_decode(sbyte) * G;
    sb[h] = sbyte;
    for (int t = 0; t < 16; ++t) {
      uint32_t c;
      if (S == 0.0f) {
        c = (uint32_t)zero_level;
      } else {
        const double y = (double)(wp[t] / S);
        c = 0;
#pragma unroll
        for (int m = 0; m < NL - 1; ++m) c += y > mid[m] ? 1u : 0u;
      }
      put_code<BITS>(w, h * 16 + t, c);
    }
  }
  store_group<BITS>(codes, row, g, KC, w);
  const int64_t tile = row / 16, i = row % 16, c = g / 4, q = g % 4;
  uint8_t* sp = scales + (tile * KC + c) * 128 + (q * 16 + i) * 2;
  sp[0] = (uint8_t)sb[0];
  sp[1] = (uint8_t)sb[1];
}

// ---------------------------------------------------------------- autocast
// LUT -> NVFP4 autocast, step 1: the dequantized LUT weight as fp32 [N, K],
// one thread per 32-code group of the tiled layout (dq.h).  PER_ROW entries
// are fp16 (exact in fp32); a PAPER_GRID value grid * e4m3 * G is computed
// as fp32(grid * e4m3) (exact: at most 15 significant bits) times G, one
// rounding of the exact product.
template <int BITS, int MODE>
__global__ __launch_bounds__(256) void lut_dequant_kernel(const uint8_t* __restrict__ codes,
                                                          const uint16_t* __restrict__ lut,
                                                          const uint8_t* __restrict__ scales,
                                                          const float* __restrict__ Gp, int64_t N, int64_t K,
                                                          int64_t tiles_c, float* __restrict__ out) {
  constexpr int GB = BITS == 3 ? 12 : 8;   // bytes per 32-code group
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t tile = gid >> 6;
  const int g = (int)(gid & 63), i = g & 15, q = g >> 4;
  const int64_t tr = tile / tiles_c, c = tile - tr * tiles_c;
  const int64_t row = tr * 16 + i, col0 = c * 128 + q * 32;
  if (row >= N || col0 >= K) return;
  const uint8_t* gp = codes + tile * 64 * GB + g * GB;
  uint32_t d[3];
  d[0] = *reinterpret_cast<const uint32_t*>(gp);
  d[1] = *reinterpret_cast<const uint32_t*>(gp + 4);
  d[2] = BITS == 3 ? *reinterpret_cast<const uint32_t*>(gp + 8) : 0u;
  float sb[2] = {1.0f, 1.0f};
  float G = 1.0f;
  if (MODE == 1) {
    sb[0] = e4m3_decode(scales[tile * 128 + g * 2]);
    sb[1] = e4m3_decode(scales[tile * 128 + g * 2 + 1]);
    G = *Gp;
  }
  float* o = out + row * K + col0;
#pragma unroll
  for (int t = 0; t < 32; ++t) {
    const int sl = t >> 2, b = t & 3;
    uint32_t code;
    if (BITS == 3) {
      if (sl < 6)
        code = (d[sl >> 1] >> (8 * b + 3 * (sl & 1))) & 7u;
      else
        code = ((d[sl - 6] >> (8 * b + 6)) & 3u) | (((d[2] >> (8 * b + 6 + (sl - 6))) & 1u) << 2);
    } else {
      code = (d[sl >> 2] >> (8 * b + 2 * (sl & 3))) & 3u;
    }
    const uint16_t e = MODE == 0 ? lut[row * (1 << BITS) + code] : lut[code];
    const float v = (float)__builtin_bit_cast(_Float16, e);
    if (MODE == 0) {
      o[t] = v;
    } else {
      const float p = v * sb[t >> 4];   // exact
      o[t] = p * G;
    }
  }
}

}  // namespace

// paper grids (App. A "LUT formats") rounded to fp16
static const uint16_t kPaperLut3[8] = {0xC4B4, 0xC1BD, 0xBD7A, 0x0000, 0x3CE2, 0x410F, 0x440C, 0x4600};
static const uint16_t kPaperLut2[4] = {0xC34E, 0x0000, 0x410C, 0x4600};

const uint16_t* paper_grid_fp16(int bits) { return bits == 3 ? kPaperLut3 : kPaperLut2; }

hipError_t launch_pack_lut(const float* W, int64_t N, int64_t K, const uint16_t* grid_host, const LutView& out,
                           hipStream_t s) {
  const int64_t N16 = round_up(N, 16), KC = round_up(K, 128) / 128;
  if (N16 == 0) return hipSuccess;
  if (out.mode == 0) {
    int64_t P = 64;
    while (P < K) P <<= 1;
    const size_t lds = (size_t)P * 4;
    auto kern = out.bits == 3 ? pack_lut_per_row_kernel<3> : pack_lut_per_row_kernel<2>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)N16), dim3(1024), lds, s, W, N, K, P, KC, out.codes, out.lut);
    return hipGetLastError();
  }
  const int NL = 1 << out.bits;
  Grid g{};
  const uint16_t* src = grid_host ? grid_host : paper_grid_fp16(out.bits);
  int zl = -1;
  for (int i = 0; i < NL; ++i) {
    g.v[i] = src[i];
    if ((src[i] & 0x7FFFu) == 0) zl = i;
  }
  hipError_t e = launch_global_scale_f32(W, N * K, out.G, s);   // G = max|W| / 2688, the NVFP4 rule
  if (e != hipSuccess) return e;
  const int64_t threads = N16 * KC * 4;
  const int64_t blocks = (threads + 255) / 256;
  if (out.bits == 3)
    hipLaunchKernelGGL(pack_lut_paper_kernel<3>, dim3((unsigned)blocks), dim3(256), 0, s, W, N, N16, K, KC, out.G, g,
                       zl, out.codes, out.scales, out.lut);
  else
    hipLaunchKernelGGL(pack_lut_paper_kernel<2>, dim3((unsigned)blocks), dim3(256), 0, s, W, N, N16, K, KC, out.G, g,
                       zl, out.codes, out.scales, out.lut);
  return hipGetLastError();
}

hipError_t launch_autocast_lut(const LutView& w, const float* G_override, const NvFp4View& out, hipStream_t s) {
  const int64_t N = w.rows, K = w.cols;
  float* tmp = nullptr;
  hipError_t e = hipSuccess;
  if (N * K > 0) {
    e = pool_alloc_async(reinterpret_cast<void**>(&tmp), (size_t)(N * K) * 4, s);
    if (e != hipSuccess) return e;
    const int64_t tiles_c = (K + 127) / 128;
    const int64_t threads = (N + 15) / 16 * tiles_c * 64;
    typedef void (*kern_t)(const uint8_t*, const uint16_t*, const uint8_t*, const float*, int64_t, int64_t, int64_t,
                           float*);
    const kern_t kern = w.bits == 3 ? (w.mode == 0 ? lut_dequant_kernel<3, 0> : lut_dequant_kernel<3, 1>)
                                    : (w.mode == 0 ? lut_dequant_kernel<2, 0> : lut_dequant_kernel<2, 1>);
    hipLaunchKernelGGL(kern, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, w.codes, w.lut, w.scales, w.G,
                       N, K, tiles_c, tmp);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = launch_pack_nvfp4(tmp, N, K, G_override, out, s);
  if (tmp != nullptr) {
    const hipError_t f = hipFreeAsync(tmp, s);
    if (e == hipSuccess) e = f;
  }
  return e;
}

}  // namespace dq
