// NVFP4 quantization kernels (paper App. A, "NVFP4-esque two-level scaling"
// and "NVFP4"): the activation quantizer (bf16 input, static or dynamic
// global scale) and the weight packer (fp32 input, round to nearest).
//
// Both are HBM-bound streaming kernels.  One wavefront owns one 32-row x
// 64-column tile of the tiled NVFP4 layout (dq.h): it reads 32 rows of 64
// elements with fully coalesced 16-byte loads (8 lanes per row), computes the
// per-16 block maxima with one cross-lane exchange, and writes the 1 KiB code
// tile and 128-byte scale tile with contiguous stores.
#include <type_traits>

#include "dq_device.hpp"
#include "dq_internal.hpp"

namespace dq {

// ------------------------------------------------------------ global amax
__global__ void zero_float_kernel(float* p) { *p = 0.0f; }

__global__ void finalize_global_scale_kernel(float* p) {
  float a = *p;
  *p = (a == 0.0f) ? 1.0f : a / kGlobalDivisor;
}

__global__ void copy_float_kernel(const float* src, float* dst) { *dst = *src; }

// Workgroup maximum, then one atomic per workgroup (a few hundred in total).
__device__ inline void block_max_to(float* out, float m) {
  __shared__ float part[4];
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) atomic_max_nonneg(out, fmaxf(fmaxf(part[0], part[1]), fmaxf(part[2], part[3])));
}

template <typename T>
__global__ __launch_bounds__(256) void amax_kernel(const T* __restrict__ x, int64_t n_vec,
                                                   int64_t n, float* out);

// bf16: 8 elements per 16-byte vector
template <>
__global__ __launch_bounds__(256) void amax_kernel<uint16_t>(const uint16_t* __restrict__ x,
                                                             int64_t n_vec, int64_t n, float* out) {
  float m = 0.0f;
  const uint4_t* xv = reinterpret_cast<const uint4_t*>(x);
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n_vec;
       i += (int64_t)gridDim.x * blockDim.x) {
    uint4_t v = __builtin_nontemporal_load(&xv[i]);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      m = fmaxf(m, fabsf(bf16_lo(v[j])));
      m = fmaxf(m, fabsf(bf16_hi(v[j])));
    }
  }
  // tail (n not a multiple of 8)
  for (int64_t i = n_vec * 8 + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    m = fmaxf(m, fabsf(__uint_as_float((uint32_t)x[i] << 16)));
  block_max_to(out, m);
}

// fp32: 4 elements per 16-byte vector
template <>
__global__ __launch_bounds__(256) void amax_kernel<float>(const float* __restrict__ x, int64_t n_vec,
                                                          int64_t n, float* out) {
  float m = 0.0f;
  const float4_t* xv = reinterpret_cast<const float4_t*>(x);
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n_vec;
       i += (int64_t)gridDim.x * blockDim.x) {
    float4_t v = __builtin_nontemporal_load(&xv[i]);
    m = fmaxf(m, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
  }
  for (int64_t i = n_vec * 4 + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    m = fmaxf(m, fabsf(x[i]));
  block_max_to(out, m);
}

// ------------------------------------------------------------ tile quantizer
// Loads 8 consecutive elements of one row as fp32 (zeros when out of range).
__device__ inline void load8(const uint16_t* __restrict__ x, int64_t ld, int64_t row, int64_t col,
                             bool ok, float (&v)[8]) {
  if (ok) {
    uint4_t w = *reinterpret_cast<const uint4_t*>(x + row * ld + col);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[2 * j] = bf16_lo(w[j]);
      v[2 * j + 1] = bf16_hi(w[j]);
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = 0.0f;
  }
}

__device__ inline void load8(const float* __restrict__ x, int64_t ld, int64_t row, int64_t col,
                             bool ok, float (&v)[8]) {
  if (ok) {
    const float4_t* p = reinterpret_cast<const float4_t*>(x + row * ld + col);
    float4_t a = p[0], b = p[1];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = a[j];
      v[4 + j] = b[j];
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = 0.0f;
  }
}

// Quantize 8 values of a 16-block whose other half lives in lane ^ 1.
// Returns the 4 code bytes (element 2j low nibble of byte j) and the scale.
__device__ inline uint32_t quantize8(const float (&v)[8], float G, uint32_t& scale_code) {
  float a = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) a = fmaxf(a, fabsf(v[j]));
  a = fmaxf(a, __shfl_xor(a, 1, 64));
  const float den = 6.0f * G;
  const float t = a / den;                       // correctly rounded division
  const uint32_t c = e4m3_encode_rne_sat(t);
  const float S = e4m3_decode(c) * G;
  scale_code = c;
  if (S == 0.0f) return 0u;
  const float rcp = 1.0f / S;
  uint32_t w = 0;
  w = cvt_pk_fp4<0>(w, div_by_scale(v[0], S, rcp), div_by_scale(v[1], S, rcp));
  w = cvt_pk_fp4<1>(w, div_by_scale(v[2], S, rcp), div_by_scale(v[3], S, rcp));
  w = cvt_pk_fp4<2>(w, div_by_scale(v[4], S, rcp), div_by_scale(v[5], S, rcp));
  w = cvt_pk_fp4<3>(w, div_by_scale(v[6], S, rcp), div_by_scale(v[7], S, rcp));
  return fp4_canonical_zero(w);
}

// One wavefront per 32x64 tile; 4 wavefronts per block.  With NORM the
// loaded values are RMSNorm-ed first: fp32(fp32(x * inv[row]) * gamma[col]).
template <typename T, bool NORM = false>
__global__ __launch_bounds__(256) void quantize_tiles_kernel(const T* __restrict__ x, int64_t rows,
                                                             int64_t cols, const float* __restrict__ Gp,
                                                             uint8_t* __restrict__ codes,
                                                             uint8_t* __restrict__ scales,
                                                             int64_t tiles_r, int64_t tiles_c,
                                                             float* G_out, const float* __restrict__ inv = nullptr,
                                                             const uint16_t* __restrict__ gamma = nullptr) {
  const int lane = threadIdx.x & 63;
  const int64_t tile = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const float G = *Gp;
  if (tile == 0 && lane == 0 && G_out != nullptr) *G_out = G;
  if (tile >= tiles_r * tiles_c) return;
  const int64_t tr = tile / tiles_c, tc = tile % tiles_c;
  const int c = lane & 7;
  const int64_t col = tc * 64 + c * 8;
  const bool col_ok = col < cols;
  uint32_t* code_tile = reinterpret_cast<uint32_t*>(codes + tile * 1024);
  uint8_t* scale_tile = scales + tile * 128;
  // all four row groups' loads first, unconditional from clamped in-bounds
  // addresses (a load under a divergent branch is waited for inside it), then
  // values outside the tensor are masked to zero: one memory round trip per
  // wavefront
  float v[4][8];
  if constexpr (std::is_same<T, uint16_t>::value) {
    const int64_t cc = min(col, cols - 8);   // cols % 16 == 0
    uint4_t w[4];
    float iv[4];
    bool ok[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t row = tr * 32 + 8 * i + (lane >> 3);
      const int64_t rc = min(row, rows - 1);
      ok[i] = col_ok && row < rows;
      w[i] = *reinterpret_cast<const uint4_t*>(x + rc * cols + cc);
      if constexpr (NORM) iv[i] = inv[rc];
    }
    uint4_t gw{0u, 0u, 0u, 0u};
    if constexpr (NORM) gw = *reinterpret_cast<const uint4_t*>(gamma + cc);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float lo = bf16_lo(w[i][j]), hi = bf16_hi(w[i][j]);
        if constexpr (NORM) {   // two roundings, in this order
          lo = (lo * iv[i]) * bf16_lo(gw[j]);
          hi = (hi * iv[i]) * bf16_hi(gw[j]);
        }
        v[i][2 * j] = ok[i] ? lo : 0.0f;
        v[i][2 * j + 1] = ok[i] ? hi : 0.0f;
      }
  } else {
    static_assert(!NORM, "the normalizing quantizer takes bf16 activations");
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t row = tr * 32 + 8 * i + (lane >> 3);
      load8(x, cols, row, col, col_ok && row < rows, v[i]);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 8 * i + (lane >> 3);
    uint32_t sc;
    const uint32_t w = quantize8(v[i], G, sc);
    code_tile[r * 8 + c] = w;
    if ((c & 1) == 0) scale_tile[r * 4 + (c >> 1)] = (uint8_t)sc;
  }
}

// ------------------------------------------------------------ RMSNorm rows
// One wavefront per row: ss = sum of the squares (each exact in fp64) in
// fp64 (lane l takes the 8-element vectors l, l + 64, ...; square t of a
// vector's 4 pairs goes to partial sum t; the four partials are added
// pairwise, then the lanes in a butterfly), ms = fp32(ss / K), inv = fp32(1 / fp32(sqrt(fp32(ms + eps))))
// (correctly rounded square root and division).  With amax != nullptr also
// the maximum |fp32(fp32(x * inv) * gamma)| of the row (dynamic global scale).
__global__ __launch_bounds__(256) void rms_rows_kernel(const uint16_t* __restrict__ x,
                                                       const uint16_t* __restrict__ gamma, float eps, int64_t M,
                                                       int64_t K, float* __restrict__ inv, float* amax) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;   // uniform over the wavefront
  const uint16_t* xr = x + row * K;
  double s4[4] = {0.0, 0.0, 0.0, 0.0};
  for (int64_t k = lane * 8; k < K; k += 512) {   // K % 16 == 0
    const uint4_t w = *reinterpret_cast<const uint4_t*>(xr + k);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const double a = bf16_lo(w[j]), b = bf16_hi(w[j]);
      s4[j] = __builtin_fma(a, a, s4[j]);   // a * a is exact: the same as a rounded add
      s4[j] = __builtin_fma(b, b, s4[j]);
    }
  }
  double ss = (s4[0] + s4[1]) + (s4[2] + s4[3]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off, 64);
  const float ms = (float)(ss / (double)K);
  const float r = ms + eps;
  const float iv = 1.0f / sqrtf(r);
  if (lane == 0) inv[row] = iv;
  if (amax != nullptr) {
    float m = 0.0f;
    for (int64_t k = lane * 8; k < K; k += 512) {
      const uint4_t w = *reinterpret_cast<const uint4_t*>(xr + k);
      const uint4_t g = *reinterpret_cast<const uint4_t*>(gamma + k);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float t0 = bf16_lo(w[j]) * iv, t1 = bf16_hi(w[j]) * iv;
        m = fmaxf(m, fabsf(t0 * bf16_lo(g[j])));
        m = fmaxf(m, fabsf(t1 * bf16_hi(g[j])));
      }
    }
    m = wave_max(m);
    if (lane == 0) atomic_max_nonneg(amax, m);
  }
}

// ------------------------------------------------------------ RMSNorm + quantization, one pass
// For a static global scale and rows of at most 64 * 8 * NV elements (tile-
// padded): one wavefront per row holds the row in registers (lane l: the
// 8-element vectors v = l + 64 j), takes the sum of squares in fp64 in the
// same order and tree as rms_rows_kernel (so `inv` is the same), normalizes
// (gamma staged once per workgroup in LDS),
// and quantizes each 16-block (vectors v and v ^ 1 in lanes l and l ^ 1) into
// the row's slots of the tiled layout: X is read once.  A workgroup of eight
// wavefronts takes eight consecutive rows of one 32-row tile row, so the row
// segments of each tile are written together.  Rows past M and columns past
// K (tile padding) are written as zero codes and scales.
template <int NV>
__global__ __launch_bounds__(512) void rmsnorm_quantize_rows_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ gamma, float eps, int64_t M, int64_t K,
    const float* __restrict__ Gp, uint8_t* __restrict__ codes, uint8_t* __restrict__ scales, int64_t tiles_c,
    float* G_out) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 8 + (threadIdx.x >> 6);
  const float G = *Gp;
  if (blockIdx.x == 0 && threadIdx.x == 0 && G_out != nullptr) *G_out = G;
  const int nvec = (int)(K / 8), nvec_pad = (int)(tiles_c * 8);
  const bool live = row < M;   // uniform over the wavefront
  uint4_t xr[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int v = lane + 64 * j;
    xr[j] = uint4_t{0u, 0u, 0u, 0u};
    if (live && v < nvec) xr[j] = *reinterpret_cast<const uint4_t*>(x + row * K + 8 * (int64_t)v);
  }
  // gamma (zero past K) into LDS once per workgroup: the eight rows share it
  __shared__ uint4_t gsh[64 * 16];
  for (int v = threadIdx.x; v < nvec_pad; v += 512)
    gsh[v] = v < nvec ? *reinterpret_cast<const uint4_t*>(gamma + 8 * v) : uint4_t{0u, 0u, 0u, 0u};
  float iv = 0.0f;
  if (live) {
    double s4[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int j = 0; j < NV; ++j)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const double a = bf16_lo(xr[j][t]), b = bf16_hi(xr[j][t]);
        s4[t] = __builtin_fma(a, a, s4[t]);   // a * a is exact: the same as a rounded add
        s4[t] = __builtin_fma(b, b, s4[t]);
      }
    double ss = (s4[0] + s4[1]) + (s4[2] + s4[3]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off, 64);
    const float ms = (float)(ss / (double)K);
    const float r = ms + eps;
    iv = 1.0f / sqrtf(r);
  }
  __syncthreads();
  const int64_t tr = row / 32, rr = row % 32;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int v = lane + 64 * j;
    if (64 * j >= nvec_pad) break;            // uniform: no vector of this j in the padded row
    float f[8];
    const uint4_t gw = v < nvec_pad ? gsh[v] : uint4_t{0u, 0u, 0u, 0u};
#pragma unroll
    for (int t = 0; t < 4; ++t) {     // two roundings, in this order (zeros stay zero)
      f[2 * t] = (bf16_lo(xr[j][t]) * iv) * bf16_lo(gw[t]);
      f[2 * t + 1] = (bf16_hi(xr[j][t]) * iv) * bf16_hi(gw[t]);
    }
    uint32_t sc;
    const uint32_t w = quantize8(f, G, sc);   // every lane takes part in the pair exchange
    // the scales of the tile row's four 16-blocks, gathered in the lane with v % 8 == 0
    const uint32_t s2 = (uint32_t)__shfl((int)sc, lane + 2, 64);
    const uint32_t s4 = (uint32_t)__shfl((int)sc, lane + 4, 64);
    const uint32_t s6 = (uint32_t)__shfl((int)sc, lane + 6, 64);
    if (v < nvec_pad) {
      const int64_t tile = tr * tiles_c + v / 8;
      *reinterpret_cast<uint32_t*>(codes + tile * 1024 + rr * 32 + 4 * (v % 8)) = w;
      if ((v & 7) == 0)
        *reinterpret_cast<uint32_t*>(scales + tile * 128 + rr * 4) = sc | (s2 << 8) | (s4 << 16) | (s6 << 24);
    }
  }
}

// ------------------------------------------------------------ launchers
static int grid_for(int64_t n_vec) {
  int64_t b = (n_vec + 255) / 256;
  if (b > 1024) b = 1024;
  if (b < 1) b = 1;
  return (int)b;
}

template <typename T>
static hipError_t launch_amax(const T* x, int64_t n, float* out, hipStream_t s) {
  const int64_t per_vec = 16 / sizeof(T);
  const int64_t n_vec = n / per_vec;
  hipLaunchKernelGGL(zero_float_kernel, dim3(1), dim3(1), 0, s, out);
  hipLaunchKernelGGL(amax_kernel<T>, dim3(grid_for(n_vec)), dim3(256), 0, s, x, n_vec, n, out);
  hipLaunchKernelGGL(finalize_global_scale_kernel, dim3(1), dim3(1), 0, s, out);
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_quantize(const T* x, int64_t rows, int64_t cols, const float* Gp,
                                  const NvFp4View& out, hipStream_t s) {
  const int64_t tiles_r = round_up(rows, 32) / 32, tiles_c = round_up(cols, 64) / 64;
  const int64_t tiles = tiles_r * tiles_c;
  if (tiles == 0) {
    if (Gp != out.G) hipLaunchKernelGGL(copy_float_kernel, dim3(1), dim3(1), 0, s, Gp, out.G);
    return hipGetLastError();
  }
  const int64_t blocks = (tiles + 3) / 4;
  hipLaunchKernelGGL(quantize_tiles_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, s, x, rows, cols,
                     Gp, out.codes, out.scales, tiles_r, tiles_c, Gp == out.G ? nullptr : out.G);
  return hipGetLastError();
}

hipError_t launch_quantize_act(const uint16_t* X, int64_t M, int64_t K, const float* G_static,
                               const NvFp4View& out, hipStream_t s) {
  if (G_static == nullptr) {
    hipError_t e = launch_amax(X, M * K, out.G, s);
    if (e != hipSuccess) return e;
    return launch_quantize(X, M, K, out.G, out, s);
  }
  return launch_quantize(X, M, K, G_static, out, s);
}

hipError_t launch_rmsnorm_quantize_act(const uint16_t* X, const uint16_t* gamma, float eps, int64_t M, int64_t K,
                                       const float* G_static, const NvFp4View& out, void* ws, hipStream_t s) {
  const int64_t tiles_r = round_up(M, 32) / 32, tiles_c = round_up(K, 64) / 64;
  if (M == 0 || K == 0) {   // nothing to normalize: an all-zero tensor (G = 1 when dynamic)
    if (G_static == nullptr) {
      hipLaunchKernelGGL(zero_float_kernel, dim3(1), dim3(1), 0, s, out.G);
      hipLaunchKernelGGL(finalize_global_scale_kernel, dim3(1), dim3(1), 0, s, out.G);
      return launch_quantize(X, M, K, out.G, out, s);
    }
    return launch_quantize(X, M, K, G_static, out, s);
  }
  if (G_static != nullptr && tiles_c * 8 <= 64 * 16) {
    // one pass: the row lives in registers (at most 16 vectors of 8 per lane)
    const int nv = (int)((tiles_c * 8 + 63) / 64);
    typedef void (*kern_t)(const uint16_t*, const uint16_t*, float, int64_t, int64_t, const float*, uint8_t*,
                           uint8_t*, int64_t, float*);
    static const kern_t kerns[16] = {
        rmsnorm_quantize_rows_kernel<1>,  rmsnorm_quantize_rows_kernel<2>,  rmsnorm_quantize_rows_kernel<3>,
        rmsnorm_quantize_rows_kernel<4>,  rmsnorm_quantize_rows_kernel<5>,  rmsnorm_quantize_rows_kernel<6>,
        rmsnorm_quantize_rows_kernel<7>,  rmsnorm_quantize_rows_kernel<8>,  rmsnorm_quantize_rows_kernel<9>,
        rmsnorm_quantize_rows_kernel<10>, rmsnorm_quantize_rows_kernel<11>, rmsnorm_quantize_rows_kernel<12>,
        rmsnorm_quantize_rows_kernel<13>, rmsnorm_quantize_rows_kernel<14>, rmsnorm_quantize_rows_kernel<15>,
        rmsnorm_quantize_rows_kernel<16>};
    hipLaunchKernelGGL(kerns[nv - 1], dim3((unsigned)(tiles_r * 4)), dim3(512), 0, s, X, gamma, eps, M, K, G_static,
                       out.codes, out.scales, tiles_c, G_static == out.G ? nullptr : out.G);
    return hipGetLastError();
  }
  float* inv = reinterpret_cast<float*>(ws);
  const bool pooled = inv == nullptr;
  hipError_t e = hipSuccess;
  if (pooled) {
    e = pool_alloc_async(reinterpret_cast<void**>(&inv), (size_t)M * 4, s);
    if (e != hipSuccess) return e;
  }
  const float* Gp = G_static;
  if (G_static == nullptr) {
    hipLaunchKernelGGL(zero_float_kernel, dim3(1), dim3(1), 0, s, out.G);
    hipLaunchKernelGGL(rms_rows_kernel, dim3((unsigned)((M + 3) / 4)), dim3(256), 0, s, X, gamma, eps, M, K, inv,
                       out.G);
    hipLaunchKernelGGL(finalize_global_scale_kernel, dim3(1), dim3(1), 0, s, out.G);
    Gp = out.G;
  } else {
    hipLaunchKernelGGL(rms_rows_kernel, dim3((unsigned)((M + 3) / 4)), dim3(256), 0, s, X, gamma, eps, M, K, inv,
                       nullptr);
  }
  const int64_t blocks = (tiles_r * tiles_c + 3) / 4;
  hipLaunchKernelGGL((quantize_tiles_kernel<uint16_t, true>), dim3((unsigned)blocks), dim3(256), 0, s, X, M, K, Gp,
                     out.codes, out.scales, tiles_r, tiles_c, Gp == out.G ? nullptr : out.G, inv, gamma);
  e = hipGetLastError();
  if (pooled) {
    const hipError_t f = hipFreeAsync(inv, s);
    if (e == hipSuccess) e = f;
  }
  return e;
}

hipError_t launch_global_scale_f32(const float* x, int64_t n, float* G, hipStream_t s) {
  return launch_amax(x, n, G, s);
}

hipError_t launch_pack_nvfp4(const float* W, int64_t N, int64_t K, const float* G_override,
                             const NvFp4View& out, hipStream_t s) {
  if (G_override == nullptr) {
    hipError_t e = launch_amax(W, N * K, out.G, s);
    if (e != hipSuccess) return e;
    return launch_quantize(W, N, K, out.G, out, s);
  }
  return launch_quantize(W, N, K, G_override, out, s);
}

}  // namespace dq
