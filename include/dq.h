/*
 * dq.h - C ABI of the MI355X (gfx950) hot path of disaggregated quantization:
 * the phase-specific quantized linear layer (arXiv 2609.26333, Sec. 2.3
 * "Format disaggregation"; App. A "Quantization formats"; App. C).
 *
 *   prefill:  dq_quantize_act_nvfp4 -> dq_prefill_gemm   (W4A4 NVFP4)
 *   decode:   dq_decode_gemv                              (weight-only LUT, bf16 x)
 *   offline:  dq_pack_nvfp4, dq_pack_lut3                 (weight packing)
 *
 * Conventions for every call
 *   - Buffers are device memory owned by the caller.  The library keeps no
 *     state except a thread-local last-error string and a per-device memory
 *     pool.  Calls that need scratch memory take a caller workspace (with a
 *     size query): dq_prefill_gemm's fused path, dq_decode_gemv,
 *     dq_decode_gemv_nvfp4 and dq_rmsnorm_quantize_act_nvfp4.  Given a
 *     workspace they allocate nothing; given NULL they take stream-ordered
 *     staging from the pool (hipMallocFromPoolAsync / hipFreeAsync on the
 *     call's stream).  dq_autocast_lut_to_nvfp4 (an offline, load-time step)
 *     always takes its fp32 staging from the pool.  No other call allocates.
 *   - Calls are asynchronous on `stream` (a hipStream_t passed as void*;
 *     NULL is the default stream).  Nothing synchronizes inside the library.
 *   - Arguments are validated on the host before any HIP call; a rejected
 *     call launches nothing and returns DQ_ERR_INVALID_ARG or
 *     DQ_ERR_UNSUPPORTED.  A failed launch returns DQ_ERR_HIP.  Faults during
 *     execution surface at the caller's next synchronization.
 *   - Device pointers must be 16-byte aligned (scalar fp32 pointers: 4-byte).
 *   - Inputs must be finite; results for non-finite inputs are unspecified
 *     (no crash).
 *   - Descriptor structs (dq_nvfp4_t, dq_lut_t) are host memory read during
 *     the call only.
 */
#ifndef DQ_H
#define DQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DQ_ABI_VERSION 3

typedef int32_t dq_status;
#define DQ_OK 0
#define DQ_ERR_INVALID_ARG (-1) /* null/misaligned pointer, bad size or enum */
#define DQ_ERR_UNSUPPORTED (-2) /* valid request the library does not implement */
#define DQ_ERR_HIP (-3)         /* a HIP launch failed; see dq_last_error() */

/* Output element kinds. */
#define DQ_OUT_F32 0
#define DQ_OUT_BF16 1
#define DQ_OUT_NVFP4 2

/* LUT modes. */
#define DQ_LUT_PER_ROW 0    /* one 2^bits-entry fp16 table per output row */
#define DQ_LUT_PAPER_GRID 1 /* fixed grid + signed E4M3 per 16 + fp32 global scale */

/* GEMM epilogue flags. */
#define DQ_EPI_SWIGLU 1

/*
 * NVFP4 tensor (App. A, "NVFP4-esque two-level scaling", "NVFP4").
 * Logical content: rows x cols E2M1 codes (code = sign << 3 | index into
 * {0, .5, 1, 1.5, 2, 3, 4, 6}; a zero magnitude has sign 0), one E4M3 scale
 * per 16 consecutive columns of a row, one fp32 global scale G.  Element
 * value = e2m1(code) * e4m3(scale) * G.  Columns are the contraction
 * dimension K.
 *
 * Physical layout ("32x64 tiles").  Let R32 = rows rounded up to 32 and
 * C64 = cols rounded up to 64.  Padding elements hold code 0 and scale 0.
 *   codes:  R32*C64/2 bytes, tiles of 32 rows x 64 cols stored tile-row-major:
 *           tile (tr, tc) starts at byte (tr*(C64/64) + tc) * 1024; inside it
 *           row r (0..31) occupies bytes r*32 .. r*32+31 and byte j holds
 *           column tc*64 + 2j in its low nibble and column tc*64 + 2j + 1 in
 *           its high nibble.
 *   scales: R32*C64/16 bytes, tile (tr, tc) starts at (tr*(C64/64) + tc) * 128;
 *           row r, block b (0..3, columns tc*64 + 16b ..) is byte r*4 + b.
 *   G:      one float.
 */
typedef struct dq_nvfp4 {
  uint8_t* codes;
  uint8_t* scales;
  float* G;
  int64_t rows;
  int64_t cols;
} dq_nvfp4_t;

/*
 * LUT weight (decode side; App. A "LUT formats" for PAPER_GRID; PER_ROW is
 * the per-row equal-count table of the benchmark workloads).
 * Logical content: rows x cols codes in [0, 2^bits).  Weight value:
 *   PER_ROW:    lut[row * 2^bits + code]                       (fp16 table)
 *   PAPER_GRID: grid[code] * e4m3(scale[row, col/16]) * G      (signed scale)
 *
 * Physical layout ("16x128 tiles").  Let R16 = rows rounded up to 16 and
 * C128 = cols rounded up to 128; padding codes are 0 and padding table
 * entries / scales are 0.
 *   codes:  tile (tr, c) = rows 16tr..16tr+15, cols 128c..128c+127, stored at
 *           byte (tr*(C128/128) + c) * 64 * G where G = 12 (bits 3) or 8
 *           (bits 2) bytes per group.  Group g = q*16 + i (i = row in tile,
 *           q = 0..3) holds the 32 codes of columns 128c + 32q + t, t = 0..31.
 *           With s = t/4 and b = t%4, code t sits in little-endian dword w of
 *           the group:
 *             bits 3: s=0..5 -> dword s/2, bits [8b + 3(s%2), +3);
 *                     s=6    -> dword 0 bits [8b+6, 8b+8) (low 2 bits) and
 *                               dword 2 bit 8b+6 (high bit);
 *                     s=7    -> dword 1 bits [8b+6, 8b+8) and dword 2 bit 8b+7.
 *             bits 2: dword s/4, bits [8b + 2(s%4), +2).
 *   lut:    PER_ROW: R16 * 2^bits fp16 (uint16 bit patterns), row-major.
 *           PAPER_GRID: 2^bits fp16, ascending, containing one 0.
 *   scales: PAPER_GRID only (NULL for PER_ROW): tile (tr, c) at byte
 *           (tr*(C128/128) + c) * 128; group g = q*16 + i holds 2 bytes at
 *           g*2: the signed E4M3 scales of column blocks 128c + 32q + 0..15
 *           and + 16..31 of row 16tr + i.
 *   G:      PAPER_GRID only: one float.
 */
typedef struct dq_lut {
  uint8_t* codes;
  uint16_t* lut;
  uint8_t* scales;
  float* G;
  int64_t rows;
  int64_t cols;
  int32_t bits;
  int32_t mode;
} dq_lut_t;

/*
 * MXFP4 tensor (OCP Microscaling: the W4A4 format the paper runs for models
 * released natively in MXFP4, Sec. 3.2).  Logical content: rows x cols E2M1
 * codes (as NVFP4) and one E8M0 scale code per 32 consecutive columns of a
 * row; element value = e2m1(code) * 2^(scale - 127).  No tensor scale.
 *
 * Physical layout ("32x64 tiles"; R32, C64 as for NVFP4, R128 = rows rounded
 * up to 128; padding elements hold code 0 and scale code 0):
 *   codes:  as NVFP4 codes (R32*C64/2 bytes).
 *   scales: R128*C64/32 bytes in groups of 4 row tiles: group (g, tc) (rows
 *           128g .. 128g+127, columns tc*64 .. +63) starts at
 *           (g*(C64/64) + tc) * 256; byte 4*(r + 32h) + q is the scale of row
 *           128g + 32q + r, columns tc*64 + 32h .. +31.
 */
typedef struct dq_mxfp4 {
  uint8_t* codes;
  uint8_t* scales;
  int64_t rows;
  int64_t cols;
} dq_mxfp4_t;

/* ---- diagnostics -------------------------------------------------------- */
int dq_abi_version(void);
const char* dq_status_string(dq_status s);
/* Message of the last failing call on this thread ("" if none). */
const char* dq_last_error(void);

/* ---- size queries (host only) ------------------------------------------- */
/* Bytes of the codes and scales buffers of a rows x cols MXFP4 tensor
 * (cols % 32 == 0, rows >= 0). */
dq_status dq_mxfp4_sizes(int64_t rows, int64_t cols, size_t* code_bytes, size_t* scale_bytes);

/* Bytes of the codes and scales buffers of a rows x cols NVFP4 tensor
 * (cols % 16 == 0, rows >= 0). */
dq_status dq_nvfp4_sizes(int64_t rows, int64_t cols, size_t* code_bytes, size_t* scale_bytes);
/* Bytes of the codes, lut and scales buffers of a LUT weight
 * (bits 2 or 3; cols % 32 == 0).  scale_bytes is 0 for PER_ROW. */
dq_status dq_lut_sizes(int bits, int mode, int64_t rows, int64_t cols, size_t* code_bytes,
                       size_t* lut_bytes, size_t* scale_bytes);

/* ---- a2: weight packing, NVFP4 (App. A "NVFP4"; round to nearest) --------
 * W: device fp32 [N, K] row-major (K contiguous), K % 16 == 0.
 * G_override: device float or NULL.  NULL -> G = fp32(max|W| / 2688) is
 *   computed on the device (1 if W is all zero).  Non-NULL -> that G is used,
 *   e.g. the shared scale of a fused projection group.
 * out: rows = N, cols = K, buffers sized by dq_nvfp4_sizes; out->G receives G.
 * Per block of 16: t = fp32(max|w| / fp32(6G)); scale = E4M3(t) (nearest,
 * ties to even, saturating at 448); S = fp32(e4m3 * G); codes =
 * E2M1(fp32(w / S)) (nearest, ties to even, |y| >= 6 -> 6); S == 0 -> codes 0. */
dq_status dq_pack_nvfp4(const float* W, int64_t N, int64_t K, const float* G_override,
                        const dq_nvfp4_t* out, void* stream);

/* ---- a5: weight packing, LUT (bits 3 = LUT3, bits 2 = LUT2) --------------
 * W: device fp32 [N, K] row-major, K % 32 == 0.
 * PER_ROW: each row is sorted, cut into 2^bits equal-count bins; entry j =
 *   fp16(round-to-nearest-even of fp64(sum of bin j) / count); code =
 *   #{j : w > (L_j + L_{j+1}) / 2} (nearest entry, ties to the lower index).
 *   K <= 32768 (the row is sorted in LDS); larger K -> DQ_ERR_UNSUPPORTED.
 * PAPER_GRID (App. A "LUT formats"): grid = host pointer to 2^bits fp16
 *   values (ascending, one exactly 0) or NULL for the paper's grid rounded to
 *   fp16; G = fp32(max|W| / 2688); per block of 16 the largest |w| (lowest k
 *   on ties) sets d = sign(w*) * E4M3(fp32(|w*| / fp32(6G))), S = fp32(d G);
 *   code = nearest grid level of fp32(w / S) (ties to the lower level);
 *   S == 0 -> the zero level.
 * out: rows = N, cols = K, bits, mode set by the caller; buffers sized by
 *   dq_lut_sizes (PER_ROW: scales and G may be NULL). */
dq_status dq_pack_lut3(const float* W, int64_t N, int64_t K, int bits, int mode,
                       const uint16_t* grid, const dq_lut_t* out, void* stream);

/* ---- a1: activation quantization to NVFP4 --------------------------------
 * X: device bf16 [M, K] row-major (uint16 bit patterns), K % 16 == 0.
 * G_static: device float or NULL.  Non-NULL: the static per-tensor input
 *   scale of a running-maximum observer (App. A "NVFP4"); values beyond it
 *   saturate.  NULL: dynamic, G = fp32(max|X| / 2688) from an extra pass.
 * out: rows = M, cols = K; out->G receives the G used.  Same block rule as
 * dq_pack_nvfp4. */
dq_status dq_quantize_act_nvfp4(const uint16_t* X, int64_t M, int64_t K, const float* G_static,
                                const dq_nvfp4_t* out, void* stream);

/* ---- a3 (+a1 fused, +a4): W4A4 NVFP4 GEMM --------------------------------
 * The prefill projection of the W4A4 NVFP4 format (App. A "Quantization
 * formats", NVFP4: activations quantized with a static per-tensor input
 * scale; App. C "Prefill measurements", compute and timing scope: the
 * quantized projections with their activation processing fused):
 *   Y[m, n] = G_a * G_w * sum_k a[m, k] * w[n, k]
 * over the dequantized NVFP4 operands (exact products, fp32 accumulation).
 * A: quantized activations (rows = M, cols = K) - or NULL together with
 *   X (device bf16 [M, K]) and G_x_static (device float): the activations are
 *   then quantized with the static scale as part of this call (fused a1), by
 *   one streaming pass into an NVFP4 copy that the GEMM reads.  That copy
 *   lives in `workspace` (at least dq_prefill_gemm_workspace_size(M, K)
 *   bytes, 16-byte aligned, not in use by other work while the call runs on
 *   `stream`); with workspace == NULL it is taken from the library's pool,
 *   stream-ordered.  Exactly one of A and X must be given (with M == 0 the
 *   fused call may pass X = NULL).  The unfused call ignores the workspace.
 * W: packed weights, rows = N, cols = K (same K as A).
 * out_kind DQ_OUT_F32 / DQ_OUT_BF16: Y is device [M, N] row-major fp32 / bf16
 *   (bf16: round to nearest even).
 * out_kind DQ_OUT_NVFP4 (a4): the fp32 result is quantized along N in blocks
 *   of 16 with the static scale *G_out_static into Yq (rows = M, cols = N, or
 *   N/2 with DQ_EPI_SWIGLU); Y must be NULL.
 * epilogue_flags DQ_EPI_SWIGLU: W rows are interleaved gate/up in groups of
 *   16 (rows 32j..32j+15 = gate rows 16j.., rows 32j+16..32j+31 = up rows
 *   16j..); the output column j = silu(gate_j) * up_j, N/2 columns.
 * K % 16 == 0, M >= 0, N >= 0; K < 2^23 (the kernel addresses a row panel of
 * each operand with 32-bit offsets; larger K -> DQ_ERR_UNSUPPORTED). */
dq_status dq_prefill_gemm_workspace_size(int64_t M, int64_t K, size_t* bytes);
dq_status dq_prefill_gemm(const dq_nvfp4_t* A, const uint16_t* X, const float* G_x_static,
                          const dq_nvfp4_t* W, int64_t M, int out_kind, void* Y,
                          const float* G_out_static, const dq_nvfp4_t* Yq, int epilogue_flags,
                          void* workspace, size_t workspace_bytes, void* stream);

/* ---- RMSNorm fused with the NVFP4 activation quantizer -------------------
 * The paper quantizes activations inside the normalization that feeds the
 * quantized projections (App. C, "Prefill measurements").  Per row of the
 * bf16 X [M, K]: ss = sum of x^2 (fp64), ms = fp32(ss / K),
 * inv = fp32(1 / fp32(sqrt(fp32(ms + eps)))), y = fp32(fp32(x * inv) * gamma)
 * with gamma device bf16 [K] (16-byte aligned); y is then quantized by the
 * a1 rule of dq_quantize_act_nvfp4 (G_static, or G = amax(y) / 2688 when
 * NULL).  out: rows = M, cols = K.  With a static scale and K <= 8192 the
 * call is one pass over X (each row normalized and quantized from registers)
 * and uses no workspace; otherwise the per-row statistics go to `workspace`:
 * device memory of at least 4 M bytes (16-byte aligned), not in use by other
 * work during the call; NULL takes it from the library's pool,
 * stream-ordered.  eps must be finite, >= 0. */
dq_status dq_rmsnorm_quantize_act_nvfp4(const uint16_t* X, const uint16_t* gamma, float eps, int64_t M,
                                        int64_t K, const float* G_static, const dq_nvfp4_t* out,
                                        void* workspace, size_t workspace_bytes, void* stream);

/* ---- LUT -> NVFP4 autocast ----------------------------------------------
 * The re-quantization of LUT weights to NVFP4 for native low-precision
 * prefill (Sec. 2.3: "autocast").  The dequantized LUT weight (PER_ROW: the
 * fp16 table entry; PAPER_GRID: fp32(grid * e4m3) * G, one rounding) is
 * packed by the NVFP4 weight rule of dq_pack_nvfp4 (G = amax / 2688 unless
 * G_override is given).  out: rows, cols as W.  The fp32 staging copy of the
 * weight (rows * cols * 4 bytes) is taken from the library's pool,
 * stream-ordered. */
dq_status dq_autocast_lut_to_nvfp4(const dq_lut_t* W, const float* G_override, const dq_nvfp4_t* out,
                                   void* stream);

/* ---- NVFP4A16 decode GEMV ------------------------------------------------
 * The weight-only NVFP4 decode of format disaggregation (Sec. 2.3: decode
 * keeps 16-bit activations and quantizes only the weights; App. A "NVFP4"):
 * y[b, n] = sum_k x[b, k] * w_hat[n, k], w_hat = e2m1 * e4m3(scale) * G.
 * x: device bf16 [B, K] row-major, 1 <= B <= 16.  W: NVFP4 weights as packed
 * by dq_pack_nvfp4 (rows = N, cols = K).  out_kind DQ_OUT_F32 / DQ_OUT_BF16:
 * y is device [B, N] row-major; x 16-byte aligned.  Small batches (B <= 8,
 * row tiles of 32 that fit one resident round of workgroups, B * K within
 * the staging limit) run in one launch that splits K inside each workgroup
 * and needs no workspace (dq_decode_gemv_nvfp4_workspace_size reports 0);
 * otherwise
 * workspace / workspace_bytes are as for dq_decode_gemv (partial sums over K
 * groups; NULL takes stream-ordered memory from the library's pool).
 * Activations are staged as fp16 after a power-of-two rescale per batch row
 * and K slice (the conversion described for dq_decode_gemv); weight products
 * are exact, sums fp32. */
dq_status dq_decode_gemv_nvfp4_workspace_size(int64_t B, const dq_nvfp4_t* W, size_t* bytes);
dq_status dq_decode_gemv_nvfp4(const uint16_t* x, int64_t B, const dq_nvfp4_t* W, int out_kind, void* y,
                               void* workspace, size_t workspace_bytes, void* stream);

/* ---- MXFP4 W4A4 prefill variant ------------------------------------------
 * Quantization of a 32-block with largest magnitude a (OCP MX conversion):
 * e = floor(log2 a) - 2, clamped to [-127, 127] (-127 for an all-zero block),
 * scale code e + 127, codes = E2M1(x * 2^-e) nearest-even with saturation at
 * 6, magnitude-zero codes with sign 0.
 * dq_pack_mxfp4: W device fp32 [N, K] row-major, K % 32 == 0; out rows = N,
 *   cols = K, buffers sized by dq_mxfp4_sizes.
 * dq_quantize_act_mxfp4: X device bf16 [M, K]; same rule.
 * dq_prefill_gemm_mxfp4: Y[m, n] = sum_k a_hat[m, k] * w_hat[n, k] with the
 *   block scales applied inside the matrix cores and fp32 accumulation;
 *   A rows = M, cols = K; W rows = N, cols = K (K = 0 gives Y = 0);
 *   out_kind DQ_OUT_F32 / DQ_OUT_BF16, Y device [M, N] row-major; K < 2^23
 *   (32-bit row-panel offsets; larger K -> DQ_ERR_UNSUPPORTED). */
dq_status dq_pack_mxfp4(const float* W, int64_t N, int64_t K, const dq_mxfp4_t* out, void* stream);
dq_status dq_quantize_act_mxfp4(const uint16_t* X, int64_t M, int64_t K, const dq_mxfp4_t* out,
                                void* stream);
dq_status dq_prefill_gemm_mxfp4(const dq_mxfp4_t* A, const dq_mxfp4_t* W, int out_kind, void* Y,
                                void* stream);

/* ---- a6: weight-only LUT GEMV (decode; no activation quantization) -------
 * The weight-only path the paper serves decode with (Sec. 2.3, format
 * disaggregation; time set by the weight bytes streamed per token, App. C
 * "Kernel specification").
 * y[b, n] = sum_k x[b, k] * w_hat[n, k], fp32 accumulation.
 * x: device bf16 [B, K] row-major, 1 <= B <= 16.  W: packed LUT weight.
 * out_kind DQ_OUT_F32 / DQ_OUT_BF16: y is device [B, N] row-major.
 * workspace: device memory of at least dq_decode_gemv_workspace_size() bytes
 *   (16-byte aligned), used for split-K partial sums when B >= 2; it must not
 *   be in use by other work while the call runs on `stream`.  NULL: the
 *   library takes it from its own pool, stream-ordered (costs ~10 us of host
 *   time per call).  workspace_bytes below the required size is rejected.
 * Activations are converted to fp16 inside the kernel after a power-of-two
 * rescale from the largest magnitude of the slice of x that one wavefront
 * (B = 1) or one K group of a batch row (B >= 2) reads; a bf16 value is
 * converted exactly unless it lies more than 2^31 below that magnitude (it
 * then becomes an fp16 subnormal, truncated toward zero: an error below 2^-38
 * of the magnitude).  Products with the fp16 table are exact; partial sums
 * are scaled back by the same power of two.  In PAPER_GRID mode the product
 * grid[code] * e4m3(scale) (up to 15 significant bits) is rounded once to an
 * fp16 operand: each weight carries a relative error of at most 2^-11. */
dq_status dq_decode_gemv_workspace_size(int64_t B, const dq_lut_t* W, size_t* bytes);
dq_status dq_decode_gemv(const uint16_t* x, int64_t B, const dq_lut_t* W, int out_kind, void* y,
                         void* workspace, size_t workspace_bytes, void* stream);

/* ---- a6 without allocation -----------------------------------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid it): dq_decode_gemv
 * with its split-K partial sums in a static scratch array of the library
 * (DQ_NOALLOC_SCRATCH_BYTES per GPU, held by each GPU the library runs on
 * until the process ends) instead of a workspace.  Same arguments, kernels
 * and results as dq_decode_gemv; it calls no allocator.  A call whose partial
 * sums exceed the scratch (dq_decode_gemv_workspace_size() above
 * DQ_NOALLOC_SCRATCH_BYTES) is rejected with DQ_ERR_UNSUPPORTED before any
 * GPU work.  Every call on one GPU shares that GPU's scratch: calls that
 * overlap in time on one GPU (different streams, or different threads
 * without ordering) race and give undefined results. */
#define DQ_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
dq_status dq_decode_gemv_noalloc(const uint16_t* x, int64_t B, const dq_lut_t* W, int out_kind, void* y,
                                 void* stream);

#ifdef __cplusplus
}
#endif
#endif /* DQ_H */
