/*
 * reqat.h -- C ABI of libreqat, the microscaled-FP4 linear layer for AMD
 * Instinct MI355X (gfx950).
 *
 * The operations are those of the W4A4 linear layer of ReQAT (QAT of large
 * reasoning models with FP4 weights and activations):
 *   - block quantization of bfloat16 tensors to E2M1 codes with per-block
 *     scales, in the two microscaled formats of App. A, Tab. mx_configs:
 *       MXFP4: E2M1 elements, one E8M0 scale per 32 elements, no global scale;
 *       NVFP4: E2M1 elements, one E4M3 scale per 16 elements, plus one FP32
 *              global (tensor) scale;
 *   - the quantize-dequantize ("fake-quant", simulated quantization noise,
 *     Sec. 2.2 and Sec. 4 Stage-2 QAT) forward, emitting bfloat16;
 *   - the block-scaled FP4 x FP4 product with FP32 accumulation that the
 *     quantized weights and activations feed (the 4-bit GEMM of Sec. 5.3).
 *
 * Numerics (the paper names the formats only; these are the library's rules):
 *   - Blocks run along the contiguous dimension (the reduction dimension K of
 *     the product), for activations X[M][K] and weights W[N][K] alike.
 *   - Block scale: the smallest representable scale s with
 *     block_absmax <= 6 * s * g (g = 1 for MXFP4), so no element clips.
 *     A block of zeros gets scale byte 0x00.  NVFP4 with a caller-given g so
 *     small that even s = 448 fails: s = 448 and elements saturate at +-6.
 *   - Element code: round to nearest, ties to the even code, of the exact
 *     quotient |x| / (s * g), saturating at 6; the sign bit of x is copied
 *     (so -0 and tiny negatives give code 0x8).
 *   - Computed NVFP4 global scale (REQAT_TS_COMPUTE): g = 2^k with k the
 *     smallest integer >= -126 such that tensor_absmax <= 6 * 448 * 2^k
 *     (absmax over finite values; g = 1 for a tensor with none nonzero).
 *   - A block containing NaN or Inf: scale byte NaN (MXFP4 0xFF, NVFP4 0x7F),
 *     codes 0; fake-quant writes bfloat16 NaN (0x7FC0) for that block, and
 *     the product propagates NaN.
 *   - E4M3 is the OCP "E4M3FN" encoding (bias 7, max 448, NaN 0x7F/0xFF).
 *   - Fake-quant output: the dequantized value code * s * g rounded once to
 *     bfloat16 (nearest, ties to even).
 *
 * Layouts (all row-major, all pointers DEVICE pointers unless stated):
 *   x      : bfloat16 [rows][ldx], the first `cols` of each row are used.
 *   codes  : uint8 [rows][cols/2]; element 2i in bits 3:0 of byte i,
 *            element 2i+1 in bits 7:4.
 *   scales : uint8 [rows][cols/B], B = 16 (NVFP4) or 32 (MXFP4).
 *   tensor_scale : one float (NVFP4 only); NULL for MXFP4.
 *   y (product): [M][ldy] float32 or bfloat16 (round to nearest even).
 *
 * Ownership and concurrency: the caller allocates and frees every buffer;
 * the library allocates nothing.  Its only global state is set up once per
 * device and read afterwards: a cache of the device's compute-unit count, and
 * the device address of the fixed scratch array of reqat_linear_w4a4_noalloc
 * (whose contents every such call on that device shares).  Every call only
 * enqueues work on `stream` (a hipStream_t passed as void*; NULL means the
 * null stream; it must belong to the current device) and returns without
 * waiting.  Calls on different streams that share a workspace race.
 *
 * Errors: arguments are validated on the host before any HIP call; a bad
 * argument returns a status != REQAT_OK and enqueues nothing.  A failed
 * launch returns REQAT_E_HIP.  Faults during execution surface at the
 * caller's next synchronisation of `stream`.
 */
#ifndef REQAT_H
#define REQAT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define REQAT_ABI_VERSION 11

/* The enums travel as C ints.  Compiled as C++ they get int as their fixed
 * underlying type, so any int a caller passes is a value the library may
 * read and reject (REQAT_E_ENUM) without undefined behaviour. */
#ifdef __cplusplus
#define REQAT_ENUM(tag) enum tag : int
#else
#define REQAT_ENUM(tag) enum tag
#endif

typedef REQAT_ENUM(reqat_format_e) {
    REQAT_FMT_NVFP4 = 0, /* B = 16, E4M3 block scale, FP32 global scale */
    REQAT_FMT_MXFP4 = 1  /* B = 32, E8M0 block scale */
} reqat_format;

typedef REQAT_ENUM(reqat_dtype_e) {
    REQAT_DT_F32 = 0,
    REQAT_DT_BF16 = 1
} reqat_dtype;

typedef REQAT_ENUM(reqat_tscale_mode_e) {
    REQAT_TS_COMPUTE = 0, /* library computes g from the tensor and writes *tensor_scale */
    REQAT_TS_GIVEN = 1    /* *tensor_scale holds the caller's g (finite, > 0) */
} reqat_tscale_mode;

typedef REQAT_ENUM(reqat_status_e) {
    REQAT_OK = 0,
    REQAT_E_NULL = 1,        /* a required pointer is NULL */
    REQAT_E_SHAPE = 2,       /* negative size, cols/K not a multiple of the block, ld too small */
    REQAT_E_ALIGN = 3,       /* a pointer or leading dimension breaks the alignment rule */
    REQAT_E_ENUM = 4,        /* unknown format, dtype or tensor-scale mode */
    REQAT_E_UNSUPPORTED = 5, /* valid but not implemented (e.g. MXFP4 with a tensor scale) */
    REQAT_E_HIP = 6,         /* a HIP launch failed */
    REQAT_E_TOO_LARGE = 7    /* beyond the fixed scratch of reqat_linear_w4a4_noalloc */
} reqat_status;

/*
 * Quantize x[rows][cols] (App. A, Tab. mx_configs; element rounding and
 * scale rule as above).
 *   fmt          : REQAT_FMT_NVFP4 or REQAT_FMT_MXFP4.
 *   x, ldx       : bfloat16 input, row stride ldx >= cols elements.
 *   codes        : out, [rows][cols/2] bytes.
 *   scales       : out, [rows][cols/B] bytes.
 *   tensor_scale : NVFP4: device float; written (COMPUTE) or read (GIVEN).
 *                  MXFP4: must be NULL.
 *   ts           : REQAT_TS_COMPUTE or REQAT_TS_GIVEN (ignored for MXFP4).
 *   workspace    : device scratch of reqat_workspace_bytes() bytes, needed for
 *                  NVFP4 with REQAT_TS_COMPUTE (may be NULL otherwise).
 * Requirements: cols % B == 0; x, codes, scales 16-byte aligned; ldx % 8 == 0.
 * rows == 0 or cols == 0 is a no-op (COMPUTE still writes g = 1).
 */
reqat_status reqat_quantize_fp4(reqat_format fmt, const void *x, int64_t rows, int64_t cols,
                                int64_t ldx, uint8_t *codes, uint8_t *scales, float *tensor_scale,
                                reqat_tscale_mode ts, void *workspace, void *stream);

/*
 * Fake-quant: y = bfloat16(dequantize(quantize(x))) (QAT forward, Sec. 2.2,
 * Sec. 4 Stage-2 QAT; every linear layer, App. D.1).  Same rules and
 * tensor-scale handling as reqat_quantize_fp4; y[rows][ldy] bfloat16.
 * Requirements: cols % B == 0; x, y 16-byte aligned; ldx % 8 == 0, ldy % 8 == 0.
 * In place (y == x, ldy == ldx) is allowed for MXFP4 and for NVFP4 with a
 * given tensor scale; any other overlap of y with x, and in place with
 * NVFP4 and REQAT_TS_COMPUTE (whose second pass re-reads x), returns
 * REQAT_E_UNSUPPORTED.
 */
reqat_status reqat_fakequant_fp4(reqat_format fmt, const void *x, int64_t rows, int64_t cols,
                                 int64_t ldx, void *y, int64_t ldy, float *tensor_scale,
                                 reqat_tscale_mode ts, void *workspace, void *stream);

/*
 * Quantize and fake-quant in one pass over x: codes and scales exactly as
 * reqat_quantize_fp4 writes them, y exactly as reqat_fakequant_fp4 writes it
 * (the QAT forward's quantize-dequantize, Sec. 2.2, together with the codes
 * its 4-bit product consumes, Sec. 5.3), one tensor scale g for both.  Reads
 * x once instead of twice.
 *   codes [rows][cols/2], scales [rows][cols/B]: out, as reqat_quantize_fp4;
 *   y [rows][ldy] bfloat16: out, as reqat_fakequant_fp4 (ldy >= cols);
 *   tensor_scale, ts, workspace: as reqat_quantize_fp4.
 * Requirements: cols % B == 0; x, codes, scales, y 16-byte aligned;
 * ldx % 8 == 0, ldy % 8 == 0; y must not overlap x (REQAT_E_UNSUPPORTED);
 * codes and scales must not overlap x or y.
 * rows == 0 or cols == 0 is a no-op (COMPUTE still writes g = 1).
 */
reqat_status reqat_quantize_fakequant_fp4(reqat_format fmt, const void *x, int64_t rows, int64_t cols,
                                          int64_t ldx, uint8_t *codes, uint8_t *scales, void *y, int64_t ldy,
                                          float *tensor_scale, reqat_tscale_mode ts, void *workspace,
                                          void *stream);

/*
 * MXFP4 quantization of block-rotated rows (the block rotation ReQAT applies
 * to MXFP4 activations before quantizing them, Sec. 4.3 "Additional
 * implementation details" and App. C.2): each 32-element block x of a row
 * becomes
 *     y = H_32 * D * x / sqrt(32),   D = diag(d), d_j = -1 where bit j of signs is set,
 * H_32 the Sylvester Hadamard matrix (H[i][j] = (-1)^popcount(i & j)), and the
 * exact real y is quantized as an MXFP4 block by the rules of
 * reqat_quantize_fp4: scale 2^e with e the smallest integer in [-127, 127]
 * with max|y_i| <= 6 * 2^e (byte 0 for y == 0; 127 when none fits, elements
 * then saturate), each code the E2M1 value nearest to |y_i| / 2^e with the
 * sign of y_i (a zero y_i gives code 0).  No tie can occur (y_i is an
 * irrational multiple of 2^e unless it is zero).  The map is orthonormal:
 * rotating the weights' rows with the same signs leaves the product X W^T
 * unchanged.  A block with a NaN or Inf input gets scale 0xFF and zero codes.
 *   x [rows][ldx] bfloat16 (cols % 32 == 0, 16-byte aligned, ldx % 8 == 0);
 *   signs: the random sign draw, bit j for position j of every block;
 *   codes [rows][cols/2], scales [rows][cols/32] as reqat_quantize_fp4 (MXFP4).
 * rows == 0 or cols == 0 is a no-op.  Errors as reqat_quantize_fp4.
 */
reqat_status reqat_quantize_mxfp4_rht(const void *x, int64_t rows, int64_t cols, int64_t ldx,
                                      uint32_t signs, uint8_t *codes, uint8_t *scales, void *stream);

/*
 * Fake-quant of block-rotated rows: y_out = dequantize(quantize(y)), i.e.
 * code * 2^e (exact in bfloat16), with y the rotated blocks of
 * reqat_quantize_mxfp4_rht (values stay in the rotated basis; NaN 0x7FC0 for a
 * block with a NaN or Inf input).  y_out [rows][ldy] bfloat16,
 * 16-byte aligned, ldy % 8 == 0, ldy >= cols.
 */
reqat_status reqat_fakequant_mxfp4_rht(const void *x, int64_t rows, int64_t cols, int64_t ldx,
                                       uint32_t signs, void *y_out, int64_t ldy, void *stream);

/*
 * W4A16 product (the MXFP4 W4A16 deployment setting, Sec. 2 "Microscaled FP4
 * formats", Sec. 5.1, App. D.1): MXFP4 weights, bfloat16 activations,
 *     Y[m][n] = sum_k x[m][k] * w^[n][k],   w^ = RN_bf16(E2M1(c) * 2^e),
 * i.e. each weight dequantized to bfloat16 (exact for E8M0 bytes 2..252; the
 * bfloat16 rounding, overflow to Inf included, otherwise; NaN for 0xFF),
 * products exact, FP32 accumulation.
 *   x [M][ldx] bfloat16 (16-byte aligned, ldx % 8 == 0, ldx >= K);
 *   w_codes [N][K/2] (16-byte aligned), w_scales [N][K/32] (4-byte aligned),
 *   as reqat_quantize_fp4 writes them for MXFP4;
 *   y [M][ldy] of y_dtype, ldy >= N.
 *   workspace: device scratch of reqat_w4a16_workspace_bytes(M, N, K) bytes
 *              (4-byte aligned; may be NULL when that is 0): FP32 partial sums
 *              when K is split over several workgroups (few weight rows).
 * Requirements: K % 128 == 0.  M == 0 or N == 0 is a no-op; K == 0 writes zeros.
 * Designed for decode (small M): one pass over the weights.  The result is
 * deterministic: the split is a function of (M, N, K) alone and the partial
 * sums are added in a fixed order.
 */
reqat_status reqat_gemm_w4a16(int64_t M, int64_t N, int64_t K, const void *x, int64_t ldx,
                              const uint8_t *w_codes, const uint8_t *w_scales, void *y, reqat_dtype y_dtype,
                              int64_t ldy, void *workspace, void *stream);

/* Bytes of workspace reqat_gemm_w4a16 needs for an M x N x K product (0: none; 0 on bad arguments). */
size_t reqat_w4a16_workspace_bytes(int64_t M, int64_t N, int64_t K);

/*
 * Packed W4A16 weight image (weights are fixed in W4A16 serving, so they are
 * re-laid out once, when loaded): the MXFP4 weights of reqat_gemm_w4a16 in
 * the order its matrix-core tiles consume them, so that the product reads
 * each wave's weights as contiguous 1 KB runs instead of 64 bytes from each
 * of 16 rows.  Rows go in groups of 16 (the last padded with zero codes and
 * scales), K in chunks of 128 elements; with G = ceil(N / 16), C = K / 128:
 *   bytes [0, 1024 G C): unit (g, c) at 1024 (g C + c) holds, at byte
 *     16 (r + 16 q) + i, byte 16 q + i of chunk c of row 16 g + r, i.e.
 *     w_codes[16 g + r][64 c + 16 q + i]  (r < 16, q < 4, i < 16);
 *   bytes [1024 G C, 1088 G C): unit (g, c) at 1024 G C + 64 (g C + c) holds,
 *     at byte 4 r + j, w_scales[16 g + r][4 c + j]  (j < 4).
 * reqat_w4a16_packed_bytes: the image's size, 1088 G C (0 on bad arguments:
 * N < 0, K < 0 or K % 128).
 * reqat_pack_w4a16: writes the image of w_codes [N][K/2] (16-byte aligned) and
 * w_scales [N][K/32] (4-byte aligned) into `packed` (16-byte aligned, not
 * overlapping them), on `stream`.  A pure re-layout: no value changes.
 * Errors: REQAT_E_SHAPE (N < 0, K < 0, K % 128), REQAT_E_NULL, REQAT_E_ALIGN,
 * REQAT_E_UNSUPPORTED (packed overlaps w_codes or w_scales).
 */
size_t reqat_w4a16_packed_bytes(int64_t N, int64_t K);
reqat_status reqat_pack_w4a16(const uint8_t *w_codes, const uint8_t *w_scales, int64_t N, int64_t K, void *packed,
                              void *stream);

/*
 * reqat_gemm_w4a16 on the packed image of its weights (same result, bit for
 * bit: the same splits and the same order of operations).  packed: the
 * reqat_w4a16_packed_bytes(N, K) bytes reqat_pack_w4a16 wrote (16-byte
 * aligned).  Other arguments, requirements, workspace and errors as
 * reqat_gemm_w4a16.
 */
reqat_status reqat_gemm_w4a16_packed(int64_t M, int64_t N, int64_t K, const void *x, int64_t ldx, const void *packed,
                                     void *y, reqat_dtype y_dtype, int64_t ldy, void *workspace, void *stream);

/*
 * KV-cache quantization of the NVFP4 W4A4KV4 setting: E1M2 elements (the KV4
 * element format, Sec. 4.3 "Additional implementation details") with the
 * Q-FIT post-RoPE shift applied first (Sec. 4.3, K~ = R(K_pre / s) - m):
 *     d[r][c] = RN_fp32(x[r][c] - shift[c])            (shift == NULL: d = x)
 * quantized along c in blocks of 16: an E4M3 block scale, the smallest with
 * block_amax <= 3.5 * s * g, an FP32 tensor scale g (REQAT_TS_COMPUTE: the
 * smallest power of two 2^k, k >= -126, with tensor_amax <= 3.5 * 448 * 2^k,
 * g = 1 for a tensor without non-zero finite values; REQAT_TS_GIVEN: as
 * given), E1M2 codes (magnitudes 0, 0.5, ..., 3.5; bit 3 sign, bit 2 exponent,
 * bits 1:0 mantissa) rounded to nearest with ties to the even code.  A block
 * with a non-finite d gets scale 0x7F and zero codes.  Layouts as
 * reqat_quantize_fp4 with B = 16.
 *   shift: NULL or cols FP32 values, 16-byte aligned (keys: the calibrated
 *          channel means m; values: NULL).
 *   workspace: reqat_workspace_bytes() bytes, needed for REQAT_TS_COMPUTE.
 * Requirements and errors as reqat_quantize_fp4 (NVFP4).
 */
reqat_status reqat_quantize_kv4(const void *x, int64_t rows, int64_t cols, int64_t ldx, const float *shift,
                                uint8_t *codes, uint8_t *scales, float *tensor_scale, reqat_tscale_mode ts,
                                void *workspace, void *stream);

/*
 * Fake-quant of the KV4 quantization above: y[r][c] = RN_bf16(E1M2(code) * s * g)
 * in the shifted domain (NaN for a non-finite block).  y [rows][ldy] bfloat16,
 * 16-byte aligned, ldy % 8 == 0, ldy >= cols.  In place under the rules of
 * reqat_fakequant_fp4 for NVFP4: not with REQAT_TS_COMPUTE, whose fix-up
 * re-reads x.
 */
reqat_status reqat_fakequant_kv4(const void *x, int64_t rows, int64_t cols, int64_t ldx, const float *shift,
                                 void *y, int64_t ldy, float *tensor_scale, reqat_tscale_mode ts, void *workspace,
                                 void *stream);

/*
 * SEM loss, the training objective of ReQAT's TAQ stage (Sec. 4.2):
 *     L = (1/T) sum_t NLL_t + lambda (1/T) sum_t w_t H_t,
 *     w_t = max(0, 1 - (H_t - H_min) / (tau - H_min + eps)),
 * with, per token t (a row of bfloat16 logits over the vocabulary, p its
 * softmax), the predictive entropy H_t = -sum_j p_j log p_j and
 * NLL_t = -log p_{y_t}; H_min the minimum of H over the T tokens and tau its
 * 75th percentile (linear interpolation between order statistics at
 * position 0.75 (T - 1)).  Computed in FP32 (sums of the weighted terms in
 * FP64).  The logits are read once.
 *   logits [T][ld] bfloat16 (finite; 16-byte aligned, ld % 8 == 0, V % 8 == 0);
 *   targets [T] int32 in [0, V) (outside: NLL_t = NaN, no read);
 *   stats [T][4] FP32 out: H_t, NLL_t, log-sum-exp_t, 0 (kept for the backward);
 *   weights [T] FP32 out: w_t;  loss [4] FP32 out: L, mean NLL, mean w H, tau.
 * T == 0 is a no-op.
 */
reqat_status reqat_sem_loss(const void *logits, int64_t T, int64_t V, int64_t ld, const int32_t *targets,
                            float lambda, float eps, float *stats, float *weights, float *loss, void *stream);

/*
 * Gradient of the SEM loss with the weights w_t held fixed (they select
 * tokens, they are not optimized):
 *     dL/dz_tj = (scale / T) [(p_tj - [j == y_t]) - lambda w_t p_tj (log p_tj + H_t)],
 * using stats and weights from reqat_sem_loss on the same logits.  With the
 * quantizers' straight-through estimator (ReQAT's QAT forward quantizes with
 * fake-quant; every scale rule here is "ceil", so nothing clips and the
 * estimator passes the gradient through unchanged) this is the whole backward
 * of the loss head.  grad [T][ldg] of grad_dtype (16-byte aligned; ldg >= V,
 * a multiple of 8 for bfloat16, 4 for FP32).
 */
reqat_status reqat_sem_loss_backward(const void *logits, int64_t T, int64_t V, int64_t ld, const int32_t *targets,
                                     const float *stats, const float *weights, float lambda, float scale,
                                     void *grad, reqat_dtype grad_dtype, int64_t ldg, void *stream);

/*
 * Block-scaled FP4 x FP4 product (the W4A4 GEMM of Sec. 5.3):
 *   Y[m][n] = g_a * g_b * sum_k A^[m][k] * B^[n][k]
 * with A^ = E2M1(a_codes) * block scale (and likewise B^), FP32 accumulation.
 *   a_codes [M][K/2], a_scales [M][K/B], a_tensor_scale (NVFP4: device float; MXFP4: NULL)
 *   b_codes [N][K/2], b_scales [N][K/B], b_tensor_scale (same rule)
 *   y [M][ldy] of y_dtype.
 * Requirements: K % 128 == 0 (so every row pitch, K/2 and K/B bytes, is a
 * multiple of 4); code and scale pointers 16-byte aligned; y aligned to its
 * element size; ldy >= N.  M == 0 or N == 0 is a no-op; K == 0 writes zeros.
 */
reqat_status reqat_gemm_w4a4(reqat_format fmt, int64_t M, int64_t N, int64_t K,
                             const uint8_t *a_codes, const uint8_t *a_scales,
                             const float *a_tensor_scale,
                             const uint8_t *b_codes, const uint8_t *b_scales,
                             const float *b_tensor_scale,
                             void *y, reqat_dtype y_dtype, int64_t ldy, void *stream);

/*
 * W4A4 linear layer: quantize the activations x[M][K] (bfloat16) and multiply
 * them by already-quantized weights (the "4-bit GEMM enabled by activation
 * quantization" of Sec. 5.3):
 *   Y = gemm_w4a4(quantize(x), W)
 * The activation quantization follows reqat_quantize_fp4 exactly (same codes,
 * scales and computed g); it runs as a kernel on `stream` immediately before
 * the product, with the activation codes and scales kept in `workspace`.
 *   x, ldx         : bfloat16 activations, ldx >= K, ldx % 8 == 0, 16-byte aligned.
 *   x_tensor_scale : NVFP4: device float, written (COMPUTE) or read (GIVEN);
 *                    MXFP4: must be NULL.
 *   ts             : REQAT_TS_COMPUTE or REQAT_TS_GIVEN (ignored for MXFP4).
 *   w_codes, w_scales, w_tensor_scale : the weights, as b_* of reqat_gemm_w4a4.
 *   y, y_dtype, ldy: as reqat_gemm_w4a4.
 *   workspace      : device scratch of reqat_linear_workspace_bytes(fmt, M, K)
 *                    bytes, 256-byte aligned; it holds the activation codes
 *                    and scales until the product has run.
 * Requirements: K % 128 == 0, plus those of the two operations.  M == 0 is a
 * no-op except that COMPUTE writes g = 1; N == 0 (M > 0) enqueues nothing.
 */
reqat_status reqat_linear_w4a4(reqat_format fmt, int64_t M, int64_t N, int64_t K,
                               const void *x, int64_t ldx, float *x_tensor_scale,
                               reqat_tscale_mode ts, const uint8_t *w_codes,
                               const uint8_t *w_scales, const float *w_tensor_scale,
                               void *y, reqat_dtype y_dtype, int64_t ldy, void *workspace,
                               void *stream);

/*
 * Packed decode weight image (weights are fixed in serving, so they can be
 * re-laid out once, when loaded): the weights of reqat_gemm_w4a4 in the order
 * the decode-shaped product (M <= 64) consumes them, so that each of its
 * weight loads reads 1 KB of consecutive bytes instead of 64 bytes from each
 * of 16 rows.  Rows go in groups of 16 (the last padded with zero codes and
 * scales), K in chunks of 256 elements (when K % 256 == 128 the last chunk's
 * second half is zero); with G = ceil(N / 16), C = ceil(K / 256) and
 * S = 16 (NVFP4) or 8 (MXFP4) scale bytes per row and chunk:
 *   bytes [0, 2048 G C): unit (g, c) at 2048 (g C + c) holds, at byte
 *     1024 h + 16 (r + 16 q) + i, w_codes[16 g + r][128 c + 32 q + 16 h + i]
 *     (h < 2, r < 16, q < 4, i < 16);
 *   bytes [2048 G C, (2048 + 16 S) G C): unit (g, c) at 2048 G C + 16 S (g C + c)
 *     holds, at byte (S / 4)(r + 16 q) + j, w_scales[16 g + r][S c + (S / 4) q + j]
 *     (j < S / 4).
 * reqat_w4a4_packed_bytes: the image's size, (2048 + 16 S) G C (0 on bad
 * arguments: unknown format, N < 0, K < 0 or K % 128).
 * reqat_pack_w4a4: writes the image of w_codes [N][K/2] and w_scales [N][K/B]
 * (both 16-byte aligned, as for reqat_gemm_w4a4) into `packed` (16-byte
 * aligned, not overlapping them), on `stream`.  A pure re-layout: no value
 * changes; the weights' tensor scale stays with the caller.
 * Errors: REQAT_E_ENUM, REQAT_E_SHAPE (N < 0, K < 0, K % 128), REQAT_E_NULL,
 * REQAT_E_ALIGN, REQAT_E_UNSUPPORTED (packed overlaps w_codes or w_scales).
 */
size_t reqat_w4a4_packed_bytes(reqat_format fmt, int64_t N, int64_t K);
reqat_status reqat_pack_w4a4(reqat_format fmt, const uint8_t *w_codes, const uint8_t *w_scales, int64_t N, int64_t K,
                             void *packed, void *stream);

/*
 * reqat_gemm_w4a4 and reqat_linear_w4a4 (the 4-bit GEMM of Sec. 5.3) for
 * decode-shaped products (1 <= M <= 64) on the packed image of the weights (same results, bit for
 * bit: the same kernel and order of operations, only the weight addresses
 * differ).  packed: the reqat_w4a4_packed_bytes(fmt, N, K) bytes
 * reqat_pack_w4a4 wrote for the same format (16-byte aligned); it takes the
 * place of b_codes / b_scales (w_codes / w_scales).  Other arguments,
 * requirements, workspace and errors as the row-major calls, plus
 * REQAT_E_UNSUPPORTED for M > 64.
 */
reqat_status reqat_gemm_w4a4_packed(reqat_format fmt, int64_t M, int64_t N, int64_t K,
                                    const uint8_t *a_codes, const uint8_t *a_scales,
                                    const float *a_tensor_scale, const void *packed,
                                    const float *b_tensor_scale, void *y, reqat_dtype y_dtype, int64_t ldy,
                                    void *stream);
reqat_status reqat_linear_w4a4_packed(reqat_format fmt, int64_t M, int64_t N, int64_t K,
                                      const void *x, int64_t ldx, float *x_tensor_scale,
                                      reqat_tscale_mode ts, const void *packed,
                                      const float *w_tensor_scale, void *y, reqat_dtype y_dtype, int64_t ldy,
                                      void *workspace, void *stream);

/* Bytes of workspace reqat_linear_w4a4 needs for M x K activations (0 on bad arguments). */
size_t reqat_linear_workspace_bytes(reqat_format fmt, int64_t M, int64_t K);

/*
 * reqat_linear_w4a4 for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same operation, kernels and results, with the workspace replaced by a
 * fixed scratch array the library holds on each device (REQAT_NOALLOC_SCRATCH_BYTES
 * bytes, from the first call on a device until the process ends).  It calls
 * no allocating routine.  Arguments as reqat_linear_w4a4 without `workspace`;
 * returns REQAT_E_TOO_LARGE, enqueueing nothing, when
 * reqat_linear_workspace_bytes(fmt, M, K) exceeds the scratch (NVFP4: about
 * 14.8 million activation elements, MXFP4: 15.3 million).  Every call on a
 * device uses the same scratch, so calls that overlap in time on one device
 * (different streams, or host threads) race; calls in order on one stream do not.
 */
#define REQAT_NOALLOC_SCRATCH_BYTES (8u << 20)
reqat_status reqat_linear_w4a4_noalloc(reqat_format fmt, int64_t M, int64_t N, int64_t K,
                                       const void *x, int64_t ldx, float *x_tensor_scale,
                                       reqat_tscale_mode ts, const uint8_t *w_codes,
                                       const uint8_t *w_scales, const float *w_tensor_scale,
                                       void *y, reqat_dtype y_dtype, int64_t ldy, void *stream);

/* Bytes of device workspace that a quantize / fake-quant call may use. */
size_t reqat_workspace_bytes(void);

/* Static, human-readable name of a status code. */
const char *reqat_status_str(reqat_status s);

/* REQAT_ABI_VERSION of the built library. */
int reqat_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* REQAT_H */
