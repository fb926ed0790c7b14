// C ABI of libreqat: host-side argument validation and dispatch to the kernels.
// Validation happens before any HIP call, so a bad argument is reported without
// touching the device (and can be tested on a host without a GPU).
#include <mutex>

#include "../../include/reqat.h"
#include "internal.h"

namespace {

using namespace reqat;

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int block_of(reqat_format f) { return f == REQAT_FMT_MXFP4 ? 32 : 16; }

bool fmt_ok(reqat_format f) { return f == REQAT_FMT_NVFP4 || f == REQAT_FMT_MXFP4; }

// Shared validation of quantize / fake-quant arguments.
reqat_status check_quant(reqat_format fmt, const void *x, int64_t rows, int64_t cols, int64_t ldx,
                         const void *out0, const void *out1, int64_t ldy, const float *ts_ptr,
                         reqat_tscale_mode ts, const void *workspace, bool fake) {
    if (!fmt_ok(fmt)) return REQAT_E_ENUM;
    if (fmt == REQAT_FMT_NVFP4 && ts != REQAT_TS_COMPUTE && ts != REQAT_TS_GIVEN) return REQAT_E_ENUM;
    if (rows < 0 || cols < 0) return REQAT_E_SHAPE;
    if (cols % block_of(fmt)) return REQAT_E_SHAPE;
    if (ldx < cols || (fake && ldy < cols)) return REQAT_E_SHAPE;
    if (fmt == REQAT_FMT_MXFP4 && ts_ptr != nullptr) return REQAT_E_UNSUPPORTED;
    if (fmt == REQAT_FMT_NVFP4 && ts_ptr == nullptr) return REQAT_E_NULL;
    if (fmt == REQAT_FMT_NVFP4 && ts == REQAT_TS_COMPUTE && workspace == nullptr) return REQAT_E_NULL;
    if (rows == 0 || cols == 0) return REQAT_OK;
    if (!x || !out0 || (!fake && !out1)) return REQAT_E_NULL;
    if (!aligned16(x) || !aligned16(out0) || (!fake && !aligned16(out1))) return REQAT_E_ALIGN;
    if (ldx % 8 || (fake && ldy % 8)) return REQAT_E_ALIGN;
    if (fmt == REQAT_FMT_NVFP4 && (reinterpret_cast<uintptr_t>(ts_ptr) & 3u)) return REQAT_E_ALIGN;
    if (workspace && (reinterpret_cast<uintptr_t>(workspace) & 3u)) return REQAT_E_ALIGN;
    return REQAT_OK;
}

// Whether the bytes [a, a + na) and [b, b + nb) overlap.
bool overlaps(const void *a, size_t na, const void *b, size_t nb) {
    const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
    return na && nb && pa < pb + nb && pb < pa + na;
}

// Bytes spanned by a rows x cols bfloat16 matrix with leading dimension ld.
size_t span_bf16(int64_t rows, int64_t cols, int64_t ld) {
    return rows > 0 && cols > 0 ? (size_t)(((rows - 1) * ld + cols) * 2) : 0;
}

// `workspace` holds the kMaxPartials partial maxima; `seg_table` (NVFP4 with
// a computed g) has room for seg_capacity segments, else the quantizer reads x twice.
reqat_status run_quant(reqat_format fmt, const void *x, int64_t rows, int64_t cols, int64_t ldx,
                       uint8_t *codes, uint8_t *scales, void *y, int64_t ldy, float *tensor_scale,
                       reqat_tscale_mode ts, void *workspace, uint16_t *seg_table, int64_t seg_capacity,
                       void *stream, QuantOut out) {
    const bool fake = out == kFakeQuant;
    reqat_status st = check_quant(fmt, x, rows, cols, ldx, fake ? y : codes, scales, ldy,
                                  tensor_scale, ts, workspace, fake);
    if (st != REQAT_OK) return st;
    if (out == kBoth && rows > 0 && cols > 0) {
        if (!y) return REQAT_E_NULL;
        if (ldy < cols) return REQAT_E_SHAPE;
        if (!aligned16(y) || ldy % 8) return REQAT_E_ALIGN;
    }
    if (out != kCodes && overlaps(x, span_bf16(rows, cols, ldx), y, span_bf16(rows, cols, ldy))) {
        // in place is allowed for fake-quant alone when x is not read again
        // after y is written: not with a computed NVFP4 scale (the fix-up
        // pass re-quantizes some blocks from x), and never with codes too
        const bool reread = fmt == REQAT_FMT_NVFP4 && ts == REQAT_TS_COMPUTE;
        if (out == kBoth || reread || x != y || ldx != ldy) return REQAT_E_UNSUPPORTED;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const bool nv = fmt == REQAT_FMT_NVFP4;
    const bool compute = nv && ts == REQAT_TS_COMPUTE;
    if (rows == 0 || cols == 0) {
        if (compute && launch_unit_scale(tensor_scale, s) != hipSuccess) return REQAT_E_HIP;
        return REQAT_OK;
    }
    GSrc gsrc = !nv ? kGNone : (compute ? kGComputed : kGGiven);
    hipError_t e = launch_quantize(nv ? kNV : kMX, out,
                                   reinterpret_cast<const uint16_t *>(x), rows, cols, ldx, codes,
                                   scales, reinterpret_cast<uint16_t *>(y), ldy, tensor_scale, gsrc,
                                   reinterpret_cast<uint32_t *>(workspace), compute ? seg_table : nullptr,
                                   seg_capacity, s);
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

// Quantize workspace: [kMaxPartials uint32 partial maxima | kMaxSegments uint16 segment table].
uint16_t *quant_seg_table(void *workspace) {
    return workspace ? reinterpret_cast<uint16_t *>(reinterpret_cast<uint8_t *>(workspace) +
                                                    sizeof(uint32_t) * kMaxPartials)
                     : nullptr;
}

size_t round256(size_t n) { return (n + 255) & ~(size_t)255; }

// Segments of 64 blocks in an M x K activation (NVFP4), and whether the linear
// workspace carries a segment table for them.
int64_t linear_segments(int64_t M, int64_t K) { return (M * (K / 16) + 63) / 64; }

}  // namespace

extern "C" {

reqat_status reqat_quantize_fp4(reqat_format fmt, const void *x, int64_t rows, int64_t cols,
                                int64_t ldx, uint8_t *codes, uint8_t *scales, float *tensor_scale,
                                reqat_tscale_mode ts, void *workspace, void *stream) {
    return run_quant(fmt, x, rows, cols, ldx, codes, scales, nullptr, 0, tensor_scale, ts,
                     workspace, quant_seg_table(workspace), kMaxSegments, stream, kCodes);
}

reqat_status reqat_fakequant_fp4(reqat_format fmt, const void *x, int64_t rows, int64_t cols,
                                 int64_t ldx, void *y, int64_t ldy, float *tensor_scale,
                                 reqat_tscale_mode ts, void *workspace, void *stream) {
    return run_quant(fmt, x, rows, cols, ldx, nullptr, nullptr, y, ldy, tensor_scale, ts,
                     workspace, quant_seg_table(workspace), kMaxSegments, stream, kFakeQuant);
}

reqat_status reqat_quantize_fakequant_fp4(reqat_format fmt, const void *x, int64_t rows, int64_t cols,
                                          int64_t ldx, uint8_t *codes, uint8_t *scales, void *y, int64_t ldy,
                                          float *tensor_scale, reqat_tscale_mode ts, void *workspace,
                                          void *stream) {
    return run_quant(fmt, x, rows, cols, ldx, codes, scales, y, ldy, tensor_scale, ts, workspace,
                     quant_seg_table(workspace), kMaxSegments, stream, kBoth);
}

static reqat_status run_kv4(const void *x, int64_t rows, int64_t cols, int64_t ldx, const float *shift,
                            uint8_t *codes, uint8_t *scales, void *y, int64_t ldy, float *tensor_scale,
                            reqat_tscale_mode ts, void *workspace, void *stream, bool fake) {
    // same rules as the NVFP4 quantizer (blocks of 16, a tensor scale), plus the shift
    reqat_status st = check_quant(REQAT_FMT_NVFP4, x, rows, cols, ldx, fake ? y : codes, scales, ldy,
                                  tensor_scale, ts, workspace, fake);
    if (st != REQAT_OK) return st;
    if (shift && (reinterpret_cast<uintptr_t>(shift) & 15u)) return REQAT_E_ALIGN;
    if (fake && overlaps(x, span_bf16(rows, cols, ldx), y, span_bf16(rows, cols, ldy))) {
        // in place only when x is not read again after y is written: every
        // block is read before its values are stored, but a computed g's
        // fix-up re-quantizes some blocks from x
        if (ts == REQAT_TS_COMPUTE || x != y || ldx != ldy) return REQAT_E_UNSUPPORTED;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const bool compute = ts == REQAT_TS_COMPUTE;
    if (rows == 0 || cols == 0) {
        if (compute && launch_unit_scale(tensor_scale, s) != hipSuccess) return REQAT_E_HIP;
        return REQAT_OK;
    }
    hipError_t e = launch_kv4(fake ? kFakeQuant : kCodes, reinterpret_cast<const uint16_t *>(x), rows, cols, ldx,
                              shift, codes, scales, reinterpret_cast<uint16_t *>(y), ldy, tensor_scale, compute,
                              reinterpret_cast<uint32_t *>(workspace), compute ? quant_seg_table(workspace) : nullptr,
                              s);
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

reqat_status reqat_quantize_kv4(const void *x, int64_t rows, int64_t cols, int64_t ldx, const float *shift,
                                uint8_t *codes, uint8_t *scales, float *tensor_scale, reqat_tscale_mode ts,
                                void *workspace, void *stream) {
    return run_kv4(x, rows, cols, ldx, shift, codes, scales, nullptr, 0, tensor_scale, ts, workspace, stream,
                   false);
}

reqat_status reqat_fakequant_kv4(const void *x, int64_t rows, int64_t cols, int64_t ldx, const float *shift,
                                 void *y, int64_t ldy, float *tensor_scale, reqat_tscale_mode ts, void *workspace,
                                 void *stream) {
    return run_kv4(x, rows, cols, ldx, shift, nullptr, nullptr, y, ldy, tensor_scale, ts, workspace, stream, true);
}

static reqat_status run_rht(const void *x, int64_t rows, int64_t cols, int64_t ldx, uint32_t signs,
                            uint8_t *codes, uint8_t *scales, void *y, int64_t ldy, void *stream, bool fake) {
    reqat_status st = check_quant(REQAT_FMT_MXFP4, x, rows, cols, ldx, fake ? y : codes, scales, ldy,
                                  nullptr, REQAT_TS_GIVEN, nullptr, fake);
    if (st != REQAT_OK || rows == 0 || cols == 0) return st;
    hipError_t e = launch_quantize_rht(fake ? kFakeQuant : kCodes, reinterpret_cast<const uint16_t *>(x), rows,
                                       cols, ldx, signs, codes, scales, reinterpret_cast<uint16_t *>(y), ldy,
                                       reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

reqat_status reqat_quantize_mxfp4_rht(const void *x, int64_t rows, int64_t cols, int64_t ldx, uint32_t signs,
                                      uint8_t *codes, uint8_t *scales, void *stream) {
    return run_rht(x, rows, cols, ldx, signs, codes, scales, nullptr, 0, stream, false);
}

reqat_status reqat_fakequant_mxfp4_rht(const void *x, int64_t rows, int64_t cols, int64_t ldx, uint32_t signs,
                                       void *y, int64_t ldy, void *stream) {
    return run_rht(x, rows, cols, ldx, signs, nullptr, nullptr, y, ldy, stream, true);
}

reqat_status reqat_gemm_w4a4(reqat_format fmt, int64_t M, int64_t N, int64_t K,
                             const uint8_t *a_codes, const uint8_t *a_scales,
                             const float *a_tensor_scale, const uint8_t *b_codes,
                             const uint8_t *b_scales, const float *b_tensor_scale, void *y,
                             reqat_dtype y_dtype, int64_t ldy, void *stream) {
    if (!fmt_ok(fmt)) return REQAT_E_ENUM;
    if (y_dtype != REQAT_DT_F32 && y_dtype != REQAT_DT_BF16) return REQAT_E_ENUM;
    if (M < 0 || N < 0 || K < 0) return REQAT_E_SHAPE;
    if (K % 128) return REQAT_E_SHAPE;
    if (ldy < N) return REQAT_E_SHAPE;
    const bool nv = fmt == REQAT_FMT_NVFP4;
    if (!nv && (a_tensor_scale || b_tensor_scale)) return REQAT_E_UNSUPPORTED;
    if (nv && (!a_tensor_scale || !b_tensor_scale)) return REQAT_E_NULL;
    if (M == 0 || N == 0) return REQAT_OK;
    if (!y) return REQAT_E_NULL;
    if (K > 0 && (!a_codes || !a_scales || !b_codes || !b_scales)) return REQAT_E_NULL;
    if (reinterpret_cast<uintptr_t>(y) & (y_dtype == REQAT_DT_BF16 ? 1u : 3u)) return REQAT_E_ALIGN;
    if (K > 0 && (!aligned16(a_codes) || !aligned16(b_codes) || !aligned16(a_scales) ||
                  !aligned16(b_scales)))
        return REQAT_E_ALIGN;
    if (nv && ((reinterpret_cast<uintptr_t>(a_tensor_scale) & 3u) ||
               (reinterpret_cast<uintptr_t>(b_tensor_scale) & 3u)))
        return REQAT_E_ALIGN;
    hipError_t e = launch_gemm(nv ? kNV : kMX, M, N, K, a_codes, a_scales, a_tensor_scale, b_codes,
                               b_scales, b_tensor_scale, y, y_dtype == REQAT_DT_BF16, ldy,
                               reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

size_t reqat_w4a16_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    if (M < 0 || N < 0 || K < 0 || K % 128) return 0;
    return gemm_w4a16_workspace_bytes(M, N, K);
}

reqat_status reqat_gemm_w4a16(int64_t M, int64_t N, int64_t K, const void *x, int64_t ldx,
                              const uint8_t *w_codes, const uint8_t *w_scales, void *y, reqat_dtype y_dtype,
                              int64_t ldy, void *workspace, void *stream) {
    if (y_dtype != REQAT_DT_F32 && y_dtype != REQAT_DT_BF16) return REQAT_E_ENUM;
    if (M < 0 || N < 0 || K < 0) return REQAT_E_SHAPE;
    if (K % 128 || ldx < K || ldy < N) return REQAT_E_SHAPE;
    if (M == 0 || N == 0) return REQAT_OK;
    if (!y || (K > 0 && (!x || !w_codes || !w_scales))) return REQAT_E_NULL;
    if (gemm_w4a16_workspace_bytes(M, N, K) > 0 && !workspace) return REQAT_E_NULL;
    if (K > 0 && (!aligned16(x) || ldx % 8 || !aligned16(w_codes) || (reinterpret_cast<uintptr_t>(w_scales) & 3u)))
        return REQAT_E_ALIGN;
    if (reinterpret_cast<uintptr_t>(y) & (y_dtype == REQAT_DT_BF16 ? 1u : 3u)) return REQAT_E_ALIGN;
    if (reinterpret_cast<uintptr_t>(workspace) & 3u) return REQAT_E_ALIGN;
    hipError_t e = launch_gemm_w4a16(M, N, K, reinterpret_cast<const uint16_t *>(x), ldx, w_codes, w_scales, false,
                                     y, y_dtype == REQAT_DT_BF16, ldy, reinterpret_cast<float *>(workspace),
                                     reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

size_t reqat_w4a16_packed_bytes(int64_t N, int64_t K) {
    if (N < 0 || K < 0 || K % 128) return 0;
    return w4a16_packed_bytes(N, K);
}

reqat_status reqat_pack_w4a16(const uint8_t *w_codes, const uint8_t *w_scales, int64_t N, int64_t K, void *packed,
                              void *stream) {
    if (N < 0 || K < 0 || K % 128) return REQAT_E_SHAPE;
    if (N == 0 || K == 0) return REQAT_OK;
    if (!w_codes || !w_scales || !packed) return REQAT_E_NULL;
    if (!aligned16(w_codes) || (reinterpret_cast<uintptr_t>(w_scales) & 3u) || !aligned16(packed))
        return REQAT_E_ALIGN;
    const size_t pbytes = w4a16_packed_bytes(N, K);
    if (overlaps(packed, pbytes, w_codes, (size_t)N * (size_t)(K / 2)) ||
        overlaps(packed, pbytes, w_scales, (size_t)N * (size_t)(K / 32)))
        return REQAT_E_UNSUPPORTED;
    hipError_t e = launch_w4a16_pack(w_codes, w_scales, N, K, reinterpret_cast<uint8_t *>(packed),
                                     reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

reqat_status reqat_gemm_w4a16_packed(int64_t M, int64_t N, int64_t K, const void *x, int64_t ldx, const void *packed,
                                     void *y, reqat_dtype y_dtype, int64_t ldy, void *workspace, void *stream) {
    if (y_dtype != REQAT_DT_F32 && y_dtype != REQAT_DT_BF16) return REQAT_E_ENUM;
    if (M < 0 || N < 0 || K < 0) return REQAT_E_SHAPE;
    if (K % 128 || ldx < K || ldy < N) return REQAT_E_SHAPE;
    if (M == 0 || N == 0) return REQAT_OK;
    if (!y || (K > 0 && (!x || !packed))) return REQAT_E_NULL;
    if (gemm_w4a16_workspace_bytes(M, N, K) > 0 && !workspace) return REQAT_E_NULL;
    if (K > 0 && (!aligned16(x) || ldx % 8 || !aligned16(packed))) return REQAT_E_ALIGN;
    if (reinterpret_cast<uintptr_t>(y) & (y_dtype == REQAT_DT_BF16 ? 1u : 3u)) return REQAT_E_ALIGN;
    if (reinterpret_cast<uintptr_t>(workspace) & 3u) return REQAT_E_ALIGN;
    const uint8_t *pc = reinterpret_cast<const uint8_t *>(packed);
    const uint8_t *ps = pc + (size_t)((N + 15) / 16) * (size_t)(K / 128) * 1024u;
    hipError_t e = launch_gemm_w4a16(M, N, K, reinterpret_cast<const uint16_t *>(x), ldx, pc, ps, true, y,
                                     y_dtype == REQAT_DT_BF16, ldy, reinterpret_cast<float *>(workspace),
                                     reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

reqat_status reqat_sem_loss(const void *logits, int64_t T, int64_t V, int64_t ld, const int32_t *targets,
                            float lambda, float eps, float *stats, float *weights, float *loss, void *stream) {
    if (T < 0 || V <= 0 || V % 8 || ld < V) return REQAT_E_SHAPE;
    if (T > 0x7FFFFFFF) return REQAT_E_SHAPE;
    if (!loss) return REQAT_E_NULL;
    if (T > 0 && (!logits || !targets || !stats || !weights)) return REQAT_E_NULL;
    if (T > 0 && (!aligned16(logits) || ld % 8)) return REQAT_E_ALIGN;
    if ((reinterpret_cast<uintptr_t>(stats) | reinterpret_cast<uintptr_t>(weights) |
         reinterpret_cast<uintptr_t>(loss) | reinterpret_cast<uintptr_t>(targets)) & 3u)
        return REQAT_E_ALIGN;
    if (T == 0) return REQAT_OK;
    hipError_t e = launch_sem_forward(reinterpret_cast<const uint16_t *>(logits), T, V, ld, targets, lambda, eps,
                                      stats, weights, loss, reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

reqat_status reqat_sem_loss_backward(const void *logits, int64_t T, int64_t V, int64_t ld, const int32_t *targets,
                                     const float *stats, const float *weights, float lambda, float scale,
                                     void *grad, reqat_dtype grad_dtype, int64_t ldg, void *stream) {
    if (grad_dtype != REQAT_DT_F32 && grad_dtype != REQAT_DT_BF16) return REQAT_E_ENUM;
    if (T < 0 || V <= 0 || V % 8 || ld < V || ldg < V) return REQAT_E_SHAPE;
    if (T > 0x7FFFFFFF) return REQAT_E_SHAPE;
    if (T == 0) return REQAT_OK;
    if (!logits || !targets || !stats || !weights || !grad) return REQAT_E_NULL;
    if (!aligned16(logits) || ld % 8 || !aligned16(grad) || ldg % (grad_dtype == REQAT_DT_BF16 ? 8 : 4))
        return REQAT_E_ALIGN;
    if ((reinterpret_cast<uintptr_t>(stats) | reinterpret_cast<uintptr_t>(weights) |
         reinterpret_cast<uintptr_t>(targets)) & 3u)
        return REQAT_E_ALIGN;
    hipError_t e = launch_sem_backward(reinterpret_cast<const uint16_t *>(logits), T, V, ld, targets, stats, weights,
                                       lambda, scale, grad, grad_dtype == REQAT_DT_BF16, ldg,
                                       reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

size_t reqat_workspace_bytes(void) {
    return sizeof(uint32_t) * kMaxPartials + sizeof(uint16_t) * kMaxSegments;
}

// Linear workspace: [partial maxima | activation codes | activation scales |
// NVFP4 segment table (when the activation fits kMaxSegments)], each part
// starting on a 256-byte boundary.
size_t reqat_linear_workspace_bytes(reqat_format fmt, int64_t M, int64_t K) {
    if (!fmt_ok(fmt) || M < 0 || K < 0 || K % 128) return 0;
    const size_t codes = (size_t)M * (size_t)(K / 2);
    const size_t scales = (size_t)M * (size_t)(K / block_of(fmt));
    const int64_t nseg = fmt == REQAT_FMT_NVFP4 ? linear_segments(M, K) : 0;
    const size_t table = nseg <= kMaxSegments ? sizeof(uint16_t) * (size_t)nseg : 0;
    return round256(sizeof(uint32_t) * kMaxPartials) + round256(codes) + round256(scales) + round256(table);
}

}  // extern "C"

namespace {

// Validation of the linear layer's arguments, workspace excluded.
reqat_status check_linear(reqat_format fmt, int64_t M, int64_t N, int64_t K, const void *x, int64_t ldx,
                          const float *x_tensor_scale, reqat_tscale_mode ts, const uint8_t *w_codes,
                          const uint8_t *w_scales, const float *w_tensor_scale, const void *y,
                          reqat_dtype y_dtype, int64_t ldy) {
    if (!fmt_ok(fmt)) return REQAT_E_ENUM;
    if (y_dtype != REQAT_DT_F32 && y_dtype != REQAT_DT_BF16) return REQAT_E_ENUM;
    const bool nv = fmt == REQAT_FMT_NVFP4;
    if (nv && ts != REQAT_TS_COMPUTE && ts != REQAT_TS_GIVEN) return REQAT_E_ENUM;
    if (M < 0 || N < 0 || K < 0) return REQAT_E_SHAPE;
    if (K % 128 || ldx < K || ldy < N) return REQAT_E_SHAPE;
    if (!nv && (x_tensor_scale || w_tensor_scale)) return REQAT_E_UNSUPPORTED;
    if (nv && (!x_tensor_scale || !w_tensor_scale)) return REQAT_E_NULL;
    if (M > 0 && N > 0) {
        if (!x || !y) return REQAT_E_NULL;
        if (K > 0 && (!w_codes || !w_scales)) return REQAT_E_NULL;
        if (!aligned16(x) || ldx % 8) return REQAT_E_ALIGN;
        if (reinterpret_cast<uintptr_t>(y) & (y_dtype == REQAT_DT_BF16 ? 1u : 3u)) return REQAT_E_ALIGN;
        if (K > 0 && (!aligned16(w_codes) || !aligned16(w_scales))) return REQAT_E_ALIGN;
        if (nv && ((reinterpret_cast<uintptr_t>(x_tensor_scale) & 3u) ||
                   (reinterpret_cast<uintptr_t>(w_tensor_scale) & 3u)))
            return REQAT_E_ALIGN;
    }
    return REQAT_OK;
}

// Quantize x into `workspace` (laid out as reqat_linear_workspace_bytes describes)
// and run the product; arguments already validated.
reqat_status run_linear(reqat_format fmt, int64_t M, int64_t N, int64_t K, const void *x, int64_t ldx,
                        float *x_tensor_scale, reqat_tscale_mode ts, const uint8_t *w_codes,
                        const uint8_t *w_scales, const float *w_tensor_scale, void *y, reqat_dtype y_dtype,
                        int64_t ldy, void *workspace, void *stream, bool packed = false) {
    const bool nv = fmt == REQAT_FMT_NVFP4;
    uint8_t *ws = reinterpret_cast<uint8_t *>(workspace);
    uint8_t *a_codes = ws + round256(sizeof(uint32_t) * kMaxPartials);
    uint8_t *a_scales = a_codes + round256((size_t)M * (size_t)(K / 2));
    if (M == 0 || N == 0) {
        // nothing to multiply; a computed activation scale is still defined
        if (nv && ts == REQAT_TS_COMPUTE && M == 0 &&
            launch_unit_scale(x_tensor_scale, reinterpret_cast<hipStream_t>(stream)) != hipSuccess)
            return REQAT_E_HIP;
        return REQAT_OK;
    }
    const int64_t nseg = nv ? linear_segments(M, K) : 0;
    uint16_t *table = reinterpret_cast<uint16_t *>(a_scales + round256((size_t)M * (size_t)(K / block_of(fmt))));
    reqat_status st = run_quant(fmt, x, M, K, ldx, a_codes, a_scales, nullptr, 0, x_tensor_scale, ts,
                                workspace, nseg <= kMaxSegments ? table : nullptr, nseg, stream, kCodes);
    if (st != REQAT_OK) return st;
    hipError_t e = packed && K > 0
                       ? launch_gemm_skinny(nv ? kNV : kMX, M, N, K, a_codes, a_scales, x_tensor_scale, w_codes,
                                            w_scales, w_tensor_scale, y, y_dtype == REQAT_DT_BF16, ldy, true,
                                            reinterpret_cast<hipStream_t>(stream))
                       : launch_gemm(nv ? kNV : kMX, M, N, K, a_codes, a_scales, x_tensor_scale, w_codes,
                                     w_scales, w_tensor_scale, y, y_dtype == REQAT_DT_BF16, ldy,
                                     reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

// Code and scale parts of a packed decode image (reqat_pack_w4a4).
const uint8_t *packed_scales(const void *packed, int64_t N, int64_t K) {
    const size_t code_bytes = (size_t)((N + 15) / 16) * (size_t)((K + 255) / 256) * 2048u;
    return reinterpret_cast<const uint8_t *>(packed) + code_bytes;
}

}  // namespace

extern "C" {

reqat_status reqat_linear_w4a4(reqat_format fmt, int64_t M, int64_t N, int64_t K, const void *x,
                               int64_t ldx, float *x_tensor_scale, reqat_tscale_mode ts,
                               const uint8_t *w_codes, const uint8_t *w_scales,
                               const float *w_tensor_scale, void *y, reqat_dtype y_dtype,
                               int64_t ldy, void *workspace, void *stream) {
    reqat_status st = check_linear(fmt, M, N, K, x, ldx, x_tensor_scale, ts, w_codes, w_scales, w_tensor_scale,
                                   y, y_dtype, ldy);
    if (st != REQAT_OK) return st;
    if (!workspace) return REQAT_E_NULL;
    if (reinterpret_cast<uintptr_t>(workspace) & 255u) return REQAT_E_ALIGN;
    return run_linear(fmt, M, N, K, x, ldx, x_tensor_scale, ts, w_codes, w_scales, w_tensor_scale, y, y_dtype,
                      ldy, workspace, stream);
}

size_t reqat_w4a4_packed_bytes(reqat_format fmt, int64_t N, int64_t K) {
    if (!fmt_ok(fmt) || N < 0 || K < 0 || K % 128) return 0;
    return skinny_packed_bytes(fmt == REQAT_FMT_NVFP4 ? kNV : kMX, N, K);
}

reqat_status reqat_pack_w4a4(reqat_format fmt, const uint8_t *w_codes, const uint8_t *w_scales, int64_t N, int64_t K,
                             void *packed, void *stream) {
    if (!fmt_ok(fmt)) return REQAT_E_ENUM;
    if (N < 0 || K < 0 || K % 128) return REQAT_E_SHAPE;
    if (N == 0 || K == 0) return REQAT_OK;
    if (!w_codes || !w_scales || !packed) return REQAT_E_NULL;
    if (!aligned16(w_codes) || !aligned16(w_scales) || !aligned16(packed)) return REQAT_E_ALIGN;
    const Fmt f = fmt == REQAT_FMT_NVFP4 ? kNV : kMX;
    const size_t pbytes = skinny_packed_bytes(f, N, K);
    if (overlaps(packed, pbytes, w_codes, (size_t)N * (size_t)(K / 2)) ||
        overlaps(packed, pbytes, w_scales, (size_t)N * (size_t)(K / block_of(fmt))))
        return REQAT_E_UNSUPPORTED;
    hipError_t e = launch_skinny_pack(f, w_codes, w_scales, N, K, reinterpret_cast<uint8_t *>(packed),
                                      reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

reqat_status reqat_gemm_w4a4_packed(reqat_format fmt, int64_t M, int64_t N, int64_t K, const uint8_t *a_codes,
                                    const uint8_t *a_scales, const float *a_tensor_scale, const void *packed,
                                    const float *b_tensor_scale, void *y, reqat_dtype y_dtype, int64_t ldy,
                                    void *stream) {
    if (!fmt_ok(fmt)) return REQAT_E_ENUM;
    if (y_dtype != REQAT_DT_F32 && y_dtype != REQAT_DT_BF16) return REQAT_E_ENUM;
    if (M < 0 || N < 0 || K < 0) return REQAT_E_SHAPE;
    if (K % 128) return REQAT_E_SHAPE;
    if (ldy < N) return REQAT_E_SHAPE;
    const bool nv = fmt == REQAT_FMT_NVFP4;
    if (!nv && (a_tensor_scale || b_tensor_scale)) return REQAT_E_UNSUPPORTED;
    if (nv && (!a_tensor_scale || !b_tensor_scale)) return REQAT_E_NULL;
    if (M > 64) return REQAT_E_UNSUPPORTED;
    if (M == 0 || N == 0) return REQAT_OK;
    if (!y) return REQAT_E_NULL;
    if (K > 0 && (!a_codes || !a_scales || !packed)) return REQAT_E_NULL;
    if (reinterpret_cast<uintptr_t>(y) & (y_dtype == REQAT_DT_BF16 ? 1u : 3u)) return REQAT_E_ALIGN;
    if (K > 0 && (!aligned16(a_codes) || !aligned16(a_scales) || !aligned16(packed))) return REQAT_E_ALIGN;
    if (nv && ((reinterpret_cast<uintptr_t>(a_tensor_scale) & 3u) ||
               (reinterpret_cast<uintptr_t>(b_tensor_scale) & 3u)))
        return REQAT_E_ALIGN;
    const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    // K == 0: the generic product writes zeros and reads no operand
    hipError_t e = K > 0 ? launch_gemm_skinny(nv ? kNV : kMX, M, N, K, a_codes, a_scales, a_tensor_scale,
                                              reinterpret_cast<const uint8_t *>(packed),
                                              packed_scales(packed, N, K), b_tensor_scale, y,
                                              y_dtype == REQAT_DT_BF16, ldy, true, st)
                         : launch_gemm(nv ? kNV : kMX, M, N, 0, nullptr, nullptr, a_tensor_scale, nullptr, nullptr,
                                       b_tensor_scale, y, y_dtype == REQAT_DT_BF16, ldy, st);
    return e == hipSuccess ? REQAT_OK : REQAT_E_HIP;
}

reqat_status reqat_linear_w4a4_packed(reqat_format fmt, int64_t M, int64_t N, int64_t K, const void *x,
                                      int64_t ldx, float *x_tensor_scale, reqat_tscale_mode ts, const void *packed,
                                      const float *w_tensor_scale, void *y, reqat_dtype y_dtype, int64_t ldy,
                                      void *workspace, void *stream) {
    const uint8_t *pc = reinterpret_cast<const uint8_t *>(packed);
    reqat_status st = check_linear(fmt, M, N, K, x, ldx, x_tensor_scale, ts, pc, pc, w_tensor_scale, y, y_dtype,
                                   ldy);
    if (st != REQAT_OK) return st;
    if (M > 64) return REQAT_E_UNSUPPORTED;
    if (!workspace) return REQAT_E_NULL;
    if (reinterpret_cast<uintptr_t>(workspace) & 255u) return REQAT_E_ALIGN;
    return run_linear(fmt, M, N, K, x, ldx, x_tensor_scale, ts, pc, pc ? packed_scales(packed, N, K) : nullptr,
                      w_tensor_scale, y, y_dtype, ldy, workspace, stream, true);
}

}  // extern "C"

// ------------------------------------------------------ linear layer without allocation
// For callers that cannot allocate: the linear layer's workspace is this
// file-scope array, one copy on each GPU the library runs on, held until the
// process ends.  In host code its name is only a stand-in; the kernels get the
// device address hipGetSymbolAddress returns, taken once per device with that
// device current.  Nothing in it needs clearing: every part (partial maxima,
// activation codes and scales, segment table) is written before it is read.
namespace {

__device__ __align__(256) uint8_t scratch[REQAT_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch[kMaxDevices] = {};

// Device address of `scratch` on the current device (nullptr on failure).
void *scratch_on_current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_scratch[dev] = p;
    }
    return g_scratch[dev];
}

}  // namespace

extern "C" {

reqat_status reqat_linear_w4a4_noalloc(reqat_format fmt, int64_t M, int64_t N, int64_t K, const void *x,
                                       int64_t ldx, float *x_tensor_scale, reqat_tscale_mode ts,
                                       const uint8_t *w_codes, const uint8_t *w_scales,
                                       const float *w_tensor_scale, void *y, reqat_dtype y_dtype, int64_t ldy,
                                       void *stream) {
    reqat_status st = check_linear(fmt, M, N, K, x, ldx, x_tensor_scale, ts, w_codes, w_scales, w_tensor_scale,
                                   y, y_dtype, ldy);
    if (st != REQAT_OK) return st;
    if (reqat_linear_workspace_bytes(fmt, M, K) > (size_t)REQAT_NOALLOC_SCRATCH_BYTES) return REQAT_E_TOO_LARGE;
    void *ws = scratch_on_current_device();
    if (!ws) return REQAT_E_HIP;
    return run_linear(fmt, M, N, K, x, ldx, x_tensor_scale, ts, w_codes, w_scales, w_tensor_scale, y, y_dtype,
                      ldy, ws, stream);
}

const char *reqat_status_str(reqat_status s) {
    switch (s) {
    case REQAT_OK: return "REQAT_OK";
    case REQAT_E_NULL: return "REQAT_E_NULL: a required pointer is NULL";
    case REQAT_E_SHAPE: return "REQAT_E_SHAPE: invalid size or leading dimension";
    case REQAT_E_ALIGN: return "REQAT_E_ALIGN: pointer or leading dimension misaligned";
    case REQAT_E_ENUM: return "REQAT_E_ENUM: unknown format, dtype or tensor-scale mode";
    case REQAT_E_UNSUPPORTED: return "REQAT_E_UNSUPPORTED: combination not supported";
    case REQAT_E_HIP: return "REQAT_E_HIP: HIP launch failed";
    case REQAT_E_TOO_LARGE: return "REQAT_E_TOO_LARGE: input exceeds the fixed scratch of the no-allocation entry point";
    }
    return "unknown reqat_status";
}

int reqat_abi_version(void) { return REQAT_ABI_VERSION; }

}  // extern "C"
