// Internal launcher interface between the C ABI layer and the kernels.
// Every launcher only enqueues work on `stream` and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace reqat {

// Maximum number of partial maxima the absmax pass produces; the workspace
// holds one uint32 per partial.
#ifndef REQAT_MAX_PARTIALS
#define REQAT_MAX_PARTIALS 4096
#endif
constexpr int kMaxPartials = REQAT_MAX_PARTIALS;

// Segment-table capacity of the quantize workspace (segments of 64 blocks).
constexpr int64_t kMaxSegments = int64_t(1) << 19;

// Tensors of at most this many elements are small enough for every workgroup
// to read whole (<= 128 KB): their NVFP4 global scale is computed in one launch
// (kGLocal).
constexpr int64_t kLocalMaxElems = int64_t(1) << 16;

// Format selector shared by the launchers (same values as the C ABI enum).
enum Fmt : int { kNV = 0, kMX = 1 };

// Output selector for the block quantizer.
// kBoth writes codes, scales and fake-quant values in one pass over x.
enum QuantOut : int { kCodes = 0, kFakeQuant = 1, kBoth = 2 };

// Global-scale source for NVFP4.
enum GSrc : int { kGComputed = 0, kGGiven = 1, kGNone = 2 };

hipError_t launch_unit_scale(float *gptr, hipStream_t stream);

hipError_t launch_absmax(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                         uint32_t *partials, int *nparts_out, hipStream_t stream);

// NVFP4 with a computed g reads x once when the segment table (one uint16 per
// 64 blocks) has room for the tensor, and twice (absmax pass first) otherwise.
hipError_t launch_quantize(Fmt fmt, QuantOut out, const uint16_t *x, int64_t rows, int64_t cols,
                           int64_t ldx, uint8_t *codes, uint8_t *scales, uint16_t *y, int64_t ldy,
                           float *gptr, GSrc gsrc, uint32_t *partials, uint16_t *seg_table,
                           int64_t seg_capacity, hipStream_t stream);

// MXFP4 quantize / fake-quant of block-rotated rows (randomized Hadamard of 32).
hipError_t launch_quantize_rht(QuantOut out, const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                               uint32_t signs, uint8_t *codes, uint8_t *scales, uint16_t *y, int64_t ldy,
                               hipStream_t stream);

// W4A16: bfloat16 x [M][ldx] times MXFP4 weights [N][K/2] (+ scales [N][K/32]), K % 128 == 0.
// `workspace` holds gemm_w4a16_workspace_bytes(M, N, K) bytes of split-K partial sums.
int gemm_w4a16_splits(int64_t M, int64_t N, int64_t K);
size_t gemm_w4a16_workspace_bytes(int64_t M, int64_t N, int64_t K);
// packed: w_codes / w_scales are the code and scale parts of the packed image
// that launch_w4a16_pack writes (w4a16_packed_bytes(N, K) bytes).
hipError_t launch_gemm_w4a16(int64_t M, int64_t N, int64_t K, const uint16_t *x, int64_t ldx,
                             const uint8_t *w_codes, const uint8_t *w_scales, bool packed, void *y, bool y_bf16,
                             int64_t ldy, float *workspace, hipStream_t stream);
size_t w4a16_packed_bytes(int64_t N, int64_t K);
hipError_t launch_w4a16_pack(const uint8_t *codes, const uint8_t *scales, int64_t N, int64_t K, uint8_t *packed,
                             hipStream_t stream);

// KV4 (E1M2 elements, E4M3 block scales of 16, FP32 global scale) of x - shift.
// A computed g takes one pass over x and a fix-up kernel when the segment
// table (one uint16 per 64 blocks) has room for the tensor, else an absmax pass
// into `partials` (<= kMaxPartials) and then the quantizer.
hipError_t launch_kv4(QuantOut out, const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx, const float *shift,
                      uint8_t *codes, uint8_t *scales, uint16_t *y, int64_t ldy, float *gptr, bool computed,
                      uint32_t *partials, uint16_t *seg_table, hipStream_t stream);

// SEM loss: per-row statistics ([T][4]: H, NLL, lse, 0), weights [T], loss[4]
// (L, L_SFT, L_ent, tau); backward writes dL/dlogits.  V % 8 == 0.
hipError_t launch_sem_forward(const uint16_t *logits, int64_t T, int64_t V, int64_t ld, const int32_t *targets,
                              float lambda, float eps, float *stats, float *weights, float *loss,
                              hipStream_t stream);
hipError_t launch_sem_backward(const uint16_t *logits, int64_t T, int64_t V, int64_t ld, const int32_t *targets,
                               const float *stats, const float *weights, float lambda, float scale, void *grad,
                               bool grad_bf16, int64_t ldg, hipStream_t stream);

bool gemm_tile256_supported(Fmt fmt, int64_t M, int64_t N, int64_t K, int64_t ldy);
// Skinny product for M <= 64 (K % 128 == 0, K > 0).  packed: b_codes / b_scales
// are the code and scale parts of the image launch_skinny_pack writes
// (skinny_packed_bytes(fmt, N, K) bytes; the scales start 2048 G C bytes in).
hipError_t launch_gemm_skinny(Fmt fmt, int64_t M, int64_t N, int64_t K, const uint8_t *a_codes,
                              const uint8_t *a_scales, const float *ga, const uint8_t *b_codes,
                              const uint8_t *b_scales, const float *gb, void *y, bool y_bf16, int64_t ldy,
                              bool packed, hipStream_t stream);
size_t skinny_packed_bytes(Fmt fmt, int64_t N, int64_t K);
hipError_t launch_skinny_pack(Fmt fmt, const uint8_t *codes, const uint8_t *scales, int64_t N, int64_t K,
                              uint8_t *packed, hipStream_t stream);

hipError_t launch_gemm_tile256(Fmt fmt, int64_t M, int64_t N, int64_t K, const uint8_t *a_codes,
                               const uint8_t *a_scales, const float *ga, const uint8_t *b_codes,
                               const uint8_t *b_scales, const float *gb, void *y, bool y_bf16,
                               int64_t ldy, hipStream_t stream);

hipError_t launch_gemm(Fmt fmt, int64_t M, int64_t N, int64_t K, const uint8_t *a_codes,
                       const uint8_t *a_scales, const float *ga, const uint8_t *b_codes,
                       const uint8_t *b_scales, const float *gb, void *y, bool y_bf16, int64_t ldy,
                       hipStream_t stream);

}  // namespace reqat
