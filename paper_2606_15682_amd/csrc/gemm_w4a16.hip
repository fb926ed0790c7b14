// W4A16 product for gfx950 (the MXFP4 W4A16 deployment setting: MXFP4 weights,
// bfloat16 activations):
//   Y[m][n] = sum_k x[m][k] * w^[n][k],   w^ = RN_bf16(E2M1(c) * 2^e),
// FP32 accumulation.  The weight is dequantized to the activation type in
// registers: v_cvt_scalef32_pk_bf16_fp4 returns exactly RN_bf16(code * 2^e) for
// every E8M0 scale byte 0..254 (overflow to Inf and bfloat16 subnormals
// included; checked on gfx950 for all 255 x 16 cases), and
// v_mfma_f32_16x16x32_bf16 multiplies exactly (it keeps subnormal inputs) and
// sums in FP32.  A NaN scale byte (0xFF) makes its 32 weights NaN.
//
// Decode-shaped work streams W once: a workgroup owns 16 rows of W (one
// 16-wide MFMA tile of the output; N/16 workgroups) and 16*MT rows of x.  Its
// WAVES waves take contiguous shares of K in 128-element chunks and meet in
// LDS at the end.  Every workgroup reads all of x (from L2): for M = 16 that is
// four times the weight bytes, and it, not HBM, bounds the rate (a probe of
// the same load pattern streams the weights alone at 4.8 TB/s and 0.95 TB/s
// with the x reads added).  In a chunk, lane l takes the 32-element MX block
// kg = l / 16 of W row n = l % 16 (16 code bytes + its scale byte) and the
// same 32 K positions of x row m = l % 16 (64 bytes); MFMA step s uses the
// lane's elements 8s .. 8s+7, so A and B agree on which K each lane holds and
// the sum over K is the product's.  Rows past M or N re-read the last real row
// and are never stored.
#include "fp4_device.h"
#include "internal.h"

namespace reqat {

namespace {

typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

#ifndef REQAT_W16_DEPTH
#define REQAT_W16_DEPTH 4
#endif
#ifndef REQAT_W16_WAVES
#define REQAT_W16_WAVES 8
#endif


template <int MT>
struct W16Chunk {
    uint4 w;             // 32 E2M1 codes of the lane's block
    uint32_t s;          // its E8M0 scale byte
    uint4 x[MT][4];      // 32 bfloat16 activations per x row tile
};

template <int MT>
__device__ __forceinline__ void load_w16(W16Chunk<MT> &q, int64_t c, int r, int kg, int64_t M, int64_t N,
                                         int64_t m0, int64_t n0, int64_t K, const uint16_t *x, int64_t ldx,
                                         const uint8_t *w_codes, const uint8_t *w_scales) {
    const int64_t blk = c * 4 + kg;                             // MX block index along K
    const int64_t nrow = (n0 + r) < N ? (n0 + r) : N - 1;
    q.w = *reinterpret_cast<const uint4 *>(w_codes + nrow * (K / 2) + blk * 16);
    q.s = w_scales[nrow * (K / 32) + blk];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int64_t row = (m0 + 16 * mt + r) < M ? (m0 + 16 * mt + r) : M - 1;
        const uint4 *xp = reinterpret_cast<const uint4 *>(x + row * ldx + blk * 32);
#pragma unroll
        for (int i = 0; i < 4; ++i) q.x[mt][i] = xp[i];
    }
}

__device__ __forceinline__ uint32_t pick4(const uint4 &q, int s) {
    return s == 0 ? q.x : s == 1 ? q.y : s == 2 ? q.z : q.w;
}

template <int MT>
__device__ __forceinline__ void mul_w16(v4f (&acc)[MT], const W16Chunk<MT> &q) {
    const float p2 = __builtin_bit_cast(float, q.s << 23);
    const bool nan = q.s == 0xFFu;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const uint32_t word = pick4(q.w, s);
        const v2bf d0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 0);
        const v2bf d1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 1);
        const v2bf d2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 2);
        const v2bf d3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 3);
        v8bf wb = v8bf{d0[0], d0[1], d1[0], d1[1], d2[0], d2[1], d3[0], d3[1]};
        if (nan) {
            const __bf16 qn = __builtin_bit_cast(__bf16, (uint16_t)0x7FC0u);
            wb = v8bf{qn, qn, qn, qn, qn, qn, qn, qn};
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, q.x[mt][s]), wb, acc[mt],
                                                             0, 0, 0);
    }
}

template <int MT, int DEPTH, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void gemm_w4a16_kernel(
    int64_t M, int64_t N, int64_t K, const uint16_t *__restrict__ x, int64_t ldx,
    const uint8_t *__restrict__ w_codes, const uint8_t *__restrict__ w_scales, void *__restrict__ y,
    int y_bf16, int64_t ldy) {
    __shared__ float part[WAVES][MT][4][64];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, kg = lane >> 4;
    const int64_t n0 = (int64_t)blockIdx.x * 16;
    const int64_t m0 = (int64_t)blockIdx.y * 16 * MT;
    const int64_t nch = K / 128;
    const int64_t c0 = nch * wave / WAVES, my = nch * (wave + 1) / WAVES - c0;   // this wave's chunks

    v4f acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = v4f{};

    auto chunk = [&](int64_t i) { return c0 + i; };
    W16Chunk<MT> q[DEPTH];
#pragma unroll
    for (int j = 0; j < DEPTH; ++j)
        if (j < my) load_w16<MT>(q[j], chunk(j), r, kg, M, N, m0, n0, K, x, ldx, w_codes, w_scales);
    for (int64_t i0 = 0; i0 < my; i0 += DEPTH) {
#pragma unroll
        for (int j = 0; j < DEPTH; ++j) {
            const int64_t i = i0 + j;
            if (i < my) {
                mul_w16<MT>(acc, q[j]);
                if (i + DEPTH < my)
                    load_w16<MT>(q[j], chunk(i + DEPTH), r, kg, M, N, m0, n0, K, x, ldx, w_codes, w_scales);
            }
        }
    }

    // the waves' partial sums, added in wave order; D[m][n] of a 16 x 16 tile
    // is in lane n + 16 * (m / 4), register m % 4.  Thread t < 256 finishes
    // register t / 64 of every row tile.
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) part[wave][mt][i][lane] = acc[mt][i];
    __syncthreads();
    if (tid >= 256) return;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int i = tid >> 6;                                 // register index 0..3
        float v = part[0][mt][i][lane];
#pragma unroll
        for (int w = 1; w < WAVES; ++w) v += part[w][mt][i][lane];
        const int64_t row = m0 + 16 * mt + 4 * (lane >> 4) + i;
        const int64_t col = n0 + (lane & 15);
        if (row < M && col < N) {
            if (y_bf16) reinterpret_cast<__bf16 *>(y)[row * ldy + col] = (__bf16)v;
            else reinterpret_cast<float *>(y)[row * ldy + col] = v;
        }
    }
}

template <int MT, int DEPTH, int WAVES>
hipError_t launch_mt(int64_t M, int64_t N, int64_t K, const uint16_t *x, int64_t ldx, const uint8_t *w_codes,
                     const uint8_t *w_scales, void *y, bool y_bf16, int64_t ldy, hipStream_t stream) {
    const dim3 grid((unsigned)((N + 15) / 16), (unsigned)((M + 16 * MT - 1) / (16 * MT))), block(64 * WAVES);
    hipLaunchKernelGGL((gemm_w4a16_kernel<MT, DEPTH, WAVES>), grid, block, 0, stream, M, N, K, x, ldx, w_codes,
                       w_scales, y, (int)y_bf16, ldy);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_w4a16(int64_t M, int64_t N, int64_t K, const uint16_t *x, int64_t ldx,
                             const uint8_t *w_codes, const uint8_t *w_scales, void *y, bool y_bf16,
                             int64_t ldy, hipStream_t stream) {
    if (M == 0 || N == 0) return hipSuccess;
    if (M <= 16) return launch_mt<1, REQAT_W16_DEPTH, REQAT_W16_WAVES>(M, N, K, x, ldx, w_codes, w_scales, y, y_bf16,
                                                                      ldy, stream);
    if (M <= 32) return launch_mt<2, 3, 8>(M, N, K, x, ldx, w_codes, w_scales, y, y_bf16, ldy, stream);
    return launch_mt<4, 2, 4>(M, N, K, x, ldx, w_codes, w_scales, y, y_bf16, ldy, stream);
}

}  // namespace reqat
