// Skinny W4A4 GEMM for gfx950 (M <= 64: decode-shaped products).
//
// Y[M][N] = g_a g_b * sum_k A^[m][k] B^[n][k] with few activation rows: the
// weights B dominate the traffic and must stream from HBM once, spread over
// every CU, with enough bytes in flight to cover the memory latency.
//
// Each 256-thread workgroup owns 32 rows of B (one 32-wide MFMA tile of the
// output) and all of K; its four waves take contiguous quarters of the K
// chunks (64 elements each) and their partial sums meet in LDS at the end.
// A lane loads its operands straight into registers in the MFMA layout
// (row = lane % 32, 32 consecutive K elements = 16 bytes per lane, lane half
// h = lane / 32 taking the chunk's second 32 elements), up to kDepth chunks
// ahead of the one it multiplies (for decode-sized K that is all of them, so
// a workgroup's whole share of B is in flight at once).  The activation tile
// (M rows padded to 32 or 64, padding rows re-reading the last real row and
// never stored) is reread by every workgroup from L2.
//
// MXFP4: v_mfma_scale_f32_32x32x64_f8f6f4 on the codes, the lane's 32
// elements being one MX block whose E8M0 byte rides along.
// NVFP4: the lane's 32 elements are two 16-element blocks; their E4M3 byte
// pair becomes two FP16 scales (v_cvt_scalef32_pk_f16_fp8, exact), codes are
// decoded at unit scale (v_cvt_scalef32_pk_f16_fp4) and multiplied by their
// block's scale (exact: <= 6 significant bits, range [2^-10, 2688]), and
// v_mfma_f32_32x32x16_f16 sums four 8-element steps per chunk.  A and B use
// the same assignment of K elements to lanes, so the sum over K is unchanged.
#include "fp4_device.h"
#include "internal.h"

namespace reqat {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kDepth = 8;                       // chunks in flight per wave

template <int MT>
struct Chunk {
    uint4 a[MT], b;
    uint32_t sa[MT], sb;
};

// Loads chunk c (64 K elements) of this lane's rows.
template <int FMT, int MT>
__device__ __forceinline__ void load_chunk(Chunk<MT> &q, int64_t c, int r, int h, int64_t M, int64_t N,
                                           int64_t n0, int64_t cpr, int64_t spr, const uint8_t *a_codes,
                                           const uint8_t *a_scales, const uint8_t *b_codes,
                                           const uint8_t *b_scales) {
    const int64_t cb = c * 32 + 16 * h;             // code byte of the lane's 32 elements
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int64_t row = (32 * mt + r) < M ? (32 * mt + r) : M - 1;
        q.a[mt] = *reinterpret_cast<const uint4 *>(a_codes + row * cpr + cb);
        if (FMT == kMX) q.sa[mt] = a_scales[row * spr + 2 * c + h];
        else q.sa[mt] = *reinterpret_cast<const uint16_t *>(a_scales + row * spr + 4 * c + 2 * h);
    }
    const int64_t nrow = (n0 + r) < N ? (n0 + r) : N - 1;
    q.b = *reinterpret_cast<const uint4 *>(b_codes + nrow * cpr + cb);
    if (FMT == kMX) q.sb = b_scales[nrow * spr + 2 * c + h];
    else q.sb = *reinterpret_cast<const uint16_t *>(b_scales + nrow * spr + 4 * c + 2 * h);
}

__device__ __forceinline__ v8i as_v8i(uint4 q) {
    return v8i{(int)q.x, (int)q.y, (int)q.z, (int)q.w, 0, 0, 0, 0};
}

__device__ __forceinline__ uint32_t pick(const uint4 &q, int s) {
    return s == 0 ? q.x : s == 1 ? q.y : s == 2 ? q.z : q.w;
}

// Eight codes (one dword) times a block scale (FP16, in both halves) -> FP16 (exact).
__device__ __forceinline__ v8h decode8(uint32_t c, v2h s) {
    v2h p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 0) * s;
    v2h p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 1) * s;
    v2h p2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 2) * s;
    v2h p3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 3) * s;
    return v8h{p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

template <int FMT, int MT>
__device__ __forceinline__ void mul_chunk(v16f (&acc)[MT], const Chunk<MT> &q) {
    if constexpr (FMT == kMX) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            acc[mt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(as_v8i(q.a[mt]), as_v8i(q.b), acc[mt], 4,
                                                                      4, 0, (int)q.sa[mt], 0, (int)q.sb);
    } else {
        const v2h fb = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q.sb, 1.0f, false);
        v2h fa[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) fa[mt] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(q.sa[mt], 1.0f, false);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            // steps 0,1: the lane's first 16-block; steps 2,3: its second
            const v2h sb = s < 2 ? v2h{fb[0], fb[0]} : v2h{fb[1], fb[1]};
            const v8h bv = decode8(pick(q.b, s), sb);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const v2h sa = s < 2 ? v2h{fa[mt][0], fa[mt][0]} : v2h{fa[mt][1], fa[mt][1]};
                acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(decode8(pick(q.a[mt], s), sa), bv, acc[mt],
                                                                 0, 0, 0);
            }
        }
    }
}

template <int FMT, int MT>
__global__ __launch_bounds__(kThreads) void gemm_skinny_kernel(
    int64_t M, int64_t N, int64_t K, const uint8_t *__restrict__ a_codes,
    const uint8_t *__restrict__ a_scales, const float *__restrict__ ga,
    const uint8_t *__restrict__ b_codes, const uint8_t *__restrict__ b_scales,
    const float *__restrict__ gb, void *__restrict__ y, int y_bf16, int64_t ldy) {
    constexpr int B = FMT == kMX ? 32 : 16;
    __shared__ float part[4][MT][16][64];           // per-wave partial sums

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 31, h = lane >> 5;
    const int64_t n0 = (int64_t)blockIdx.x * 32;
    const int64_t cpr = K / 2, spr = K / B;
    const int64_t nch = K / 64;
    const int64_t c0 = nch * wave / 4, my = nch * (wave + 1) / 4 - c0;   // this wave's chunks

    v16f acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = v16f{};

    Chunk<MT> q[kDepth];
#pragma unroll
    for (int j = 0; j < kDepth; ++j)
        if (j < my)
            load_chunk<FMT, MT>(q[j], c0 + j, r, h, M, N, n0, cpr, spr, a_codes, a_scales, b_codes,
                                b_scales);
    for (int64_t i0 = 0; i0 < my; i0 += kDepth) {
#pragma unroll
        for (int j = 0; j < kDepth; ++j) {
            const int64_t i = i0 + j;
            if (i < my) {
                mul_chunk<FMT, MT>(acc, q[j]);
                if (i + kDepth < my)
                    load_chunk<FMT, MT>(q[j], c0 + i + kDepth, r, h, M, N, n0, cpr, spr, a_codes,
                                        a_scales, b_codes, b_scales);
            }
        }
    }

    // the four waves' partial sums; wave w then finishes registers 4w .. 4w+3
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int k = 0; k < 16; ++k) part[wave][mt][k][lane] = acc[mt][k];
    __syncthreads();
    const float scale = FMT == kNV ? (*ga) * (*gb) : 1.0f;
    const int64_t col = n0 + r;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const int k = 4 * wave + kk;
            // D[i][j] of a 32 x 32 tile is in lane j + 32*((i/4)%2), register (i/8)*4 + i%4
            const int64_t row = 32 * mt + 8 * (k >> 2) + 4 * h + (k & 3);
            const float v = (part[0][mt][k][lane] + part[1][mt][k][lane] + part[2][mt][k][lane] +
                             part[3][mt][k][lane]) * scale;
            if (row < M && col < N) {
                if (y_bf16) reinterpret_cast<__bf16 *>(y)[row * ldy + col] = (__bf16)v;
                else reinterpret_cast<float *>(y)[row * ldy + col] = v;
            }
        }
}

template <int FMT, int MT>
hipError_t launch(int64_t M, int64_t N, int64_t K, const uint8_t *a_codes, const uint8_t *a_scales,
                  const float *ga, const uint8_t *b_codes, const uint8_t *b_scales, const float *gb, void *y,
                  bool y_bf16, int64_t ldy, hipStream_t stream) {
    const dim3 grid((unsigned)((N + 31) / 32)), block(kThreads);
    hipLaunchKernelGGL((gemm_skinny_kernel<FMT, MT>), grid, block, 0, stream, M, N, K, a_codes, a_scales, ga,
                       b_codes, b_scales, gb, y, (int)y_bf16, ldy);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_skinny(Fmt fmt, int64_t M, int64_t N, int64_t K, const uint8_t *a_codes,
                              const uint8_t *a_scales, const float *ga, const uint8_t *b_codes,
                              const uint8_t *b_scales, const float *gb, void *y, bool y_bf16, int64_t ldy,
                              hipStream_t stream) {
    if (fmt == kMX)
        return M <= 32 ? launch<kMX, 1>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy,
                                        stream)
                       : launch<kMX, 2>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy,
                                        stream);
    return M <= 32 ? launch<kNV, 1>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy, stream)
                   : launch<kNV, 2>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy, stream);
}

}  // namespace reqat
