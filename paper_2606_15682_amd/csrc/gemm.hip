// W4A4 block-scaled GEMM for gfx950: Y[M][N] = g_a g_b * sum_k A^[m][k] B^[n][k].
//
// Both operands arrive as packed E2M1 codes with K contiguous (A = activations
// [M][K/2], B = weights [N][K/2]) plus per-block scale bytes, so both MFMA
// operands are read K-contiguous straight from the same row-major layout.
//
// MXFP4: the contraction runs on the block-scaled FP4 MFMA
// (v_mfma_scale_f32_32x32x64_f8f6f4, E2M1 x E2M1): each lane feeds 32
// consecutive K-elements of one row (16 bytes) together with that 32-block's
// E8M0 scale byte, which is exactly the MXFP4 block, so the scales go to the
// matrix core unchanged.
//
// NVFP4: the matrix core's scale input is a power of two per 32 elements,
// while NVFP4 carries an E4M3 scale (4 significant bits) per 16 elements, so
// its scales cannot ride on the FP4 MFMA exactly.  Instead each code is
// decoded with its block scale into FP16: |code| * s has at most 6
// significant bits and lies in [2^-10, 2688], inside FP16's normal range, so
// the decode is exact, and the FP16 MFMA (v_mfma_f32_32x32x16_f16) sums the
// exact products in FP32.  One 32x32x16 step covers exactly one 16-element
// NVFP4 block per row.  g_a * g_b is applied in the epilogue.
//
// Tiling: 128 x 128 output tile per 256-thread workgroup, 2 x 2 waves of
// 64 x 64 (2 x 2 MFMA tiles of 32 x 32), K staged 128 elements at a time
// through LDS.
#include "fp4_device.h"
#include "internal.h"

namespace reqat {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int BM = 128, BN = 128, BK = 128;   // tile sizes in elements
constexpr int ROWB = BK / 2;                  // code bytes per row per stage (64)
constexpr int PITCH = ROWB + 16;              // padded LDS row pitch (bytes)

// E2M1 code nibble -> FP16 value (exact).
__device__ __forceinline__ _Float16 e2m1_to_f16(uint32_t nib) {
    uint32_t mag = nib & 7u, e = mag >> 1, man = mag & 1u;
    uint32_t bits = e ? (((e + 14u) << 10) | (man << 9)) : (man ? 0x3800u : 0u);
    bits |= (nib & 8u) << 12;
    return __builtin_bit_cast(_Float16, (uint16_t)bits);
}

// Eight codes (one dword) times an NVFP4 block scale, as FP16 (exact).
__device__ __forceinline__ v8h decode8_nv(uint32_t c, _Float16 s) {
    v8h r;
#pragma unroll
    for (int j = 0; j < 8; ++j) r[j] = e2m1_to_f16((c >> (4 * j)) & 0xFu) * s;
    return r;
}

template <int FMT>
__global__ __launch_bounds__(kThreads) void gemm_w4a4_kernel(
    int64_t M, int64_t N, int64_t K, const uint8_t *__restrict__ a_codes,
    const uint8_t *__restrict__ a_scales, const float *__restrict__ ga,
    const uint8_t *__restrict__ b_codes, const uint8_t *__restrict__ b_scales,
    const float *__restrict__ gb, void *__restrict__ y, int y_bf16, int64_t ldy) {
    constexpr int B = FMT == kMX ? 32 : 16;
    constexpr int SPR = BK / B;                   // scale bytes per row per stage (4 or 8)

    __shared__ __attribute__((aligned(16))) uint8_t sA[BM * PITCH];
    __shared__ __attribute__((aligned(16))) uint8_t sB[BN * PITCH];
    __shared__ __attribute__((aligned(16))) uint8_t sAs[BM * SPR];
    __shared__ __attribute__((aligned(16))) uint8_t sBs[BN * SPR];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
    const int64_t cpr = K / 2, spr = K / B;      // code / scale bytes per global row

    v16f acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    for (int64_t k0 = 0; k0 < K; k0 += BK) {
        // ---- global -> registers (zero rows outside M / N)
        uint4 ra[2], rb[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            int id = tid + kThreads * i, r = id >> 2, c = id & 3;
            int64_t gm = m0 + r, gn = n0 + r;
            ra[i] = gm < M ? *reinterpret_cast<const uint4 *>(a_codes + gm * cpr + k0 / 2 + c * 16)
                           : make_uint4(0, 0, 0, 0);
            rb[i] = gn < N ? *reinterpret_cast<const uint4 *>(b_codes + gn * cpr + k0 / 2 + c * 16)
                           : make_uint4(0, 0, 0, 0);
        }
        uint2 rs = make_uint2(0, 0);
        {
            int r = tid & 127;
            bool isA = tid < 128;
            int64_t g = (isA ? m0 : n0) + r;
            const uint8_t *sp = isA ? a_scales : b_scales;
            if (g < (isA ? M : N)) {
                if (SPR == 8) rs = *reinterpret_cast<const uint2 *>(sp + g * spr + k0 / B);
                else rs.x = *reinterpret_cast<const uint32_t *>(sp + g * spr + k0 / B);
            }
        }
        __syncthreads();   // the previous stage's reads are done
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            int id = tid + kThreads * i, r = id >> 2, c = id & 3;
            *reinterpret_cast<uint4 *>(sA + r * PITCH + c * 16) = ra[i];
            *reinterpret_cast<uint4 *>(sB + r * PITCH + c * 16) = rb[i];
        }
        {
            int r = tid & 127;
            uint8_t *dst = (tid < 128 ? sAs : sBs) + r * SPR;
            if (SPR == 8) *reinterpret_cast<uint2 *>(dst) = rs;
            else *reinterpret_cast<uint32_t *>(dst) = rs.x;
        }
        __syncthreads();

        if constexpr (FMT == kMX) {
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {           // two 64-wide K chunks per stage
                const int half = lane >> 5;            // which 32-block of the chunk
                v8i av[2], bv[2];
                int as[2], bs[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    int ra_ = wm * 64 + i * 32 + (lane & 31);
                    uint4 q = *reinterpret_cast<const uint4 *>(sA + ra_ * PITCH + kc * 32 + half * 16);
                    av[i] = v8i{(int)q.x, (int)q.y, (int)q.z, (int)q.w, 0, 0, 0, 0};
                    as[i] = sAs[ra_ * SPR + kc * 2 + half];
                    int rb_ = wn * 64 + i * 32 + (lane & 31);
                    uint4 p = *reinterpret_cast<const uint4 *>(sB + rb_ * PITCH + kc * 32 + half * 16);
                    bv[i] = v8i{(int)p.x, (int)p.y, (int)p.z, (int)p.w, 0, 0, 0, 0};
                    bs[i] = sBs[rb_ * SPR + kc * 2 + half];
                }
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                            av[i], bv[j], acc[i][j], 4, 4, 0, as[i], 0, bs[j]);
            }
        } else {
#pragma unroll
            for (int kk = 0; kk < 8; ++kk) {           // one NVFP4 block per step
                const int half = lane >> 5;            // which 8 elements of the block
                v8h av[2], bv[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    int ra_ = wm * 64 + i * 32 + (lane & 31);
                    uint32_t ca = *reinterpret_cast<const uint32_t *>(sA + ra_ * PITCH + kk * 8 + half * 4);
                    _Float16 sa = (_Float16)e4m3_value(sAs[ra_ * SPR + kk]);
                    av[i] = decode8_nv(ca, sa);
                    int rb_ = wn * 64 + i * 32 + (lane & 31);
                    uint32_t cb = *reinterpret_cast<const uint32_t *>(sB + rb_ * PITCH + kk * 8 + half * 4);
                    _Float16 sb = (_Float16)e4m3_value(sBs[rb_ * SPR + kk]);
                    bv[i] = decode8_nv(cb, sb);
                }
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[i], bv[j], acc[i][j],
                                                                            0, 0, 0);
            }
        }
    }

    // ---- epilogue: D[i][j] of a 32x32 tile sits in lane j + 32*((i/4)%2), register (i/8)*4 + i%4
    float scale = 1.0f;
    if (FMT == kNV) scale = (*ga) * (*gb);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                int64_t gm = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                int64_t gn = n0 + wn * 64 + j * 32 + (lane & 31);
                if (gm < M && gn < N) {
                    float v = acc[i][j][r] * scale;
                    if (y_bf16)
                        reinterpret_cast<uint16_t *>(y)[gm * ldy + gn] = (uint16_t)bf16_rne_from_float(v);
                    else
                        reinterpret_cast<float *>(y)[gm * ldy + gn] = v;
                }
            }
}

}  // namespace

hipError_t launch_gemm(Fmt fmt, int64_t M, int64_t N, int64_t K, const uint8_t *a_codes,
                       const uint8_t *a_scales, const float *ga, const uint8_t *b_codes,
                       const uint8_t *b_scales, const float *gb, void *y, bool y_bf16, int64_t ldy,
                       hipStream_t stream) {
    if (M == 0 || N == 0) return hipSuccess;
    if (M > 64 && gemm_tile256_supported(fmt, M, N, K, ldy))
        return launch_gemm_tile256(fmt, M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y,
                                   y_bf16, ldy, stream);
    if (M <= 64 && K > 0)
        return launch_gemm_skinny(fmt, M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16,
                                  ldy, false, stream);
    dim3 grid((unsigned)((N + BN - 1) / BN), (unsigned)((M + BM - 1) / BM)), block(kThreads);
    if (fmt == kMX)
        hipLaunchKernelGGL(gemm_w4a4_kernel<kMX>, grid, block, 0, stream, M, N, K, a_codes, a_scales,
                           ga, b_codes, b_scales, gb, y, (int)y_bf16, ldy);
    else
        hipLaunchKernelGGL(gemm_w4a4_kernel<kNV>, grid, block, 0, stream, M, N, K, a_codes, a_scales,
                           ga, b_codes, b_scales, gb, y, (int)y_bf16, ldy);
    return hipGetLastError();
}

}  // namespace reqat
