// Skinny W4A4 GEMM for gfx950 (M <= 64: decode-shaped products).
//
// Y[M][N] = g_a g_b * sum_k A^[m][k] B^[n][k] with few activation rows: the
// weights B dominate the traffic and must stream from memory once, spread
// over every CU, with enough bytes in flight to cover the latency.
//
// Each 512-thread workgroup (eight waves) owns 16 rows of B and all of K.  K
// is cut into chunks of 256 elements (one 128-byte line of codes and 16 (NV)
// or 8 (MX) scale bytes per row) and the waves take contiguous shares of the
// chunks; their partial sums meet in LDS at the end.  In a chunk, lane
// (r, g) = (lane % 16, lane / 16) holds the 64 consecutive elements
// 64g .. 64g+63 of row r: 32 code bytes (two 16-byte loads) and the scale
// bytes of those elements in one aligned 4-byte (NV: four 16-blocks) or
// 2-byte (MX: two 32-blocks) load.  Loading a row's scales four blocks at a
// time, instead of two, and a line of codes per row per chunk measured
// 8.2 -> 5.7 us on the 16 x 8960 x 1536 decode product.  Loads run up to
// kDepth chunks ahead of the chunk being multiplied.
//
// From row-major weights each 16-byte weight load of a wave still touches 16
// rows (64 scattered bytes of each row's line).  Served weights can instead
// be re-laid out once into a packed image (skinny_pack_kernel) in which a
// unit of 16 rows x 256 elements holds the 2 KB of codes in lane order and,
// after all code units, its scale bytes in lane order: every weight load of
// a wave is then 1 KB (codes) or 256 / 128 bytes (scales) of consecutive
// bytes (kPacked; 6.2 -> 5.2 us on the decode product above, weights from
// HBM).  Only the weight addresses differ, so both forms give the same
// result bit for bit.
//
// Operands go to the 16 x 16 MFMAs in the layout the loads produce: in step s
// a lane feeds elements 8s .. 8s+7 (NV, v_mfma_f32_16x16x32_f16) or the
// 32-block s (MX, v_mfma_scale_f32_16x16x128_f8f6f4) of its 64; A and B use
// the same assignment of K elements to lanes, so the sum over K is unchanged.
// Activation rows (up to four 16-row tiles, rows past M re-reading the last
// real row and never stored) are read by every workgroup from L2.  K % 128 ==
// 0, so the last chunk is whole or half; lanes past K contribute exactly 0.
//
// MXFP4: the lane's 32-block goes to the matrix core as E2M1 codes with its
// E8M0 byte (op_sel picks it from the 2-byte load).
// NVFP4: the lane's four E4M3 bytes become FP16 scales
// (v_cvt_scalef32_pk_f16_fp8, exact for every E4M3 value), codes are decoded
// at unit scale (v_cvt_scalef32_pk_f16_fp4) and multiplied by their block's
// scale (exact: <= 6 significant bits, range [2^-10, 2688]).
#include "fp4_device.h"
#include "internal.h"

namespace reqat {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kDepth = 2;                       // chunks in flight per wave
constexpr int kRows = 16;                       // rows of B per workgroup

template <int MT>
struct Chunk {
    uint4 a0[MT], a1[MT], b0, b1;               // 32 code bytes per row (two 16-byte halves)
    uint32_t sa[MT], sb;                        // scale bytes of the lane's 64 elements
    bool ok;                                    // the lane's elements lie inside K
};

// Loads chunk c of the lane's rows.  The row pointers exclude the lane's
// offset in the chunk; a lane past K loads the chunk's first elements (always
// in range) and mul_chunk discards them, so every load is unconditional and
// no select waits on a load before the chunk is multiplied.  kPacked: bc / bs
// point at the lane's place in the workgroup's first unit of the packed image
// (units of a row group are consecutive; the 2 KB of codes are two 1 KB
// halves, one per load), where a lane past K finds zeros.
template <int FMT, int MT, bool kPacked>
__device__ __forceinline__ void load_chunk(Chunk<MT> &q, int64_t c, int g, int64_t K,
                                           const uint8_t *const (&ac)[MT], const uint8_t *const (&as)[MT],
                                           const uint8_t *bc, const uint8_t *bs) {
    constexpr int SB = FMT == kMX ? 8 : 16;     // scale bytes per row per chunk
    constexpr int LSB = SB / 4;                 // scale bytes per lane per chunk
    q.ok = 256 * c + 64 * g < K;
    const int gg = q.ok ? g : 0;
    const int64_t co = 128 * c + 32 * gg, so = SB * c + LSB * gg;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        q.a0[mt] = *reinterpret_cast<const uint4 *>(ac[mt] + co);
        q.a1[mt] = *reinterpret_cast<const uint4 *>(ac[mt] + co + 16);
        if constexpr (FMT == kMX) q.sa[mt] = *reinterpret_cast<const uint16_t *>(as[mt] + so);
        else q.sa[mt] = *reinterpret_cast<const uint32_t *>(as[mt] + so);
    }
    const int64_t bco = kPacked ? 2048 * c : co, bso = kPacked ? 16 * SB * c : so;
    q.b0 = *reinterpret_cast<const uint4 *>(bc + bco);
    q.b1 = *reinterpret_cast<const uint4 *>(bc + bco + (kPacked ? 1024 : 16));
    if constexpr (FMT == kMX) q.sb = *reinterpret_cast<const uint16_t *>(bs + bso);
    else q.sb = *reinterpret_cast<const uint32_t *>(bs + bso);
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

// FP16 scale of 16-block `blk` (0..3) of the lane's chunk, in both halves.
__device__ __forceinline__ v2h nv_scale(v2h lo, v2h hi, int blk) {
    const v2h p = blk < 2 ? lo : hi;
    return (blk & 1) ? v2h{p[1], p[1]} : v2h{p[0], p[0]};
}

// A lane past K contributes exactly 0: its scale bytes are taken as 0 (NV: the
// decoded operands are then +-0; MX: finite 2^-127) and, for MX, its
// activation codes as 0 too, so every product it feeds is 0.
template <int FMT, int MT>
__device__ __forceinline__ void mul_chunk(v4f (&acc)[MT], const Chunk<MT> &q) {
    const uint32_t sb = q.ok ? q.sb : 0u;
    if constexpr (FMT == kMX) {
        const uint4 z = uint4{0, 0, 0, 0};
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const uint32_t sa = q.ok ? q.sa[mt] : 0u;
            const uint4 a0 = q.ok ? q.a0[mt] : z, a1 = q.ok ? q.a1[mt] : z;
            acc[mt] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(as_v8i(a0), as_v8i(q.b0), acc[mt], 4, 4,
                                                                       0, (int)sa, 0, (int)sb);
            acc[mt] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(as_v8i(a1), as_v8i(q.b1), acc[mt], 4, 4,
                                                                       1, (int)sa, 1, (int)sb);
        }
    } else {
        const v2h fb01 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sb, 1.0f, false);
        const v2h fb23 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sb, 1.0f, true);
        v2h fa01[MT], fa23[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const uint32_t sa = q.ok ? q.sa[mt] : 0u;
            fa01[mt] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sa, 1.0f, false);
            fa23[mt] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sa, 1.0f, true);
        }
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            // elements 8s .. 8s+7 of the lane's 64 lie in its 16-block s / 2
            const int blk = s >> 1;
            const v8h bv = decode8(pick(s < 4 ? q.b0 : q.b1, s & 3), nv_scale(fb01, fb23, blk));
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const v8h av = decode8(pick(s < 4 ? q.a0[mt] : q.a1[mt], s & 3), nv_scale(fa01[mt], fa23[mt], blk));
                acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bv, acc[mt], 0, 0, 0);
            }
        }
    }
}

template <int FMT, int MT, bool kPacked>
__global__ __launch_bounds__(kThreads) void gemm_skinny_kernel(
    int64_t M, int64_t N, int64_t K, const uint8_t *__restrict__ a_codes,
    const uint8_t *__restrict__ a_scales, const float *__restrict__ ga,
    const uint8_t *__restrict__ b_codes, const uint8_t *__restrict__ b_scales,
    const float *__restrict__ gb, void *__restrict__ y, int y_bf16, int64_t ldy) {
    constexpr int B = FMT == kMX ? 32 : 16;
    __shared__ float part[kWaves][MT][4][64];       // per-wave partial sums

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, g = lane >> 4;
    const int64_t n0 = (int64_t)blockIdx.x * kRows;
    const int64_t cpr = K / 2, spr = K / B;
    const int64_t nch = (K + 255) / 256;
    const int64_t c0 = nch * wave / kWaves, my = nch * (wave + 1) / kWaves - c0;   // this wave's chunks

    const uint8_t *ac[MT], *as[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int64_t row = (16 * mt + r) < M ? (16 * mt + r) : M - 1;
        ac[mt] = a_codes + row * cpr;
        as[mt] = a_scales + row * spr;
    }
    const uint8_t *bc, *bs;
    if constexpr (kPacked) {
        // b_codes / b_scales: the code and scale parts of the packed image
        constexpr int SU = FMT == kMX ? 128 : 256;  // scale bytes per unit
        bc = b_codes + (int64_t)blockIdx.x * nch * 2048 + lane * 16;
        bs = b_scales + (int64_t)blockIdx.x * nch * SU + lane * (SU / 64);
    } else {
        const int64_t brow = (n0 + r) < N ? n0 + r : N - 1;
        bc = b_codes + brow * cpr;
        bs = b_scales + brow * spr;
    }

    v4f acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = v4f{0, 0, 0, 0};

    Chunk<MT> q[kDepth];
#pragma unroll
    for (int j = 0; j < kDepth; ++j)
        if (j < my) load_chunk<FMT, MT, kPacked>(q[j], c0 + j, g, K, ac, as, bc, bs);
    for (int64_t i0 = 0; i0 < my; i0 += kDepth) {
#pragma unroll
        for (int j = 0; j < kDepth; ++j) {
            const int64_t i = i0 + j;
            if (i < my) {
                mul_chunk<FMT, MT>(acc, q[j]);
                if (i + kDepth < my) load_chunk<FMT, MT, kPacked>(q[j], c0 + i + kDepth, g, K, ac, as, bc, bs);
            }
        }
    }

#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int k = 0; k < 4; ++k) part[wave][mt][k][lane] = acc[mt][k];
    __syncthreads();
    const float scale = FMT == kNV ? (*ga) * (*gb) : 1.0f;
    for (int idx = tid; idx < MT * 256; idx += kThreads) {
        const int mt = idx >> 8, k = (idx >> 6) & 3, l = idx & 63;
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) v += part[w][mt][k][l];
        v *= scale;
        // D[m][n] of a 16 x 16 tile sits in lane n + 16 * (m / 4), register m % 4
        const int64_t m = 16 * mt + 4 * (l >> 4) + k, n = n0 + (l & 15);
        if (m < M && n < N) {
            if (y_bf16) reinterpret_cast<__bf16 *>(y)[m * ldy + n] = (__bf16)v;
            else reinterpret_cast<float *>(y)[m * ldy + n] = v;
        }
    }
}

// Packed image of skinny_pack_kernel: per 16-row group g and 256-element chunk
// c (unit u = g C + c, C = ceil(K / 256)), 2 KB of codes at 2048 u, in the
// order the lanes load them: byte 1024 h + 16 l + i is code byte
// 128 c + 32 (l / 16) + 16 h + i of row 16 g + l % 16; after all code units,
// 16 SB scale bytes per unit at 2048 G C + 16 SB u: byte (SB / 4) l + j is
// scale byte SB c + (SB / 4)(l / 16) + j of that row (SB = 16 NV, 8 MX).
// Rows past N and elements past K are zero.
template <int FMT>
__global__ __launch_bounds__(256) void skinny_pack_kernel(const uint8_t *__restrict__ codes,
                                                          const uint8_t *__restrict__ scales, int64_t N, int64_t K,
                                                          uint8_t *__restrict__ packed) {
    constexpr int SB = FMT == kMX ? 8 : 16;     // scale bytes per row per chunk
    constexpr int LSB = SB / 4;                 // scale bytes per lane per chunk
    const int64_t nch = (K + 255) / 256, units = (N + 15) / 16 * nch;
    const int64_t cpr = K / 2, spr = K / (FMT == kMX ? 32 : 16);
    uint8_t *pscales = packed + units * 2048;
    for (int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x; p < units * 128; p += (int64_t)gridDim.x * 256) {
        const int64_t u = p >> 7, g = u / nch, c = u - g * nch;
        const int h = (int)(p >> 6) & 1, l = (int)(p & 63), q = l >> 4;
        const int64_t row = 16 * g + (l & 15), cb = 128 * c + 32 * q + 16 * h, sb = SB * c + LSB * q;
        uint4 v = uint4{0u, 0u, 0u, 0u};
        if (row < N && cb < cpr) v = *reinterpret_cast<const uint4 *>(codes + row * cpr + cb);
        *reinterpret_cast<uint4 *>(packed + u * 2048 + h * 1024 + l * 16) = v;
        if (h == 0) {
            const bool in = row < N && sb < spr;
            if constexpr (FMT == kMX)
                *reinterpret_cast<uint16_t *>(pscales + u * 128 + l * 2) =
                    in ? *reinterpret_cast<const uint16_t *>(scales + row * spr + sb) : (uint16_t)0;
            else
                *reinterpret_cast<uint32_t *>(pscales + u * 256 + l * 4) =
                    in ? *reinterpret_cast<const uint32_t *>(scales + row * spr + sb) : 0u;
        }
    }
}

template <int FMT, int MT, bool kPacked>
hipError_t launch(int64_t M, int64_t N, int64_t K, const uint8_t *a_codes, const uint8_t *a_scales,
                  const float *ga, const uint8_t *b_codes, const uint8_t *b_scales, const float *gb, void *y,
                  bool y_bf16, int64_t ldy, hipStream_t stream) {
    const dim3 grid((unsigned)((N + kRows - 1) / kRows)), block(kThreads);
    hipLaunchKernelGGL((gemm_skinny_kernel<FMT, MT, kPacked>), grid, block, 0, stream, M, N, K, a_codes, a_scales,
                       ga, b_codes, b_scales, gb, y, (int)y_bf16, ldy);
    return hipGetLastError();
}

template <int FMT, bool kPacked>
hipError_t launch_fmt(int64_t M, int64_t N, int64_t K, const uint8_t *a_codes, const uint8_t *a_scales,
                      const float *ga, const uint8_t *b_codes, const uint8_t *b_scales, const float *gb, void *y,
                      bool y_bf16, int64_t ldy, hipStream_t stream) {
    if (M <= 16)
        return launch<FMT, 1, kPacked>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy, stream);
    if (M <= 32)
        return launch<FMT, 2, kPacked>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy, stream);
    if (M <= 48)
        return launch<FMT, 3, kPacked>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy, stream);
    return launch<FMT, 4, kPacked>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy, stream);
}

}  // namespace

hipError_t launch_gemm_skinny(Fmt fmt, int64_t M, int64_t N, int64_t K, const uint8_t *a_codes,
                              const uint8_t *a_scales, const float *ga, const uint8_t *b_codes,
                              const uint8_t *b_scales, const float *gb, void *y, bool y_bf16, int64_t ldy,
                              bool packed, hipStream_t stream) {
    if (M < 1 || M > 64 || K <= 0 || K % 128) return hipErrorInvalidValue;
    if (fmt == kMX)
        return packed ? launch_fmt<kMX, true>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy,
                                              stream)
                      : launch_fmt<kMX, false>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy,
                                               stream);
    return packed ? launch_fmt<kNV, true>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy,
                                          stream)
                  : launch_fmt<kNV, false>(M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, y_bf16, ldy,
                                           stream);
}

size_t skinny_packed_bytes(Fmt fmt, int64_t N, int64_t K) {
    return (size_t)((N + 15) / 16) * (size_t)((K + 255) / 256) * (fmt == kMX ? 2176u : 2304u);
}

hipError_t launch_skinny_pack(Fmt fmt, const uint8_t *codes, const uint8_t *scales, int64_t N, int64_t K,
                              uint8_t *packed, hipStream_t stream) {
    const int64_t pieces = (N + 15) / 16 * ((K + 255) / 256) * 128;
    if (pieces == 0) return hipSuccess;
    const int64_t blocks = (pieces + 255) / 256;
    const dim3 grid((unsigned)(blocks < 4096 ? blocks : 4096)), block(256);
    if (fmt == kMX)
        hipLaunchKernelGGL(skinny_pack_kernel<kMX>, grid, block, 0, stream, codes, scales, N, K, packed);
    else
        hipLaunchKernelGGL(skinny_pack_kernel<kNV>, grid, block, 0, stream, codes, scales, N, K, packed);
    return hipGetLastError();
}

}  // namespace reqat
