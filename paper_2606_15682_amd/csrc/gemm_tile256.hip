// Large-tile W4A4 GEMM for gfx950 (K a multiple of 256).
//
// Workgroup tile 256 x 256, four waves of 128 x 128 (4 x 4 MFMA tiles of 32 x 32,
// 256 FP32 accumulators per lane).  K advances 256 elements per stage; each
// stage's packed codes (128 B per row) and scale bytes go global -> LDS with
// direct-to-LDS 16-byte loads (global_load_lds_dwordx4), double-buffered, so
// the next stage streams in while the current one is multiplied.
//
// LDS code layout: one row = 8 chunks of 16 B (32 E2M1 codes each); chunk c of
// row r is stored at chunk position c ^ (r & 7).  A wave's 16-byte operand read
// has 8 consecutive rows at the same logical chunk in each group of 8 lanes,
// which the XOR spreads over all 8 positions: no bank conflicts.  The
// direct-to-LDS write of one instruction is 1 KB contiguous (8 rows), and each
// lane fetches whichever 16 global bytes belong at its LDS slot.
//
// MXFP4 (v_mfma_scale_f32_32x32x64_f8f6f4, E2M1 x E2M1): in substep s of a
// stage, lanes 0-31 feed 32-block s and lanes 32-63 feed 32-block 4 + s of
// their row; a lane's four scale bytes for the stage are one dword and the
// instruction's op_sel picks byte s.  A and B use the same K assignment, so
// the sum over K is unchanged.
//
// NVFP4 (v_mfma_f32_32x32x16_f16): per 64-element chunk a lane loads 32 codes
// (16 B) and decodes 8 per MFMA step: v_cvt_scalef32_pk_f16_fp4 applies the
// power-of-two part of the E4M3 block scale (the instruction reads only the
// exponent of its FP32 scale operand) and v_pk_mul_f16 the 4-bit mantissa
// part; code * scale has <= 6 significant bits within FP16's normal range, so
// both steps are exact.  The per-byte (scale, mantissa) pairs come from a
// 256-entry table built in LDS at kernel start.
//
// Tile order: workgroups are dealt round-robin to the 8 XCDs, so workgroup b
// is mapped to the (b % 8)-th contiguous range of tiles, and tiles are walked
// in groups of 8 tile-rows, keeping the A and B panels a group reuses in the
// L2 of the XCD that owns it.
#include "fp4_device.h"
#include "internal.h"

namespace reqat {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kThreads = 256;
constexpr int TM = 256, TN = 256, KS = 256;
constexpr int ROW_BYTES = KS / 2;                       // 128
constexpr int CODE_BYTES = TM * ROW_BYTES;              // 32 KB per operand per stage
constexpr int GROUP_M = 8;

template <int FMT>
struct Layout {
    static constexpr int B = FMT == kMX ? 32 : 16;
    static constexpr int SB = KS / B;                   // scale bytes per row per stage (8 | 16)
    static constexpr int SCALE_BYTES = TM * SB;
    static constexpr int A_CODES = 0;
    static constexpr int B_CODES = CODE_BYTES;
    static constexpr int A_SC = 2 * CODE_BYTES;
    static constexpr int B_SC = 2 * CODE_BYTES + SCALE_BYTES;
    static constexpr int STAGE = 2 * CODE_BYTES + 2 * SCALE_BYTES;
    static constexpr int LUT = 2 * STAGE;               // NVFP4 scale table (256 x 8 B)
    static constexpr int TOTAL = 2 * STAGE + (FMT == kNV ? 2048 : 0);
};

__device__ __forceinline__ void g2l16(const void *g, uint8_t *l) {
    __builtin_amdgcn_global_load_lds(g, (lds_void *)l, 16, 0, 0);
}
__device__ __forceinline__ void g2l4(const void *g, uint8_t *l) {
    __builtin_amdgcn_global_load_lds(g, (lds_void *)l, 4, 0, 0);
}

__device__ __forceinline__ uint4 lds16(const uint8_t *p) { return *reinterpret_cast<const uint4 *>(p); }
__device__ __forceinline__ uint32_t lds4(const uint8_t *p) { return *reinterpret_cast<const uint32_t *>(p); }

// Issue the direct-to-LDS loads of one stage (this wave's share).  a/b point at
// the first row of the tile and at column k0; full tiles use one per-lane
// 32-bit offset plus wave-uniform steps, edge tiles clamp every row to the
// last valid one (those rows are loaded but never stored).
template <int FMT>
__device__ __forceinline__ void load_stage(uint8_t *buf, int wave, int lane, bool full_a,
                                           bool full_b, int64_t rows_a, int64_t rows_b,
                                           int64_t cpr, int64_t spr,
                                           const uint8_t *a_codes, const uint8_t *b_codes,
                                           const uint8_t *a_scales, const uint8_t *b_scales) {
    using L = Layout<FMT>;
    const int sub = lane >> 3;                            // row within the 8-row instruction
    const int c = (lane & 7) ^ sub;                       // logical chunk stored at this slot
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
        const int j = wave * 8 + jj;                      // 32 instructions per operand
        int ra = 8 * j + sub, rb = ra;
        if (!full_a) ra = ra < rows_a ? ra : (int)rows_a - 1;
        if (!full_b) rb = rb < rows_b ? rb : (int)rows_b - 1;
        g2l16(a_codes + (int64_t)ra * cpr + c * 16, buf + L::A_CODES + j * 1024);
        g2l16(b_codes + (int64_t)rb * cpr + c * 16, buf + L::B_CODES + j * 1024);
    }
    if constexpr (FMT == kMX) {
        // 8 scale bytes per row: 8 instructions of 64 x 4 B per operand, two per wave
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
            const int j = wave * 2 + jj;
            int ra = 32 * j + (lane >> 1), rb = ra;
            if (!full_a) ra = ra < rows_a ? ra : (int)rows_a - 1;
            if (!full_b) rb = rb < rows_b ? rb : (int)rows_b - 1;
            g2l4(a_scales + (int64_t)ra * spr + (lane & 1) * 4, buf + L::A_SC + j * 256);
            g2l4(b_scales + (int64_t)rb * spr + (lane & 1) * 4, buf + L::B_SC + j * 256);
        }
    } else {
        // 16 scale bytes per row: 4 instructions of 64 x 16 B per operand, one per wave
        int ra = 64 * wave + lane, rb = ra;
        if (!full_a) ra = ra < rows_a ? ra : (int)rows_a - 1;
        if (!full_b) rb = rb < rows_b ? rb : (int)rows_b - 1;
        g2l16(a_scales + (int64_t)ra * spr, buf + L::A_SC + wave * 1024);
        g2l16(b_scales + (int64_t)rb * spr, buf + L::B_SC + wave * 1024);
    }
}

// Byte address of logical 16-byte chunk c of tile row r.
__device__ __forceinline__ int code_off(int r, int c) { return r * ROW_BYTES + ((c ^ (r & 7)) << 4); }

template <int S>
__device__ __forceinline__ void mx_substep(v16f (&acc)[4][4], const uint8_t *buf, int rA0, int rB0,
                                           int h, const uint32_t (&sa)[4], const uint32_t (&sb)[4]) {
    using L = Layout<kMX>;
    v8i av[4], bv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint4 q = lds16(buf + L::A_CODES + code_off(rA0 + 32 * i, 4 * h + S));
        av[i] = v8i{(int)q.x, (int)q.y, (int)q.z, (int)q.w, 0, 0, 0, 0};
        uint4 p = lds16(buf + L::B_CODES + code_off(rB0 + 32 * i, 4 * h + S));
        bv[i] = v8i{(int)p.x, (int)p.y, (int)p.z, (int)p.w, 0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                av[i], bv[j], acc[i][j], 4, 4, S, (int)sa[i], S, (int)sb[j]);
}

// Eight codes (one dword) times an NVFP4 block scale -> FP16 (exact).
__device__ __forceinline__ v8h nv_decode8(uint32_t c, float pow2, v2h mant) {
    v2h p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, pow2, 0) * mant;
    v2h p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, pow2, 1) * mant;
    v2h p2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, pow2, 2) * mant;
    v2h p3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, pow2, 3) * mant;
    return v8h{p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

template <int FMT>
__global__ __launch_bounds__(kThreads, 1) void gemm_tile256_kernel(
    int64_t M, int64_t N, int64_t K, const uint8_t *__restrict__ a_codes,
    const uint8_t *__restrict__ a_scales, const float *__restrict__ ga,
    const uint8_t *__restrict__ b_codes, const uint8_t *__restrict__ b_scales,
    const float *__restrict__ gb, void *__restrict__ y, int y_bf16, int64_t ldy) {
    using L = Layout<FMT>;
    extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = lane >> 5;
    const int wm = wave >> 1, wn = wave & 1;

    // ---- tile order: XCD-contiguous ranges, then groups of GROUP_M tile-rows
    const int64_t tm_n = (M + TM - 1) / TM, tn_n = (N + TN - 1) / TN, T = tm_n * tn_n;
    const int64_t bid = blockIdx.x;
    const int64_t xcd = bid % 8, local = bid / 8, per = T / 8, rem = T % 8;
    const int64_t t = xcd * per + (xcd < rem ? xcd : rem) + local;
    const int64_t width = GROUP_M * tn_n;
    const int64_t first_m = (t / width) * GROUP_M;
    const int64_t gsz = (tm_n - first_m) < GROUP_M ? (tm_n - first_m) : GROUP_M;
    const int64_t tm = first_m + (t % width) % gsz, tn = (t % width) / gsz;
    const int64_t m0 = tm * TM, n0 = tn * TN;
    const int64_t cpr = K / 2, spr = K / L::B;

    if constexpr (FMT == kNV) {
        // (pow2 operand for the convert, mantissa pair for the multiply) per E4M3 byte
        uint32_t b = tid;
        float s = e4m3_value(b);
        uint32_t sb = bits_from_f32(s);
        _Float16 mh;
        if (s != s) mh = __builtin_bit_cast(_Float16, (uint16_t)0x7E00);
        else mh = (_Float16)f32_from_bits((sb & 0x807FFFFFu) | 0x3F800000u);
        uint32_t mm = (uint32_t)__builtin_bit_cast(uint16_t, mh);
        reinterpret_cast<uint2 *>(smem + L::LUT)[b] = make_uint2(sb, mm | (mm << 16));
    }

    v16f acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    const int64_t nst = K / KS;
    const int64_t rows_a = M - m0, rows_b = N - n0;
    const bool full_a = rows_a >= TM, full_b = rows_b >= TN;
    const uint8_t *ac = a_codes + m0 * cpr, *bc = b_codes + n0 * cpr;
    const uint8_t *as_ = a_scales + m0 * spr, *bs_ = b_scales + n0 * spr;
    load_stage<FMT>(smem, wave, lane, full_a, full_b, rows_a, rows_b, cpr, spr, ac, bc, as_, bs_);

    const int rA0 = wm * 128 + (lane & 31);               // this lane's A row in tile i: rA0 + 32 i
    const int rB0 = wn * 128 + (lane & 31);

    for (int64_t st = 0; st < nst; ++st) {
        uint8_t *buf = smem + (st & 1) * L::STAGE;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (st + 1 < nst) {
            const int64_t k1 = (st + 1) * KS;
            load_stage<FMT>(smem + ((st + 1) & 1) * L::STAGE, wave, lane, full_a, full_b, rows_a,
                            rows_b, cpr, spr, ac + k1 / 2, bc + k1 / 2, as_ + k1 / L::B,
                            bs_ + k1 / L::B);
        }

        if constexpr (FMT == kMX) {
            uint32_t sa[4], sb[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                sa[i] = lds4(buf + L::A_SC + (rA0 + 32 * i) * 8 + 4 * h);
                sb[i] = lds4(buf + L::B_SC + (rB0 + 32 * i) * 8 + 4 * h);
            }
            mx_substep<0>(acc, buf, rA0, rB0, h, sa, sb);
            mx_substep<1>(acc, buf, rA0, rB0, h, sa, sb);
            mx_substep<2>(acc, buf, rA0, rB0, h, sa, sb);
            mx_substep<3>(acc, buf, rA0, rB0, h, sa, sb);
        } else {
            const uint2 *lut = reinterpret_cast<const uint2 *>(smem + L::LUT);
#pragma unroll
            for (int q = 0; q < 4; ++q) {               // 64-element chunks
                uint4 ca[4], cb[4];
                uint2 ea[4][2], eb[4][2];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int ra = rA0 + 32 * i, rb = rB0 + 32 * i;
                    ca[i] = lds16(buf + L::A_CODES + code_off(ra, 2 * q + h));
                    cb[i] = lds16(buf + L::B_CODES + code_off(rb, 2 * q + h));
                    uint32_t wa = lds4(buf + L::A_SC + ra * 16 + 4 * q);
                    uint32_t wb = lds4(buf + L::B_SC + rb * 16 + 4 * q);
#pragma unroll
                    for (int hb = 0; hb < 2; ++hb) {
                        ea[i][hb] = lut[(wa >> (8 * (2 * h + hb))) & 0xFFu];
                        eb[i][hb] = lut[(wb >> (8 * (2 * h + hb))) & 0xFFu];
                    }
                }
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    v8h av[4], bv[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const uint32_t wa = s == 0 ? ca[i].x : s == 1 ? ca[i].y : s == 2 ? ca[i].z : ca[i].w;
                        const uint32_t wb = s == 0 ? cb[i].x : s == 1 ? cb[i].y : s == 2 ? cb[i].z : cb[i].w;
                        const uint2 e = ea[i][s >> 1], f = eb[i][s >> 1];
                        av[i] = nv_decode8(wa, f32_from_bits(e.x), __builtin_bit_cast(v2h, e.y));
                        bv[i] = nv_decode8(wb, f32_from_bits(f.x), __builtin_bit_cast(v2h, f.y));
                    }
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[i], bv[j], acc[i][j],
                                                                                0, 0, 0);
                }
            }
        }
    }

    // ---- epilogue: D[i][j] of a 32 x 32 tile is in lane j + 32*((i/4)%2), register (i/8)*4 + i%4
    float scale = 1.0f;
    if (FMT == kNV) scale = (*ga) * (*gb);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t gn = n0 + wn * 128 + j * 32 + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t gm = m0 + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
                if (gm < M && gn < N) {
                    const float v = acc[i][j][r] * scale;
                    if (y_bf16)
                        reinterpret_cast<uint16_t *>(y)[gm * ldy + gn] = (uint16_t)bf16_rne_from_float(v);
                    else
                        reinterpret_cast<float *>(y)[gm * ldy + gn] = v;
                }
            }
        }
}

}  // namespace

bool gemm_tile256_supported(int64_t M, int64_t N, int64_t K) {
    return K > 0 && K % KS == 0 && M > 0 && N > 0;
}

hipError_t launch_gemm_tile256(Fmt fmt, int64_t M, int64_t N, int64_t K, const uint8_t *a_codes,
                               const uint8_t *a_scales, const float *ga, const uint8_t *b_codes,
                               const uint8_t *b_scales, const float *gb, void *y, bool y_bf16,
                               int64_t ldy, hipStream_t stream) {
    const int64_t tiles = ((M + TM - 1) / TM) * ((N + TN - 1) / TN);
    if (fmt == kMX) {
        const size_t lds = Layout<kMX>::TOTAL;
        hipError_t e = hipFuncSetAttribute((const void *)gemm_tile256_kernel<kMX>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(gemm_tile256_kernel<kMX>, dim3((unsigned)tiles), dim3(kThreads), lds, stream,
                           M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, (int)y_bf16, ldy);
    } else {
        const size_t lds = Layout<kNV>::TOTAL;
        hipError_t e = hipFuncSetAttribute((const void *)gemm_tile256_kernel<kNV>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(gemm_tile256_kernel<kNV>, dim3((unsigned)tiles), dim3(kThreads), lds, stream,
                           M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, (int)y_bf16, ldy);
    }
    return hipGetLastError();
}

}  // namespace reqat
