// Block quantization routines of the microscaled FP4 formats for gfx950,
// shared by the quantizer kernels and the fused decode linear layer: one lane
// quantizes one block (16 bfloat16 for NVFP4, 32 for MXFP4).
//
// Element rounding (round to nearest, ties to the even code, of |x| / (s g),
// saturating at 6) has two exact implementations:
//   * fast path: v_cvt_scalef32_pk_fp4_{bf16,f32}, which on gfx950 rounds
//     x / 2^e exactly that way for every finite bfloat16 x and every power of
//     two 2^-126..2^127 (the instruction reads only the exponent of its FP32
//     scale operand).  MXFP4 scales are powers of two and feed it directly.
//     For NVFP4 with a power-of-two g, s g = m * 2^e with m = 1.mmm (4 bits):
//     x is first multiplied by 1/m in FP32 and the product snapped to 16
//     significant bits (see the quantizer's notes for why that is exact).
//   * general path (NaN/Inf blocks, all-zero NVFP4 blocks, a non-power-of-two
//     global scale, extreme exponents): integer thresholds on the bfloat16
//     magnitude pattern (see fp4_device.h).
// Fake-quant decodes the codes again with v_cvt_scalef32_pk_{bf16,f32}_fp4
// (code * 2^e, exact) and, for NVFP4, multiplies by m (exact, <= 6 bits).
#pragma once

#include "fp4_device.h"
#include "internal.h"

namespace reqat {

namespace {

typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef float v2f __attribute__((ext_vector_type(2)));
typedef unsigned short us2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        uint32_t o = __shfl_xor(v, off, 64);
        v = v > o ? v : o;
    }
    return v;
}

// Max of the finite magnitudes of two packed bfloat16 values (non-finite -> 0).
__device__ __forceinline__ uint32_t finite_mag2(uint32_t w) {
    uint32_t lo = w & 0x7FFFu, hi = (w >> 16) & 0x7FFFu;
    lo = lo >= 0x7F80u ? 0u : lo;
    hi = hi >= 0x7F80u ? 0u : hi;
    return lo > hi ? lo : hi;
}

// Packed (two 16-bit lanes) maximum of the bfloat16 magnitudes of a 16-byte vector.
__device__ __forceinline__ us2 mag_max8(uint4 d, us2 m) {
    m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, d.x & 0x7FFF7FFFu));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, d.y & 0x7FFF7FFFu));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, d.z & 0x7FFF7FFFu));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(us2, d.w & 0x7FFF7FFFu));
    return m;
}

__device__ __forceinline__ uint32_t finite_max8(uint4 d, uint32_t m) {
    uint32_t a = finite_mag2(d.x), b = finite_mag2(d.y), c = finite_mag2(d.z), e = finite_mag2(d.w);
    a = a > b ? a : b; c = c > e ? c : e; a = a > c ? a : c;
    return m > a ? m : a;
}

// Grid values of the E2M1 magnitudes 0..7.
__device__ __forceinline__ float e2m1_mag_value(int m) {
    constexpr float v[8] = {0.0f, 0.5f, 1.0f, 1.5f, 2.0f, 3.0f, 4.0f, 6.0f};
    return v[m];
}

// ---------------------------------------------------------------- general path

// Codes of one block by integer thresholds; w holds the B bfloat16 inputs.
template <int B>
__device__ __forceinline__ void codes_general(const uint32_t (&w)[B / 2], const uint32_t (&U)[7],
                                              bool bad, uint32_t (&out)[B / 8]) {
#pragma unroll
    for (int q = 0; q < B / 8; ++q) {
        uint32_t word = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            uint32_t h = (j & 1) ? (w[4 * q + j / 2] >> 16) : (w[4 * q + j / 2] & 0xFFFFu);
            uint32_t c = bad ? 0u : (e2m1_code_mag(h & 0x7FFFu, U) | ((h >> 12) & 8u));
            word |= c << (4 * j);
        }
        out[q] = word;
    }
}

// Fake-quant of one block by thresholds; P[m] = bfloat16 pattern of grid value
// m.  Stores 16 bytes at a time, so no more than one vector of results is live.
template <int B>
__device__ __forceinline__ void fq_general(const uint32_t (&w)[B / 2], const uint32_t (&U)[7],
                                           const uint32_t (&P)[8], bool bad, uint16_t *ydst) {
#pragma unroll
    for (int q = 0; q < B / 8; ++q) {
        uint32_t o[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t word = w[4 * q + k];
            uint32_t res[2];
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                uint32_t h = hf ? (word >> 16) : (word & 0xFFFFu);
                uint32_t mag = h & 0x7FFFu;
                uint32_t v = P[0];
#pragma unroll
                for (int t = 0; t < 7; ++t) v = (mag >= U[t]) ? P[t + 1] : v;
                res[hf] = bad ? 0x7FC0u : (v | (h & 0x8000u));
            }
            o[k] = res[0] | (res[1] << 16);
        }
        reinterpret_cast<uint4 *>(ydst)[q] = make_uint4(o[0], o[1], o[2], o[3]);
    }
}

// Thresholds and output patterns for the general path of a block with scale S.
template <bool NEED_P>
__device__ __forceinline__ void general_plan(double S, bool zero, uint32_t (&U)[7], uint32_t (&P)[8]) {
    if (zero) {
#pragma unroll
        for (int i = 0; i < 7; ++i) U[i] = kNever;
#pragma unroll
        for (int m = 0; m < 8; ++m) P[m] = 0u;
        return;
    }
    thresholds_exact(S, U);
    if (NEED_P) {
#pragma unroll
        for (int m = 0; m < 8; ++m) P[m] = bf16_rne_from_double((double)e2m1_mag_value(m) * S);
    }
}

// ---------------------------------------------------------------- fast paths

template <int B>
__device__ __forceinline__ void codes_fast_mx(const uint32_t (&w)[B / 2], float p2,
                                              uint32_t (&out)[B / 8]) {
#pragma unroll
    for (int q = 0; q < B / 8; ++q) {
        uint32_t word = 0;
        word = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(word, __builtin_bit_cast(v2bf, w[4 * q + 0]), p2, 0);
        word = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(word, __builtin_bit_cast(v2bf, w[4 * q + 1]), p2, 1);
        word = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(word, __builtin_bit_cast(v2bf, w[4 * q + 2]), p2, 2);
        word = __builtin_amdgcn_cvt_scalef32_pk_fp4_bf16(word, __builtin_bit_cast(v2bf, w[4 * q + 3]), p2, 3);
        out[q] = word;
    }
}

// x * (1/m), snapped to 16 significant bits.
__device__ __forceinline__ float nv_prescale(uint32_t bits32, float inv_m) {
    float y = f32_from_bits(bits32) * inv_m;
    return f32_from_bits((bits_from_f32(y) + 0x80u) & 0xFFFFFF00u);
}

template <int B>
__device__ __forceinline__ void codes_fast_nv(const uint32_t (&w)[B / 2], float p2, float inv_m,
                                              uint32_t (&out)[B / 8]) {
#pragma unroll
    for (int q = 0; q < B / 8; ++q) {
        uint32_t word = 0;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const uint32_t v = w[4 * q + t];
            const float y0 = nv_prescale(v << 16, inv_m), y1 = nv_prescale(v & 0xFFFF0000u, inv_m);
            switch (t) {
            case 0: word = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word, y0, y1, p2, 0); break;
            case 1: word = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word, y0, y1, p2, 1); break;
            case 2: word = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word, y0, y1, p2, 2); break;
            default: word = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word, y0, y1, p2, 3); break;
            }
        }
        out[q] = word;
    }
}

// Decode a code word back to 4 dwords of packed bfloat16 (MXFP4: code * 2^e).
__device__ __forceinline__ void fq_fast_mx(uint32_t word, float p2, uint32_t *o) {
    o[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 0));
    o[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 1));
    o[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 2));
    o[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 3));
}

// NVFP4: code * 2^e in FP32, times m (exact), then the upper halves as bfloat16.
__device__ __forceinline__ uint32_t fq_pair_nv(v2f d, float m) {
    const uint32_t lo = bits_from_f32(d[0] * m), hi = bits_from_f32(d[1] * m);
    return __builtin_amdgcn_perm(hi, lo, 0x07060302u);
}

__device__ __forceinline__ void fq_fast_nv(uint32_t word, float p2, float m, uint32_t *o) {
    o[0] = fq_pair_nv(__builtin_amdgcn_cvt_scalef32_pk_f32_fp4(word, p2, 0), m);
    o[1] = fq_pair_nv(__builtin_amdgcn_cvt_scalef32_pk_f32_fp4(word, p2, 1), m);
    o[2] = fq_pair_nv(__builtin_amdgcn_cvt_scalef32_pk_f32_fp4(word, p2, 2), m);
    o[3] = fq_pair_nv(__builtin_amdgcn_cvt_scalef32_pk_f32_fp4(word, p2, 3), m);
}

// ---------------------------------------------------------------- one block

// The global scale as the block routine needs it.
struct GScale {
    float g;
    bool pow2;      // g = 2^kg exactly
    int kg;
};

__device__ __forceinline__ GScale make_gscale(float g) {
    const uint32_t gb = bits_from_f32(g);
    return GScale{g, (gb & 0x807FFFFFu) == 0u && (gb >> 23) != 0u, (int)(gb >> 23) - 127};
}

// Packed maximum of the bfloat16 magnitude patterns of a block (NaN/Inf give >= 0x7F80).
template <int B>
__device__ __forceinline__ uint32_t block_mag_max(const uint32_t (&w)[B / 2]) {
    us2 mx2 = __builtin_bit_cast(us2, w[0] & 0x7FFF7FFFu);
#pragma unroll
    for (int i = 1; i < B / 2; ++i)
        mx2 = __builtin_elementwise_max(mx2, __builtin_bit_cast(us2, w[i] & 0x7FFF7FFFu));
    return mx2[0] > mx2[1] ? mx2[0] : mx2[1];
}

template <int B>
__device__ __forceinline__ uint32_t block_finite_max(const uint32_t (&w)[B / 2]) {
    uint32_t m = 0;
#pragma unroll
    for (int i = 0; i < B / 2; ++i) {
        const uint32_t f = finite_mag2(w[i]);
        m = m > f ? m : f;
    }
    return m;
}

template <int B>
__device__ __forceinline__ void load_block(const uint16_t *src16, uint32_t (&w)[B / 2]) {
    const uint4 *src = reinterpret_cast<const uint4 *>(src16);
#pragma unroll
    for (int i = 0; i < B / 8; ++i) {
        const uint4 d = src[i];
        w[4 * i + 0] = d.x; w[4 * i + 1] = d.y; w[4 * i + 2] = d.z; w[4 * i + 3] = d.w;
    }
}

// Element offset of block `blk` (row-major blocks, nb per row) in a matrix with leading dimension ld.
__device__ __forceinline__ int64_t block_offset(int64_t blk, int64_t nb, int64_t cols, int64_t ld, int B,
                                                bool narrow) {
    if (ld == cols) return blk * B;
    const int64_t r = narrow ? (int64_t)((uint32_t)blk / (uint32_t)nb) : blk / nb;
    return r * ld + (blk - r * nb) * B;
}

// Scale byte of a block and, when the exact fast conversion applies, its parameters.
struct BlockPlan {
    uint32_t sbyte;
    bool fast;
    float p2, mant;     // s * g = mant * p2 (mant = 1 for MXFP4)
};

// FULL = false stops an NVFP4 block after the closed form (fast = false and no
// scale byte when it does not apply), leaving the rest to emit_general.
template <int FMT, int OUT, bool FULL = true>
__device__ __forceinline__ BlockPlan plan_block(uint32_t am, const GScale &G) {
    const bool bad = am >= 0x7F80u;                      // NaN or Inf somewhere in the block
    BlockPlan pl{0u, false, 1.0f, 1.0f};
    if (FMT == kMX) {
        pl.sbyte = bad ? 0xFFu : mx_scale_byte(am);
        pl.fast = !bad && pl.sbyte >= (OUT == kCodes ? 1u : 3u);
        pl.p2 = f32_from_bits(pl.sbyte << 23);
        return pl;
    }
    // g = 2^kg and a normal bfloat16 amax = A * 2^(Ef - 134) (A = 128..255):
    // the smallest 4-significant-bit value >= amax / 6 is
    // Q(A) * 2^(Ef - 134), Q(A) = 2*ceil(A/12) (A <= 180) or 4*ceil(A/24),
    // = (1 + f/8) * 2^j; when amax / (6g) rounded that way is a normal E4M3
    // value it is the scale (dividing by g only moves the exponent), and
    // s * g = Q(A) * 2^(Ef - 134) exactly.
    const uint32_t Ef = am >> 7;
    if (!bad && G.pow2 && Ef != 0u) {
        const uint32_t A = 128u + (am & 0x7Fu);
        const uint32_t j = A <= 180u ? 4u : 5u;
        const uint32_t f = (A <= 180u ? (A + 11u) / 12u : (A + 23u) / 24u) - 8u;
        const int ef = (int)(j + Ef) - 127 - G.kg;
        const int eS = (int)(j + Ef) - 134;
        if (ef >= 1 && (ef < 15 || (ef == 15 && f < 7u)) && eS >= -123 && eS <= 125) {
            pl.sbyte = ((uint32_t)ef << 3) | f;
            pl.p2 = f32_from_bits((uint32_t)(eS + 127) << 23);
            pl.mant = f32_from_bits(0x3F800000u | (f << 20));
            pl.fast = true;
            return pl;
        }
    }
    if (!FULL) return pl;
    pl.sbyte = bad ? 0x7Fu : nv_scale_byte(bf16_mag_value(am), G.g);
    const float S = e4m3_value(pl.sbyte) * G.g;
    pl.fast = !bad && pl.sbyte != 0u && G.pow2 && S >= 0x1p-123f && S <= 0x1p125f;
    pl.p2 = f32_from_bits(bits_from_f32(S) & 0x7F800000u);
    pl.mant = f32_from_bits((bits_from_f32(S) & 0x007FFFFFu) | 0x3F800000u);
    return pl;
}

// Fast path: codes (and scale byte), fake-quant values, or both, of one block.
template <int FMT, int OUT>
__device__ __forceinline__ void emit_fast(const uint32_t (&w)[(FMT == kMX ? 32 : 16) / 2], const BlockPlan &pl,
                                          int64_t blk, uint8_t *codes, uint8_t *scales, uint16_t *ydst) {
    constexpr int B = FMT == kMX ? 32 : 16;
    uint32_t cw[B / 8];
    if (FMT == kMX) codes_fast_mx<B>(w, pl.p2, cw);
    else codes_fast_nv<B>(w, pl.p2, __builtin_amdgcn_rcpf(pl.mant), cw);
    if (OUT != kFakeQuant) {
        uint8_t *dst = codes + blk * (B / 2);
        if constexpr (B == 16) *reinterpret_cast<uint2 *>(dst) = make_uint2(cw[0], cw[1]);
        else *reinterpret_cast<uint4 *>(dst) = make_uint4(cw[0], cw[1], cw[2], cw[3]);
        scales[blk] = (uint8_t)pl.sbyte;
    }
    if (OUT != kCodes) {
        uint4 *dst = reinterpret_cast<uint4 *>(ydst);
#pragma unroll
        for (int q = 0; q < B / 8; ++q) {
            uint32_t o[4];
            if (FMT == kMX) fq_fast_mx(cw[q], pl.p2, o);
            else fq_fast_nv(cw[q], pl.p2, pl.mant, o);
            dst[q] = make_uint4(o[0], o[1], o[2], o[3]);
        }
    }
}

// Blocks the block loop's fast test did not take (NaN/Inf blocks, zero NVFP4
// blocks, E4M3-subnormal scales, a non-power-of-two g, extreme exponents): the
// complete scale rule, then the fast conversion when it still applies and the
// threshold path otherwise.  The block is read from x again rather than kept
// alive in the caller, so this rarely taken code does not raise the register
// count of the loop around it.  Returns the scale byte.
template <int FMT, int OUT>
__device__ __forceinline__ uint32_t emit_general(const uint16_t *xsrc, const GScale &G, int64_t blk,
                                                 uint8_t *codes, uint8_t *scales, uint16_t *ydst) {
    constexpr int B = FMT == kMX ? 32 : 16;
    asm volatile("" : "+v"(xsrc));                      // a fresh load, not the loop's registers
    uint32_t w[B / 2];
    load_block<B>(xsrc, w);
    const uint32_t am = block_mag_max<B>(w);
    const bool bad = am >= 0x7F80u;
    const BlockPlan pl = plan_block<FMT, OUT>(am, G);
    if (pl.fast) {
        emit_fast<FMT, OUT>(w, pl, blk, codes, scales, ydst);
        return pl.sbyte;
    }
    const uint32_t sbyte = pl.sbyte;
    const double Sd = FMT == kMX ? __builtin_ldexp(1.0, (int)sbyte - 127)
                                 : (double)e4m3_value(sbyte) * (double)G.g;
    const bool zero = bad || (FMT == kNV && sbyte == 0u);
    uint32_t U[7], P[8];
    general_plan<OUT != kCodes>(Sd, zero, U, P);
    if (OUT != kFakeQuant) {
        uint32_t out[B / 8];
        codes_general<B>(w, U, bad, out);
        uint8_t *dst = codes + blk * (B / 2);
        if constexpr (B == 16) *reinterpret_cast<uint2 *>(dst) = make_uint2(out[0], out[1]);
        else *reinterpret_cast<uint4 *>(dst) = make_uint4(out[0], out[1], out[2], out[3]);
        scales[blk] = (uint8_t)sbyte;
    }
    if (OUT != kCodes) fq_general<B>(w, U, P, bad, ydst);
    return sbyte;
}

// Global scale of the whole tensor, computed by one workgroup of THREADS threads:
// the finite maximum over every element, eight 16-byte loads in flight per
// thread.  Loads past the end re-read the last vector (a maximum does not
// change), so they need no branch and all go out before the first wait.
template <int THREADS, int INFLIGHT = 16>
__device__ __forceinline__ float local_global_scale(const uint16_t *__restrict__ x, int64_t rows, int64_t cols,
                                                    int64_t ldx) {
    __shared__ uint32_t red[THREADS / 64];
    const uint32_t vpr = (uint32_t)(cols / 8), nvec = (uint32_t)rows * vpr;
    auto vec = [&](uint32_t i) {
        i = i < nvec ? i : nvec - 1;
        const uint32_t r = i / vpr;
        return *reinterpret_cast<const uint4 *>(x + (int64_t)r * ldx + (int64_t)(i - r * vpr) * 8);
    };
    // 16 loads in flight per thread: a tensor of up to 16 * THREADS vectors
    // (32K elements, a decode step's activations) costs one memory round trip
    uint32_t m = 0;
    for (uint32_t i = threadIdx.x; i < nvec; i += INFLIGHT * THREADS) {
        uint4 d[INFLIGHT];
#pragma unroll
        for (int u = 0; u < INFLIGHT; ++u) d[u] = vec(i + u * THREADS);
#pragma unroll
        for (int u = 0; u < INFLIGHT; ++u) m = finite_max8(d[u], m);
    }
    m = wave_max_u32(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    uint32_t r = red[0];
#pragma unroll
    for (int k = 1; k < THREADS / 64; ++k) r = r > red[k] ? r : red[k];
    return nv_global_scale(r);
}

}  // namespace

}  // namespace reqat
