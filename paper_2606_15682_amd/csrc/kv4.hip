// KV-cache quantizer for gfx950 (the 4-bit KV cache of the NVFP4 W4A4KV4
// setting, Sec. 4.3 "Additional implementation details"; Q-FIT's post-RoPE
// shift, Sec. 4.3, K~ = R(K_pre / s) - m):
//   d = RN_fp32(x - m[c])                       (m an FP32 vector over channels, optional)
//   E1M2 elements (magnitudes 0, 0.5, ..., 3.5), an E4M3 scale per 16
//   channels (the smallest with block_amax <= 3.5 * s * g) and an FP32 global
//   scale g (given, or the smallest power of two 2^k, k >= -126, with
//   tensor_amax <= 3.5 * 448 * 2^k), elements rounded to nearest, ties to the
//   even code; a block with a non-finite d gets scale 0x7F and zero codes.
// Every decision compares d (FP32, exact in FP64) with products of at most
// 31 significant bits, so FP64 comparisons decide exactly; with a power-of-two
// g (every computed g) the element thresholds have at most 8 bits and the
// comparisons run in FP32, exactly as well.  With a power-of-two g the codes
// are normally taken by rounding d * rcp(s g / 2) (see kv4_emit), and the
// threshold comparisons run only for blocks that rounding cannot decide.
//
// One lane per 16-channel block; a wave step takes kKvU adjacent segments of
// 64 blocks.  The shift vector is staged in LDS once per workgroup (up to
// kShiftLds channels; from global memory beyond).  With a power-of-two g the
// scale byte is computed in FP32 as well, with an exact correction step.  A
// computed g takes one pass over x under per-segment reference scales and a
// fix-up kernel (kv4_quantize_deferred_kernel, kv4_fixup_kernel); a tensor
// beyond the segment table takes two passes instead (the partial maxima of
// |d| per workgroup, then the quantizer, whose workgroups fold them).
#include <type_traits>

#include "fp4_device.h"
#include "internal.h"

namespace reqat {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxKvGroups = kMaxPartials;
// Workgroups of the quantize kernels (grid-stride beyond): four per CU, so a
// wave takes several steps.  Each workgroup stages the shift vector in LDS and
// the one-pass kernel writes one partial maximum per workgroup, which the
// fix-up folds; on 32768 x 1024 keys this cap took the computed-g quantize
// from 31.5 to 28.2 us and its fake-quant from 36.9 to 32.0 us (4096 or 512
// workgroups were slower).
constexpr int kMaxKvQuantGroups = 1024;
#ifndef REQAT_KV4_U
#define REQAT_KV4_U 2
#endif
// Adjacent 64-block segments per wave step in the quantize kernels, their
// loads all issued before any block is computed.
constexpr int kKvU = REQAT_KV4_U;
// Shift vectors of up to this many channels are staged in LDS once per
// workgroup: read per block from global memory, the 64 shift bytes of a
// 16-channel block would double the bytes the vector memory path moves.
constexpr int kShiftLds = 4096;

// Where a kernel reads the shift from.
enum ShiftSrc : int { kNoShift = 0, kShiftGlobal = 1, kShiftLdsSrc = 2 };

// Copies shift[0 .. cols) into LDS (cols % 4 == 0, cols <= kShiftLds).
__device__ __forceinline__ void kv4_stage_shift(const float *__restrict__ shift, int64_t cols, float4 *lds) {
    const float4 *src = reinterpret_cast<const float4 *>(shift);
    for (int i = threadIdx.x; i < (int)(cols / 4); i += kThreads) lds[i] = src[i];
    __syncthreads();
}

__device__ __forceinline__ uint32_t kv4_wave_max(uint32_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t o = __shfl_xor(v, off, 64);
        v = v > o ? v : o;
    }
    return v;
}

// The 16 shifted values of block `blk` (FP32); the shift comes from global
// memory (SRC = kShiftGlobal), from its LDS copy (kShiftLdsSrc) or is absent.
template <int SRC>
__device__ __forceinline__ void kv4_load(const uint16_t *__restrict__ x, const float *__restrict__ shift,
                                         const float4 *lds_shift, int64_t blk, int64_t nb, int64_t ldx, bool narrow,
                                         float (&d)[16]) {
    const int64_t r = narrow ? (int64_t)((uint32_t)blk / (uint32_t)nb) : blk / nb;
    const int64_t c0 = (blk - r * nb) * 16;
    const uint4 *src = reinterpret_cast<const uint4 *>(x + r * ldx + c0);
    const uint4 a = src[0], b = src[1];
    const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        d[2 * i] = f32_from_bits(w[i] << 16);
        d[2 * i + 1] = f32_from_bits(w[i] & 0xFFFF0000u);
    }
    if (SRC != kNoShift) {
        const float4 *sp = SRC == kShiftLdsSrc ? lds_shift + c0 / 4 : reinterpret_cast<const float4 *>(shift + c0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float4 m = sp[i];
            d[4 * i + 0] = d[4 * i + 0] - m.x;
            d[4 * i + 1] = d[4 * i + 1] - m.y;
            d[4 * i + 2] = d[4 * i + 2] - m.z;
            d[4 * i + 3] = d[4 * i + 3] - m.w;
        }
    }
}

// Largest finite |d| over the shifted tensor, one partial per workgroup.
template <int SRC>
__global__ __launch_bounds__(kThreads) void kv4_absmax_kernel(const uint16_t *__restrict__ x, int64_t rows,
                                                              int64_t cols, int64_t ldx,
                                                              const float *__restrict__ shift,
                                                              uint32_t *__restrict__ partials) {
    __shared__ float4 lds_shift[SRC == kShiftLdsSrc ? kShiftLds / 4 : 1];
    if (SRC == kShiftLdsSrc) kv4_stage_shift(shift, cols, lds_shift);
    const int64_t nb = cols / 16, total = rows * nb;
    const bool narrow = total < (int64_t(1) << 32);
    uint32_t m = 0;
    for (int64_t blk = (int64_t)blockIdx.x * kThreads + threadIdx.x; blk < total;
         blk += (int64_t)gridDim.x * kThreads) {
        float d[16];
        kv4_load<SRC>(x, shift, lds_shift, blk, nb, ldx, narrow, d);
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const uint32_t a = bits_from_f32(d[j]) & 0x7FFFFFFFu;
            if (a < 0x7F800000u && a > m) m = a;
        }
    }
    __shared__ uint32_t red[kThreads / 64];
    m = kv4_wave_max(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = red[0];
        for (int i = 1; i < kThreads / 64; ++i) r = r > red[i] ? r : red[i];
        partials[blockIdx.x] = r;
    }
}

// Global scale from the FP32 pattern of the tensor amax: smallest 2^k, k >= -126,
// with amax <= 1568 * 2^k (1568 = 1.53125 * 2^10; 0.53125 = fraction bits 0x440000).
__device__ __forceinline__ float kv4_global_scale(uint32_t am) {
    if (am == 0u) return 1.0f;
    int E;
    uint32_t frac;
    if ((am >> 23) != 0u) {
        E = (int)(am >> 23) - 127;
        frac = am & 0x7FFFFFu;
    } else {
        const int p = 31 - __builtin_clz(am);
        E = p - 149;
        frac = (am << (23 - p)) & 0x7FFFFFu;
    }
    int k = frac <= 0x440000u ? E - 10 : E - 9;
    if (k < -126) k = -126;
    return f32_from_bits((uint32_t)(k + 127) << 23);
}

// The largest of the first nparts partial maxima (<= kMaxKvGroups), for the
// whole workgroup: every thread's loads are issued before any is waited on.
__device__ __forceinline__ uint32_t kv4_fold_partials(const uint32_t *__restrict__ partials, int nparts) {
    __shared__ uint32_t red[kThreads / 64];
    constexpr int kPer = (kMaxKvGroups + kThreads - 1) / kThreads;
    uint32_t p[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int i = (int)threadIdx.x + j * kThreads;
        p[j] = i < nparts ? partials[i] : 0u;
    }
    uint32_t m = 0u;
#pragma unroll
    for (int j = 0; j < kPer; ++j) m = m > p[j] ? m : p[j];
    m = kv4_wave_max(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    uint32_t r = red[0];
#pragma unroll
    for (int i = 1; i < kThreads / 64; ++i) r = r > red[i] ? r : red[i];
    return r;
}

// Smallest positive finite E4M3 s with amax <= 3.5 * s * g (0x7E when none).
__device__ __forceinline__ uint32_t kv4_scale_byte(double a, double g) {
    uint32_t b = e4m3_ceil_byte(a / (3.5 * g));
    if (b < 0x7Eu && !(a <= 3.5 * (double)e4m3_value(b) * g)) b += 1u;
    else if (b > 1u && a <= 3.5 * (double)e4m3_value(b - 1u) * g) b -= 1u;
    return b;
}

// FP32 counterpart for a power-of-two g = 2^kg in [2^-126, 2^100]: q = a / (3.5 g)
// to within a few ulp, its E4M3 ceiling, then one exact correction.  Every
// bound 3.5 * s * g has at most 7 significant bits and lies in
// [7 * 2^-136, 1568 * 2^100], so it is exact in FP32 (subnormals included).
__device__ __forceinline__ uint32_t kv4_scale_byte_f32(float a, float g, int kg) {
    const float q = __builtin_ldexpf(a * (2.0f / 7.0f), -kg);
    uint32_t b;
    if (!(q <= 448.0f)) {
        b = 0x7Eu;
    } else if (q <= 0x1p-9f) {
        b = 0x01u;
    } else {
        const uint32_t qb = bits_from_f32(q);           // normal: q > 2^-9
        int E = (int)(qb >> 23) - 127;
        if (E < -6) {
            b = (uint32_t)__builtin_ceilf(q * 0x1p9f);  // E4M3 subnormals: multiples of 2^-9 (1..8)
        } else {
            uint32_t m = ((qb & 0x7FFFFFu) + 0xFFFFFu) >> 20;   // ceil of the top three mantissa bits
            if (m == 8u) {
                m = 0u;
                E += 1;
            }
            b = ((uint32_t)(E + 7) << 3) | m;
            b = b > 0x7Eu ? 0x7Eu : b;
        }
    }
    if (b < 0x7Eu && !(a <= 3.5f * e4m3_value(b) * g)) b += 1u;
    else if (b > 1u && a <= 3.5f * e4m3_value(b - 1u) * g) b -= 1u;
    return b;
}

// E1M2 magnitude code (0..7) of |v| / S, nearest with ties to the even code.
__device__ __forceinline__ uint32_t e1m2_mag(double a, double S) {
    uint32_t m = 7u;
#pragma unroll
    for (int i = 6; i >= 0; --i) {
        const double t = (0.5 * i + 0.25) * S;
        if (a < t || (a == t && (i & 1) == 0)) m = (uint32_t)i;
    }
    return m;
}

// The same with FP32 thresholds, exact when S = s * g is a power-of-two
// multiple of an E4M3 value inside the FP32 range: (0.5 i + 0.25) * S has at
// most 8 significant bits and lies in [2^-137, 2^111].
__device__ __forceinline__ uint32_t e1m2_mag_f32(float a, float S) {
    uint32_t m = 7u;
#pragma unroll
    for (int i = 6; i >= 0; --i) {
        const float t = (0.5f * (float)i + 0.25f) * S;
        if (a < t || (a == t && (i & 1) == 0)) m = (uint32_t)i;
    }
    return m;
}

// The global scale g as the element paths use it: the FP32 path needs a
// power of two in [2^-126, 2^100] (every computed g is a power of two), so
// that every threshold and decoded value is exact in FP32.
struct Kv4G {
    float g;
    double gd;
    bool f32;
    int kg;
};

__device__ __forceinline__ Kv4G kv4_make_g(float g) {
    Kv4G G;
    G.g = g;
    G.gd = (double)g;
    const uint32_t gb = bits_from_f32(g);
    G.f32 = (gb & 0x807FFFFFu) == 0u && gb >= 0x00800000u && gb <= ((100u + 127u) << 23);
    G.kg = (int)(gb >> 23) - 127;
    return G;
}

// Largest finite |d| of a block (FP32 pattern; 0 when none).
__device__ __forceinline__ uint32_t kv4_finite_max(const float (&d)[16]) {
    uint32_t m = 0u;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const uint32_t a = bits_from_f32(d[j]) & 0x7FFFFFFFu;
        if (a < 0x7F800000u && a > m) m = a;
    }
    return m;
}

// Exact element codes of one block (sign in bit 3, magnitude 0..7) by
// threshold comparisons: FP32 thresholds for a power-of-two g, FP64 otherwise.
__device__ __forceinline__ void kv4_exact_codes(const float (&d)[16], bool bad, uint32_t sbyte, const Kv4G &G,
                                                double S, float Sf, uint32_t (&c)[16]) {
    if (G.f32) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const uint32_t sign = (bits_from_f32(d[j]) >> 28) & 8u;
            c[j] = bad ? 0u : (sbyte == 0u ? sign : (e1m2_mag_f32(__builtin_fabsf(d[j]), Sf) | sign));
        }
    } else {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const uint32_t sign = (bits_from_f32(d[j]) >> 28) & 8u;
            c[j] = bad ? 0u : (sbyte == 0u ? sign : (e1m2_mag(__builtin_fabs((double)d[j]), S) | sign));
        }
    }
}

// Packs eight codes (sign in bit 3, magnitude 0..7 = |c|) of the integral
// values c[0..8) into a word, code j in bits 4j..4j+3: magnitudes converted
// into bytes (even j in one word, odd j in another), signs gathered from the
// top bytes of the FP32 patterns.
__device__ __forceinline__ uint32_t kv4_pack8(const float *c) {
    uint32_t pe = 0u, po = 0u;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        pe = __builtin_amdgcn_cvt_pk_u8_f32(__builtin_fabsf(c[2 * k]), k, pe);
        po = __builtin_amdgcn_cvt_pk_u8_f32(__builtin_fabsf(c[2 * k + 1]), k, po);
    }
    // top byte of c[2k] (resp. c[2k+1]) into byte k; 0x0C selects a zero byte
    const uint32_t se = __builtin_amdgcn_perm(bits_from_f32(c[2]), bits_from_f32(c[0]), 0x0C0C0703u) |
                        __builtin_amdgcn_perm(bits_from_f32(c[6]), bits_from_f32(c[4]), 0x07030C0Cu);
    const uint32_t so = __builtin_amdgcn_perm(bits_from_f32(c[3]), bits_from_f32(c[1]), 0x0C0C0703u) |
                        __builtin_amdgcn_perm(bits_from_f32(c[7]), bits_from_f32(c[5]), 0x07030C0Cu);
    return (pe | (po << 4)) | ((se >> 4) & 0x08080808u) | (so & 0x80808080u);
}

// Quantizes block blk (its 16 shifted values d, am = the largest |d| pattern,
// NaN and Inf included) under G and stores codes and scale byte, or the
// fake-quant values; returns the scale byte.
//
// Fast path (power-of-two g, finite block, H = s g / 2 zero or a normal FP32
// value, am <= 7 H, i.e. the scale did not saturate): the code magnitude is
// the integer nearest |d| / H, ties to even (at most 7).  q = d * rcp(H) is
// within 2^-19 of d / H (the reciprocal's ulp and one rounding, |q| <= 7), so
// rint(q) is the code with d's sign (-0 for a small negative d) unless d / H
// lies within 2^-19 of a half-integer; q - rint(q) is exact, and a block with
// some |q - rint(q)| >= 0.5 - 2^-17 takes the threshold path instead.  The
// fake-quant value c * H has at most 7 significant bits and is normal or
// zero, so its top 16 bits are the bfloat16 value.
template <int OUT>
__device__ __forceinline__ uint32_t kv4_emit(const float (&d)[16], uint32_t am, int64_t blk, int64_t nb, bool narrow,
                                             const Kv4G &G, uint8_t *__restrict__ codes, uint8_t *__restrict__ scales,
                                             uint16_t *__restrict__ y, int64_t ldy) {
    const bool bad = am >= 0x7F800000u;
    const uint32_t sbyte = bad ? 0x7Fu
                           : am == 0u ? 0u
                           : G.f32 ? kv4_scale_byte_f32(f32_from_bits(am), G.g, G.kg)
                                   : kv4_scale_byte((double)f32_from_bits(am), G.gd);
    const float Sf = e4m3_value(sbyte) * G.g;               // exact on the FP32 path
    const float H = 0.5f * Sf;
    const bool fast_ok = G.f32 && !bad && (sbyte == 0u || (H >= 0x1p-126f && f32_from_bits(am) <= 7.0f * H));
    const float rh = (fast_ok && sbyte != 0u) ? __builtin_amdgcn_rcpf(H) : 0.0f;
    float cf[16];
    float emax = 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const float q = d[j] * rh;
        cf[j] = __builtin_rintf(q);
        emax = __builtin_fmaxf(emax, __builtin_fabsf(q - cf[j]));
    }
    const bool exact = !fast_ok || emax >= 0.5f - 0x1p-17f;
    if (OUT == kCodes) {
        uint32_t lo = kv4_pack8(cf), hi = kv4_pack8(cf + 8);
        if (exact) {
            uint32_t c[16];
            kv4_exact_codes(d, bad, sbyte, G, (double)e4m3_value(sbyte) * G.gd, Sf, c);
            lo = 0;
            hi = 0;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                lo |= c[j] << (4 * j);
                hi |= c[8 + j] << (4 * j);
            }
        }
        *reinterpret_cast<uint2 *>(codes + blk * 8) = make_uint2(lo, hi);
        scales[blk] = (uint8_t)sbyte;
    } else {
        const int64_t r = narrow ? (int64_t)((uint32_t)blk / (uint32_t)nb) : blk / nb;
        uint32_t o[8];
#pragma unroll
        for (int i = 0; i < 8; ++i)   // bytes 2, 3 of each product: the bfloat16 patterns
            o[i] = __builtin_amdgcn_perm(bits_from_f32(cf[2 * i + 1] * H), bits_from_f32(cf[2 * i] * H), 0x07060302u);
        if (exact) {
            const double S = (double)e4m3_value(sbyte) * G.gd;
            uint32_t c[16];
            kv4_exact_codes(d, bad, sbyte, G, S, Sf, c);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                uint32_t h[2];
#pragma unroll
                for (int k = 0; k < 2; ++k) {
                    const uint32_t cc = c[2 * i + k];
                    uint32_t mag;
                    if (G.f32) {
                        const float v = 0.5f * (float)(cc & 7u) * (sbyte == 0u ? 0.0f : Sf);
                        mag = bf16_rne_from_float(v);
                    } else {
                        const double v = 0.5 * (double)(cc & 7u) * (sbyte == 0u ? 0.0 : S);
                        mag = bf16_rne_from_double(v);
                    }
                    h[k] = bad ? 0x7FC0u : (mag | ((cc & 8u) << 12));
                }
                o[i] = h[0] | (h[1] << 16);
            }
        }
        uint4 *dst = reinterpret_cast<uint4 *>(y + r * ldy + (blk - r * nb) * 16);
        dst[0] = make_uint4(o[0], o[1], o[2], o[3]);
        dst[1] = make_uint4(o[4], o[5], o[6], o[7]);
    }
    return sbyte;
}

// Largest |d| of a block as an FP32 pattern.  The IEEE maximum propagates NaN,
// so a block with a NaN or an infinity gives a pattern >= 0x7F800000.
__device__ __forceinline__ uint32_t kv4_block_max(const float (&d)[16]) {
    float m = 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) m = __builtin_elementwise_maximum(m, __builtin_fabsf(d[j]));
    return bits_from_f32(m);
}

template <int OUT, int SRC>
__global__ __launch_bounds__(kThreads) void kv4_quantize_kernel(
    const uint16_t *__restrict__ x, int64_t rows, int64_t cols, int64_t ldx, const float *__restrict__ shift,
    uint8_t *__restrict__ codes, uint8_t *__restrict__ scales, uint16_t *__restrict__ y, int64_t ldy,
    float *gptr, int computed, const uint32_t *__restrict__ partials, int nparts) {
    __shared__ float4 lds_shift[SRC == kShiftLdsSrc ? kShiftLds / 4 : 1];
    if (SRC == kShiftLdsSrc) kv4_stage_shift(shift, cols, lds_shift);
    float g;
    if (computed) {
        g = kv4_global_scale(kv4_fold_partials(partials, nparts));
        if (blockIdx.x == 0 && threadIdx.x == 0) *gptr = g;
    } else {
        g = *gptr;
    }
    const Kv4G G = kv4_make_g(g);

    const int64_t nb = cols / 16, total = rows * nb;
    const bool narrow = total < (int64_t(1) << 32);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // a wave step: kKvU adjacent segments of 64 blocks, one block per lane each
    for (int64_t base = ((int64_t)blockIdx.x * 4 + wave) * (64 * kKvU); base < total;
         base += (int64_t)gridDim.x * 4 * 64 * kKvU) {
        float d[kKvU][16];
#pragma unroll
        for (int u = 0; u < kKvU; ++u) {
            const int64_t blk = base + 64 * u + lane;
            kv4_load<SRC>(x, shift, lds_shift, blk < total ? blk : total - 1, nb, ldx, narrow, d[u]);
        }
#pragma unroll
        for (int u = 0; u < kKvU; ++u) {
            const int64_t blk = base + 64 * u + lane;
            if (blk < total) kv4_emit<OUT>(d[u], kv4_block_max(d[u]), blk, nb, narrow, G, codes, scales, y, ldy);
        }
    }
}

// Largest (kMax) or smallest v over the 64 lanes of a wave (all active), as a
// wave-uniform value.  DPP row shifts by 1, 2, 4, 8 leave each row's extreme
// in its lane 15; row_bcast:15 and row_bcast:31 carry it across rows to lane
// 63.  Lanes with no source keep their own value (the operation is idempotent).
template <int kCtrl, int kRows>
__device__ __forceinline__ uint32_t kv4_dpp(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, kCtrl, kRows, 0xF, false);
}

template <bool kMax>
__device__ __forceinline__ uint32_t kv4_wave_reduce(uint32_t v) {
    auto op = [](uint32_t a, uint32_t b) { return kMax ? (a > b ? a : b) : (a < b ? a : b); };
    v = op(v, kv4_dpp<0x111, 0xF>(v));   // row_shr:1
    v = op(v, kv4_dpp<0x112, 0xF>(v));   // row_shr:2
    v = op(v, kv4_dpp<0x114, 0xF>(v));   // row_shr:4
    v = op(v, kv4_dpp<0x118, 0xF>(v));   // row_shr:8
    v = op(v, kv4_dpp<0x142, 0xA>(v));   // row_bcast:15 into rows 1 and 3
    v = op(v, kv4_dpp<0x143, 0xC>(v));   // row_bcast:31 into rows 2 and 3
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// One pass over x for a computed g.  g needs the amax of all of d, known only
// once every block is read, so each segment of 64 consecutive blocks (the 64
// lanes of a wave in one step) is quantized under its own reference g_r: the
// global-scale rule applied to the segment's largest finite |d| (g_r <= g,
// both powers of two).  Dividing g by a power of two only moves the exponent
// of the smallest E4M3 scale s with amax <= 3.5 s g, so codes, s g and
// fake-quant values under g_r equal those under g for every block whose scale
// under g is still a normal E4M3 value; kv4_fixup_kernel lowers the scale
// exponents by log2(g / g_r) and re-quantizes from x only the blocks whose
// scale would leave the normal range.  The segment table records log2(g_r) +
// 127 (0 for a segment with no non-zero finite value) and the smallest scale
// exponent field among the segment's non-zero finite blocks; partials get the
// workgroup's largest finite |d|.
template <int OUT, int SRC>
__global__ __launch_bounds__(kThreads) void kv4_quantize_deferred_kernel(
    const uint16_t *__restrict__ x, int64_t rows, int64_t cols, int64_t ldx, const float *__restrict__ shift,
    uint8_t *__restrict__ codes, uint8_t *__restrict__ scales, uint16_t *__restrict__ y, int64_t ldy,
    uint32_t *__restrict__ partials, uint16_t *__restrict__ seg_table) {
    __shared__ float4 lds_shift[SRC == kShiftLdsSrc ? kShiftLds / 4 : 1];
    if (SRC == kShiftLdsSrc) kv4_stage_shift(shift, cols, lds_shift);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nb = cols / 16, total = rows * nb;
    const bool narrow = total < (int64_t(1) << 32);
    uint32_t mloc = 0u;
    // a wave step: kKvU adjacent segments (base / 64 + u, wave-uniform), as in kv4_quantize_kernel
    for (int64_t base = ((int64_t)blockIdx.x * 4 + wave) * (64 * kKvU); base < total;
         base += (int64_t)gridDim.x * 4 * 64 * kKvU) {
        float d[kKvU][16];
#pragma unroll
        for (int u = 0; u < kKvU; ++u) {
            const int64_t blk = base + 64 * u + lane;
            kv4_load<SRC>(x, shift, lds_shift, blk < total ? blk : total - 1, nb, ldx, narrow, d[u]);   // in range
        }
#pragma unroll
        for (int u = 0; u < kKvU; ++u) {
            if (base + 64 * u >= total) break;                     // wave-uniform: no such segment
            const int64_t blk = base + 64 * u + lane;
            const bool act = blk < total;
            const uint32_t am = act ? kv4_block_max(d[u]) : 0u;
            const bool bad = am >= 0x7F800000u;
            const uint32_t fm = bad ? kv4_finite_max(d[u]) : am;
            mloc = mloc > fm ? mloc : fm;
            const uint32_t segmax = kv4_wave_reduce<true>(fm);
            const Kv4G Gr = kv4_make_g(kv4_global_scale(segmax));
            uint32_t sbyte = 0u;
            if (act) sbyte = kv4_emit<OUT>(d[u], am, blk, nb, narrow, Gr, codes, scales, y, ldy);
            const bool live = act && am != 0u && !bad;
            const uint32_t emin = kv4_wave_reduce<false>(live ? sbyte >> 3 : 0xFFu);
            if (lane == 0)
                seg_table[base / 64 + u] =
                    segmax ? (uint16_t)((uint32_t)(Gr.kg + 127) | (emin << 8)) : (uint16_t)0;
        }
    }
    __shared__ uint32_t red[kThreads / 64];
    mloc = kv4_wave_max(mloc);
    if (lane == 0) red[wave] = mloc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = red[0];
        for (int i = 1; i < kThreads / 64; ++i) r = r > red[i] ? r : red[i];
        partials[blockIdx.x] = r;
    }
}

// Subtracts sub (= sh << 3, a lowering of the exponent field by sh) from each
// of the four scale bytes in v except 0x00 (zero block) and 0x7F (NaN block),
// whose meaning does not depend on g.  Every other byte has an exponent field
// > sh, so no byte borrows from its neighbour.
__device__ __forceinline__ uint32_t kv4_lower_bytes(uint32_t v, uint32_t sub) {
    const uint32_t z = ~(((v & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | v | 0x7F7F7F7Fu);   // 0x80 where a byte is 0x00
    const uint32_t t = v ^ 0x7F7F7F7Fu;
    const uint32_t n = ~(((t & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | t | 0x7F7F7F7Fu);   // 0x80 where a byte is 0x7F
    const uint32_t mask = 0x01010101u & ~((z | n) >> 7);
    return v - mask * sub;
}

// Second kernel of the one-pass quantizer: folds the partials into g,
// publishes it, and corrects every segment whose reference scale differs from
// g by 2^sh, one lane per segment: when the segment's smallest exponent field
// exceeds sh, every block keeps a normal scale and only its scale bytes are
// lowered (codes output; fake-quant values stand).  Otherwise the wave walks
// such segments, one lane per block, lowering the bytes that stay normal and
// re-quantizing the other blocks from x under g (fake-quant output, with no
// scale bytes to tell them apart: every block of the segment).  The shift is
// read from global memory (only re-quantized blocks need it).
template <int OUT>
__global__ __launch_bounds__(kThreads) void kv4_fixup_kernel(
    const uint16_t *__restrict__ x, int64_t rows, int64_t cols, int64_t ldx, const float *__restrict__ shift,
    uint8_t *__restrict__ codes, uint8_t *__restrict__ scales, uint16_t *__restrict__ y, int64_t ldy, float *gptr,
    const uint32_t *__restrict__ partials, int nparts, const uint16_t *__restrict__ seg_table) {
    const int lane = threadIdx.x & 63;
    const int64_t nb = cols / 16, total = rows * nb;
    const int64_t nseg = (total + 63) / 64;
    const bool narrow = total < (int64_t(1) << 32);
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    const int64_t first = (int64_t)blockIdx.x * kThreads + (threadIdx.x & ~63);
    // a lane's table entry and (codes output) its segment's 64 scale bytes
    auto fetch = [&](int64_t seg, uint32_t &e, uint4 (&v)[4]) {
        e = 0u;
        if (seg < nseg) {
            e = seg_table[seg];
            if (OUT == kCodes && total - seg * 64 >= 64) {
                const uint4 *p = reinterpret_cast<const uint4 *>(scales + seg * 64);
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = p[i];
            }
        }
    };
    uint32_t e;
    uint4 v[4] = {};
    fetch(first + lane, e, v);                          // its latency overlaps the fold
    const Kv4G G = kv4_make_g(kv4_global_scale(kv4_fold_partials(partials, nparts)));
    if (blockIdx.x == 0 && threadIdx.x == 0) *gptr = G.g;

    for (int64_t s0 = first; s0 < nseg; s0 += stride) {
        if (s0 != first) fetch(s0 + lane, e, v);
        const int64_t seg = s0 + lane;
        int sh = 0;
        bool redo = false;
        if (e != 0u) sh = G.kg - ((int)(e & 0xFFu) - 127);
        if (sh > 0) {
            redo = (int)(e >> 8) <= sh;
            if (OUT == kCodes && !redo) {
                const uint32_t sub = (uint32_t)sh << 3;
                const int64_t n = total - seg * 64;
                if (n >= 64) {
                    uint4 *p = reinterpret_cast<uint4 *>(scales + seg * 64);
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        p[i] = make_uint4(kv4_lower_bytes(v[i].x, sub), kv4_lower_bytes(v[i].y, sub),
                                          kv4_lower_bytes(v[i].z, sub), kv4_lower_bytes(v[i].w, sub));
                } else {
                    for (int64_t i = 0; i < n; ++i)
                        scales[seg * 64 + i] = (uint8_t)kv4_lower_bytes(scales[seg * 64 + i], sub);
                }
            }
        }
        uint64_t flags = __ballot(redo);
        while (flags) {
            const int l = __builtin_ctzll(flags);
            flags &= flags - 1;
            const int lsh = __shfl(sh, l, 64);
            const int64_t blk = (s0 + l) * 64 + lane;
            if (blk < total) {
                bool requant = true;
                if (OUT == kCodes) {
                    const uint32_t b = scales[blk];
                    if (b == 0u || b == 0x7Fu) {
                        requant = false;
                    } else if ((int)(b >> 3) > lsh) {
                        scales[blk] = (uint8_t)(b - ((uint32_t)lsh << 3));
                        requant = false;
                    }
                }
                if (requant) {
                    float d[16];
                    if (shift) kv4_load<kShiftGlobal>(x, shift, nullptr, blk, nb, ldx, narrow, d);
                    else kv4_load<kNoShift>(x, shift, nullptr, blk, nb, ldx, narrow, d);
                    kv4_emit<OUT>(d, kv4_block_max(d), blk, nb, narrow, G, codes, scales, y, ldy);
                }
            }
        }
    }
}

}  // namespace

hipError_t launch_kv4(QuantOut out, const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx, const float *shift,
                      uint8_t *codes, uint8_t *scales, uint16_t *y, int64_t ldy, float *gptr, bool computed,
                      uint32_t *partials, uint16_t *seg_table, hipStream_t stream) {
    const int64_t total = rows * (cols / 16);
    if (total == 0) return hipSuccess;
    int64_t grid = (total + kThreads - 1) / kThreads;             // absmax pass: one block per lane
    if (grid > kMaxKvGroups) grid = kMaxKvGroups;
    int64_t qgrid = (total + kThreads * kKvU - 1) / (kThreads * kKvU);   // quantize kernels: kKvU per lane
    if (qgrid > kMaxKvQuantGroups) qgrid = kMaxKvQuantGroups;
    const int64_t nseg = (total + 63) / 64;
    const bool deferred = computed && seg_table != nullptr && nseg <= kMaxSegments;
    auto run = [&](auto src_c) {
        constexpr int SRC = decltype(src_c)::value;
        if (deferred) {
            // one pass over x under per-segment reference scales, then the fix-up
            if (out == kCodes)
                hipLaunchKernelGGL((kv4_quantize_deferred_kernel<kCodes, SRC>), dim3((unsigned)qgrid), dim3(kThreads), 0,
                                   stream, x, rows, cols, ldx, shift, codes, scales, y, ldy, partials, seg_table);
            else
                hipLaunchKernelGGL((kv4_quantize_deferred_kernel<kFakeQuant, SRC>), dim3((unsigned)qgrid),
                                   dim3(kThreads), 0, stream, x, rows, cols, ldx, shift, codes, scales, y, ldy,
                                   partials, seg_table);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            int64_t fgrid = (nseg + kThreads - 1) / kThreads;
            if (fgrid > kMaxKvGroups) fgrid = kMaxKvGroups;
            if (out == kCodes)
                hipLaunchKernelGGL(kv4_fixup_kernel<kCodes>, dim3((unsigned)fgrid), dim3(kThreads), 0, stream, x, rows,
                                   cols, ldx, shift, codes, scales, y, ldy, gptr, partials, (int)qgrid, seg_table);
            else
                hipLaunchKernelGGL(kv4_fixup_kernel<kFakeQuant>, dim3((unsigned)fgrid), dim3(kThreads), 0, stream, x,
                                   rows, cols, ldx, shift, codes, scales, y, ldy, gptr, partials, (int)qgrid,
                                   seg_table);
            return hipGetLastError();
        }
        if (computed) {
            hipLaunchKernelGGL(kv4_absmax_kernel<SRC>, dim3((unsigned)grid), dim3(kThreads), 0, stream, x, rows, cols,
                               ldx, shift, partials);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        if (out == kCodes)
            hipLaunchKernelGGL((kv4_quantize_kernel<kCodes, SRC>), dim3((unsigned)qgrid), dim3(kThreads), 0, stream, x,
                               rows, cols, ldx, shift, codes, scales, y, ldy, gptr, (int)computed, partials,
                               (int)grid);
        else
            hipLaunchKernelGGL((kv4_quantize_kernel<kFakeQuant, SRC>), dim3((unsigned)qgrid), dim3(kThreads), 0,
                               stream, x, rows, cols, ldx, shift, codes, scales, y, ldy, gptr, (int)computed,
                               partials, (int)grid);
        return hipGetLastError();
    };
    if (!shift) return run(std::integral_constant<int, kNoShift>{});
    if (cols <= kShiftLds) return run(std::integral_constant<int, kShiftLdsSrc>{});
    return run(std::integral_constant<int, kShiftGlobal>{});
}

}  // namespace reqat
