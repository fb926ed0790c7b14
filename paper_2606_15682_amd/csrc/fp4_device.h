// Device-side codecs for the microscaled FP4 formats (MXFP4 / NVFP4 of
// ReQAT App. A, Tab. mx_configs) on gfx950.
//
// Element rounding is decided in the integer domain: for a block with scale
// S = s * g, the code magnitude of an element is the number of rounding
// thresholds its bfloat16 magnitude pattern reaches.  Threshold i sits at the
// midpoint mid_i * S between grid values i and i+1 (mid = .25 .75 1.25 1.75
// 2.5 3.5 5); it is expressed as the smallest bfloat16 magnitude pattern that
// must round up: strictly above the midpoint when the tie goes down (i even)
// and at-or-above it when the tie goes up (i odd), which is round to nearest
// with ties to the even code.  Non-negative IEEE patterns order like their
// values, so the count of thresholds reached is the rounded magnitude.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace reqat {

// Magnitude pattern that no finite bfloat16 reaches (finite magnitudes <= 0x7F7F).
constexpr uint32_t kNever = 0xFFFFu;
// A block containing NaN/Inf is marked by this "absmax" pattern.
constexpr uint32_t kBadBlock = 0x10000u;

__device__ __forceinline__ float f32_from_bits(uint32_t u) { return __uint_as_float(u); }
__device__ __forceinline__ uint32_t bits_from_f32(float f) { return __float_as_uint(f); }

// Finite-magnitude pattern of a bfloat16, or kBadBlock when NaN/Inf.
__device__ __forceinline__ uint32_t bf16_mag_or_bad(uint32_t h) {
    uint32_t m = h & 0x7FFFu;
    return m >= 0x7F80u ? kBadBlock : m;
}

// Value of a non-negative finite bfloat16 magnitude pattern, exact in FP32.
__device__ __forceinline__ float bf16_mag_value(uint32_t m) { return f32_from_bits(m << 16); }

// E4M3 (OCP E4M3FN) byte -> value, exact; NaN for 0x7F/0xFF.
__device__ __forceinline__ float e4m3_value(uint32_t b) {
    uint32_t e = (b >> 3) & 15u, m = b & 7u;
    float v;
    if (e == 15u && m == 7u) return __builtin_nanf("");
    if (e == 0u) v = (float)m * 0x1p-9f;
    else v = f32_from_bits(((e + 120u) << 23) | (m << 20));   // 2^(e-7) * (1 + m/8)
    return (b & 0x80u) ? -v : v;
}

// --------------------------------------------------------------------- scales

// MXFP4 block scale byte for a finite block-absmax pattern `am` (bfloat16 magnitude):
// smallest e in [-127, 127] with amax <= 6 * 2^e.  With amax = 1.f * 2^E this is
// E - 2 when 1.f <= 1.5 (fraction bits <= 0x40 of 7), else E - 1.
__device__ __forceinline__ uint32_t mx_scale_byte(uint32_t am) {
    if (am == 0u) return 0u;
    int E;
    uint32_t frac;
    uint32_t ef = am >> 7;
    if (ef != 0u) {
        E = (int)ef - 127;
        frac = am & 0x7Fu;
    } else {                                   // bfloat16 subnormal: normalize
        uint32_t man = am & 0x7Fu;
        int p = 31 - __builtin_clz(man);        // position of the leading one (0..6)
        E = p - 133;
        frac = (man << (7 - p)) & 0x7Fu;
    }
    int e = (frac <= 0x40u) ? E - 2 : E - 1;
    e = e < -127 ? -127 : (e > 127 ? 127 : e);
    return (uint32_t)(e + 127);
}

// NVFP4 computed global scale from the finite tensor-absmax pattern `am`:
// g = 2^k, k the smallest integer >= -126 with amax <= 2688 * 2^k
// (2688 = 6 * 448 = 1.3125 * 2^11, and 1.3125 has fraction bits 0x28 of 7).
__device__ __forceinline__ float nv_global_scale(uint32_t am) {
    if (am == 0u) return 1.0f;
    int E;
    uint32_t frac;
    uint32_t ef = am >> 7;
    if (ef != 0u) {
        E = (int)ef - 127;
        frac = am & 0x7Fu;
    } else {
        uint32_t man = am & 0x7Fu;
        int p = 31 - __builtin_clz(man);
        E = p - 133;
        frac = (man << (7 - p)) & 0x7Fu;
    }
    int k = (frac <= 0x28u) ? E - 11 : E - 10;
    if (k < -126) k = -126;
    return f32_from_bits((uint32_t)(k + 127) << 23);
}

// Byte of the first positive finite E4M3 value >= q (q > 0), 0x7E when q > 448.
__device__ __forceinline__ uint32_t e4m3_ceil_byte(double q) {
    if (q > 448.0) return 0x7Eu;
    if (q <= 0x1p-9) return 0x01u;
    int E = (int)((__double_as_longlong(q) >> 52) & 0x7FF) - 1023;   // q is normal here
    if (E < -6) {                              // subnormal range: multiples of 2^-9
        double n = __builtin_ceil(q * 0x1p9);  // 1..8; 8 is 2^-6, byte 0x08
        return (uint32_t)n;
    }
    double f = q * __builtin_ldexp(1.0, -E);    // [1, 2)
    uint32_t m = (uint32_t)__builtin_ceil((f - 1.0) * 8.0);
    if (m == 8u) { m = 0u; E += 1; }
    uint32_t b = ((uint32_t)(E + 7) << 3) | m;
    return b > 0x7Eu ? 0x7Eu : b;
}

// NVFP4 block scale byte: smallest positive finite E4M3 s with amax <= 6*s*g,
// 0x00 for a zero block, 0x7E (saturate) when even 448 is too small.  The
// quotient is approximate; the two exact comparisons (6*s*g is exact in FP64)
// move it to the right value.
__device__ __forceinline__ uint32_t nv_scale_byte(float amax, float g) {
    if (amax == 0.0f) return 0u;
    double a = (double)amax, gg = (double)g;
    uint32_t b = e4m3_ceil_byte(a / (6.0 * gg));
    if (b < 0x7Eu && !(a <= 6.0 * (double)e4m3_value(b) * gg)) b += 1u;
    else if (b > 1u && a <= 6.0 * (double)e4m3_value(b - 1u) * gg) b -= 1u;
    return b;
}

// --------------------------------------------------------------------- thresholds

// Truncation of a positive double to a bfloat16 magnitude pattern, and whether
// it was exact.  Overflow gives 0x7F80 (above every finite pattern).
__device__ __forceinline__ uint32_t bf16_trunc_pattern(double t, bool &exact) {
    uint64_t u = (uint64_t)__double_as_longlong(t);
    int E = (int)((u >> 52) & 0x7FF) - 1023;
    uint64_t frac = u & ((1ull << 52) - 1);
    if (t == 0.0) { exact = true; return 0u; }
    if (E >= 128) { exact = true; return 0x7F80u; }
    if (E >= -126) {
        exact = (frac & ((1ull << 45) - 1)) == 0;
        return ((uint32_t)(E + 127) << 7) | (uint32_t)(frac >> 45);
    }
    // bfloat16 subnormal: value / 2^-133, truncated
    uint64_t sig = frac | (1ull << 52);
    int sh = -E - 81;                          // 52 - (E + 133)
    if (sh >= 64) { exact = false; return 0u; }
    exact = (sig & ((1ull << sh) - 1)) == 0;
    return (uint32_t)(sig >> sh);
}

// Rounding thresholds (see the header comment) for scale S = s * g.
// General path: FP64 products mid_i * s * g are exact (<= 31 significant bits).
__device__ __forceinline__ void thresholds_exact(double S, uint32_t U[7]) {
    const double mid[7] = {0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0};
#pragma unroll
    for (int i = 0; i < 7; ++i) {
        bool ex;
        uint32_t p = bf16_trunc_pattern(mid[i] * S, ex);
        // i even (tie rounds down): first pattern strictly above the midpoint = p + 1;
        // i odd (tie rounds up): first pattern at or above it = p if exact, else p + 1.
        U[i] = (i & 1) ? (ex ? p : p + 1u) : p + 1u;
    }
}

// Fast path: S is a float with at most 4 significant bits, 2^-124 <= S <= 2^125.
// Then mid_i * S (<= 7 bits) is an exact normal FP32 and an exact bfloat16.
__device__ __forceinline__ void thresholds_fast(float S, uint32_t U[7]) {
    const float mid[7] = {0.25f, 0.75f, 1.25f, 1.75f, 2.5f, 3.5f, 5.0f};
#pragma unroll
    for (int i = 0; i < 7; ++i) {
        uint32_t p = bits_from_f32(mid[i] * S) >> 16;
        U[i] = (i & 1) ? p : p + 1u;
    }
}

// True when the fast path is exact for this S (a float holding s * g exactly).
__device__ __forceinline__ bool fast_ok(float S, bool g_pow2) {
    return g_pow2 && S >= 0x1p-124f && S <= 0x1p125f;
}

// Count of thresholds reached by the magnitude pattern m: the E2M1 magnitude code.
__device__ __forceinline__ uint32_t e2m1_code_mag(uint32_t m, const uint32_t U[7]) {
    uint32_t c = 0;
#pragma unroll
    for (int i = 0; i < 7; ++i) c += (m >= U[i]) ? 1u : 0u;
    return c;
}

// Value of a bfloat16 magnitude pattern as a double; 0x7F80 maps to 2^128.
__device__ __forceinline__ double bf16_pattern_value(uint32_t p) {
    uint32_t ef = p >> 7;
    return ef ? __builtin_ldexp((double)(128u + (p & 0x7Fu)), (int)ef - 134)
              : (double)p * 0x1p-133;
}

// bfloat16 (round to nearest even) of an exact double; NaN -> 0x7FC0.
__device__ __forceinline__ uint32_t bf16_rne_from_double(double v) {
    if (v != v) return 0x7FC0u;
    uint32_t sign = (__double_as_longlong(v) < 0) ? 0x8000u : 0u;
    double a = __builtin_fabs(v);
    bool ex;
    uint32_t p = bf16_trunc_pattern(a, ex);
    if (p >= 0x7F80u) return sign | 0x7F80u;
    if (!ex) {
        // nearer of p and p+1; the midpoint is exact in FP64
        double midp = 0.5 * (bf16_pattern_value(p) + bf16_pattern_value(p + 1u));
        if (a > midp || (a == midp && (p & 1u))) p += 1u;
    }
    return sign | p;   // p == 0x7F80 is the overflow to infinity
}

// Round-to-nearest-even float -> bfloat16 bits (for GEMM outputs).
__device__ __forceinline__ uint32_t bf16_rne_from_float(float f) {
    uint32_t u = bits_from_f32(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

}  // namespace reqat
