// Exact decisions for the block-rotated MXFP4 quantizer (gfx950, also host-callable).
//
// A rotated block is y = H_32 D x / sqrt(32) (the randomized Hadamard rotation
// ReQAT applies to MXFP4 activations, Sec. 4.3 "Additional implementation
// details" and App. C.2), taken as the exact real value.  The quantizer's fast
// path evaluates y in FP32 and keeps its decisions only when an error bound
// proves them; the blocks it cannot prove come here.
//
// With every bfloat16 input written m_j 2^(sh_j - 133) (m_j < 256 an integer,
// 0 <= sh_j <= 253), the scaled sum S_i = sqrt(32) y_i 2^133 is an integer, and
//     |y_i| <= 6 * 2^e       <=>  S_i^2 <= 1152 * 2^(2e + 266),
//     |y_i| >  (k/4) * 2^e   <=>  S_i^2 >  2 k^2 * 2^(2e + 266),
// where the E2M1 midpoints 0.25 .. 5 are k/4 for k = 1, 3, 5, 7, 10, 14, 20.
// Equality never holds (it would make sqrt(2) rational), so no tie rule is needed.
//   * Exponent spread (max sh - min sh over the nonzero inputs) <= 40: the sums
//     in units of 2^(min sh) are integers below 2^53, so an FP64 fast
//     Walsh-Hadamard transform computes them exactly, and each comparison is
//     the sign of one FP64 fused multiply-add, S^2 - C 2^P, rounded once (it
//     is never zero and stays far above the FP64 underflow range).  The
//     quantizer runs that path with one block spread over the lanes of a wave.
//   * Larger spreads (here): the sums as 320-bit integers and their squares as
//     640-bit integers, compared word by word, by one lane, with its words in
//     a caller-provided buffer (LDS on the GPU) so that the path adds no
//     registers to the quantizer.
#pragma once

#include <stdint.h>

#ifndef REQAT_HD
#define REQAT_HD __host__ __device__ __forceinline__
#endif

namespace reqat {
namespace rht {

// k of the E2M1 midpoints k/4: 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.
REQAT_HD uint32_t mid_k(int i) {
    return i == 0 ? 1u : i == 1 ? 3u : i == 2 ? 5u : i == 3 ? 7u : i == 4 ? 10u : i == 5 ? 14u : 20u;
}

// Input j of a block (bfloat16 pattern h, finite) as sign and m * 2^(sh - 133).
REQAT_HD void int_parts(uint32_t h, bool flip, bool &neg, uint32_t &m, int &sh) {
    const uint32_t ef = (h >> 7) & 0xFFu;
    neg = (((h >> 15) & 1u) != 0u) != flip;
    m = ef ? (0x80u | (h & 0x7Fu)) : (h & 0x7Fu);
    sh = ef ? (int)ef - 1 : 0;
}

// ------------------------------------------------------------------ wide-integer path
// Taken only for blocks whose inputs span more than 40 binades and whose FP32
// evaluation left a decision open; written with plain loops (its words may
// live in private memory) so that it adds no registers to the quantizer.

constexpr int kW = 10;          // words of a sum (two's complement, |S| < 2^266)
constexpr int kW2 = 20;         // words of a square or a bound

// a += sign * t * 2^(32 q), t < 2^40, q + 1 < kW (two's complement)
REQAT_HD void add_term(uint32_t *a, uint64_t t, int q, bool negative) {
    uint64_t x = t;
    if (!negative) {
        uint64_t c = 0;
#pragma unroll 1
        for (int l = q; l < kW; ++l) {
            c += (uint64_t)a[l] + (x & 0xFFFFFFFFu);
            a[l] = (uint32_t)c;
            c >>= 32;
            x >>= 32;
        }
    } else {
        uint64_t b = 0;
#pragma unroll 1
        for (int l = q; l < kW; ++l) {
            const uint64_t sub = (x & 0xFFFFFFFFu) + b;
            b = (uint64_t)a[l] < sub ? 1u : 0u;
            a[l] = (uint32_t)((uint64_t)a[l] - sub);
            x >>= 32;
        }
    }
}

// S_i of the block (two's complement words).
REQAT_HD void sum_i(const uint32_t *w, uint32_t signs, int i, uint32_t *a) {
#pragma unroll 1
    for (int l = 0; l < kW; ++l) a[l] = 0u;
#pragma unroll 1
    for (int j = 0; j < 32; ++j) {
        bool neg;
        uint32_t m;
        int sh;
        const uint32_t h = (j & 1) ? (w[j >> 1] >> 16) : (w[j >> 1] & 0xFFFFu);
        int_parts(h, ((signs >> j) & 1u) != 0u, neg, m, sh);
        const bool hneg = (__builtin_popcount((uint32_t)(i & j)) & 1) != 0;
        if (m) add_term(a, (uint64_t)m << (sh & 31), sh >> 5, neg != hneg);
    }
}

// |a| into `mag`; returns whether a < 0.
REQAT_HD bool magnitude(const uint32_t *a, uint32_t *mag) {
    const bool neg = (a[kW - 1] >> 31) != 0u;
    uint64_t c = 1;
#pragma unroll 1
    for (int l = 0; l < kW; ++l) {
        if (neg) {
            c += (uint64_t)(~a[l]);
            mag[l] = (uint32_t)c;
            c >>= 32;
        } else {
            mag[l] = a[l];
        }
    }
    return neg;
}

REQAT_HD void square(const uint32_t *a, uint32_t *sq) {
#pragma unroll 1
    for (int l = 0; l < kW2; ++l) sq[l] = 0u;
#pragma unroll 1
    for (int i = 0; i < kW; ++i) {
        uint64_t c = 0;
#pragma unroll 1
        for (int j = 0; j < kW; ++j) {
            c += (uint64_t)a[i] * a[j] + sq[i + j];
            sq[i + j] = (uint32_t)c;
            c >>= 32;
        }
        sq[i + kW] = (uint32_t)c;           // word i + kW is still zero here
    }
}

// sign(sq - C * 2^Q): -1, 0 or 1 (C < 2^32, 0 <= Q, Q / 32 + 1 < kW2)
REQAT_HD int compare_shifted(const uint32_t *sq, uint32_t C, int Q) {
    const uint64_t t = (uint64_t)C << (Q & 31);
    const int q = Q >> 5;
#pragma unroll 1
    for (int l = kW2 - 1; l >= 0; --l) {
        const uint32_t b = l == q ? (uint32_t)t : (l == q + 1 ? (uint32_t)(t >> 32) : 0u);
        if (sq[l] != b) return sq[l] > b ? 1 : -1;
    }
    return 0;
}

REQAT_HD int compare_words(const uint32_t *a, const uint32_t *b) {
#pragma unroll 1
    for (int l = kW2 - 1; l >= 0; --l)
        if (a[l] != b[l]) return a[l] > b[l] ? 1 : -1;
    return 0;
}

// Words the wide path keeps in its buffer.
constexpr int kWideWords = 16 + 2 * kW + 2 * kW2;

// E8M0 byte and packed codes of the rotated block of 32 finite bfloat16 values,
// exactly.  `buf` holds kWideWords words: the block's 16 packed words first
// (element 2k in the low half of word k), then the path's scratch.
REQAT_HD void block_wide(uint32_t signs, uint32_t &sbyte, uint32_t *cw, uint32_t *buf) {
    uint32_t *w = buf, *a = buf + 16, *mag = a + kW, *sq = mag + kW, *amax2 = sq + kW2;
#pragma unroll 1
    for (int l = 0; l < kW2; ++l) amax2[l] = 0u;
#pragma unroll 1
    for (int i = 0; i < 32; ++i) {
        sum_i(w, signs, i, a);
        magnitude(a, mag);
        square(mag, sq);
        if (compare_words(sq, amax2) > 0)
#pragma unroll 1
            for (int l = 0; l < kW2; ++l) amax2[l] = sq[l];
    }
#pragma unroll 1
    for (int q = 0; q < 4; ++q) cw[q] = 0u;
    int top = -1;
#pragma unroll 1
    for (int l = 0; l < kW2; ++l)
        if (amax2[l]) top = 32 * l + 31 - __builtin_clz(amax2[l]);
    if (top < 0) {
        sbyte = 0u;
        return;
    }
    // amax2 < 2^(top+1) <= 1152 * 2^Q once Q >= top - 9, and amax2 >= 2^top > 1152 * 2^Q
    // while Q < top - 10: start below the smallest e and step up
    int e = (top - 9 - 266) / 2 - 2;
    e = e < -127 ? -127 : (e > 127 ? 127 : e);
    while (e < 127 && compare_shifted(amax2, 1152u, 2 * e + 266) > 0) ++e;
    sbyte = (uint32_t)(e + 127);
    const int Q = 2 * e + 266;
#pragma unroll 1
    for (int i = 0; i < 32; ++i) {
        sum_i(w, signs, i, a);
        const bool neg = magnitude(a, mag);
        square(mag, sq);
        uint32_t m3 = 0u;
#pragma unroll 1
        for (int k = 0; k < 7; ++k) m3 += compare_shifted(sq, 2u * mid_k(k) * mid_k(k), Q) > 0 ? 1u : 0u;
        const uint32_t c = m3 | (neg ? 8u : 0u);      // neg implies S_i != 0
        cw[i >> 3] |= c << (4 * (i & 7));
    }
}

}  // namespace rht
}  // namespace reqat
