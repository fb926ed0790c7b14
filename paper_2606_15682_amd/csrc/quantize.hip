// Block quantizer, fake-quant and tensor absmax kernels for gfx950.
//
// Quantize: a lane owns one scale block at a time (16 bfloat16 = 32 B for
// NVFP4, 32 = 64 B for MXFP4) and walks the blocks in a grid-stride loop, so
// the block absmax, the scale and the rounding are computed once per block
// with no cross-lane traffic, and per-thread set-up (global scale) is paid
// once.  Consecutive lanes own consecutive blocks, so every wave-wide 16-byte
// load covers whole 128-byte lines; codes leave as one 8-byte (NVFP4) or
// 16-byte (MXFP4) store per lane and scales as one byte per lane.
//
// Element rounding (round to nearest, ties to the even code, of |x| / (s g),
// saturating at 6) has two exact implementations:
//   * fast path: v_cvt_scalef32_pk_fp4_{bf16,f32}, which on gfx950 rounds
//     x / 2^e exactly that way for every finite bfloat16 x and every power of
//     two 2^-126..2^127 (the instruction reads only the exponent of its FP32
//     scale operand).  MXFP4 scales are powers of two and feed it directly.
//     For NVFP4 with a power-of-two g, s g = m * 2^e with m = 1.mmm (4 bits):
//     x is first multiplied by 1/m in FP32 and the product snapped to 16
//     significant bits.  If x / (m 2^e) is exactly a rounding midpoint
//     (<= 3 significant bits), the snapped value is that midpoint exactly
//     (FP32 error 2^-22 << 2^-16); otherwise x (8 significant bits) and the
//     midpoint times m 2^e (<= 7 bits) differ by at least 2^-8 relative, far
//     more than the 2^-16 snap, so the side of every midpoint is kept.  The
//     path is taken only when s g is in [2^-123, 2^125], so subnormal inputs
//     (which round to code 0 either way) cannot disturb it.
//   * general path (NaN/Inf blocks, all-zero NVFP4 blocks, a non-power-of-two
//     global scale, extreme exponents): integer thresholds on the bfloat16
//     magnitude pattern (see fp4_device.h).
// Fake-quant decodes the codes again with v_cvt_scalef32_pk_{bf16,f32}_fp4
// (code * 2^e, exact) and, for NVFP4, multiplies by m (exact, <= 6 bits).
//
// NVFP4 computed global scale: a first pass writes one partial absmax per
// workgroup into the workspace; each quantize workgroup folds the partials
// (<= 1024 words, L2-resident) before its block loop, and workgroup 0 publishes g.
#include "fp4_device.h"
#include "internal.h"

namespace reqat {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxGroups = 4096;      // grid cap of the quantize block loop

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

// One partial maximum of the finite bfloat16 magnitudes per workgroup.  The
// loop takes the plain packed maximum of all magnitudes (two VALU per dword);
// only a lane whose maximum reached the non-finite patterns (>= 0x7F80)
// walks its elements again with the finite filter.
__global__ __launch_bounds__(kThreads) void absmax_kernel(const uint16_t *__restrict__ x,
                                                          int64_t rows, int64_t cols, int64_t ldx,
                                                          uint32_t *__restrict__ partials) {
    uint32_t m = 0;
    if (ldx == cols) {
        const int64_t total = rows * cols / 8;          // 16-byte vectors
        const uint4 *v = reinterpret_cast<const uint4 *>(x);
        const int64_t stride = (int64_t)gridDim.x * kThreads;
        const int64_t i0 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
        us2 m2 = us2{0, 0};
        int64_t i = i0;
        for (; i + 3 * stride < total; i += 4 * stride) {
            uint4 d[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) d[u] = v[i + u * stride];
#pragma unroll
            for (int u = 0; u < 4; ++u) m2 = mag_max8(d[u], m2);
        }
        for (; i < total; i += stride) m2 = mag_max8(v[i], m2);
        m = m2[0] > m2[1] ? m2[0] : m2[1];
        if (m >= 0x7F80u) {                             // rare: a NaN or Inf among this lane's elements
            m = 0;
            for (int64_t j = i0; j < total; j += stride) m = finite_max8(v[j], m);
        }
    } else {
        const int64_t vpr = cols / 8;
        for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
            const uint4 *v = reinterpret_cast<const uint4 *>(x + r * ldx);
            for (int64_t c = threadIdx.x; c < vpr; c += kThreads) m = finite_max8(v[c], m);
        }
    }
    __shared__ uint32_t red[kThreads / 64];
    m = wave_max_u32(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = red[0];
        for (int i = 1; i < kThreads / 64; ++i) r = r > red[i] ? r : red[i];
        partials[blockIdx.x] = r;
    }
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

// Fake-quant of one block by thresholds; P[m] = bfloat16 pattern of grid value m.
template <int B>
__device__ __forceinline__ void fq_general(const uint32_t (&w)[B / 2], const uint32_t (&U)[7],
                                           const uint32_t (&P)[8], bool bad,
                                           uint32_t (&outw)[B / 2]) {
#pragma unroll
    for (int i = 0; i < B / 2; ++i) {
        uint32_t res[2];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            uint32_t h = hf ? (w[i] >> 16) : (w[i] & 0xFFFFu);
            uint32_t mag = h & 0x7FFFu;
            uint32_t v = P[0];
#pragma unroll
            for (int t = 0; t < 7; ++t) v = (mag >= U[t]) ? P[t + 1] : v;
            res[hf] = bad ? 0x7FC0u : (v | (h & 0x8000u));
        }
        outw[i] = res[0] | (res[1] << 16);
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

// ---------------------------------------------------------------- kernel

template <int FMT, int OUT>
__global__ __launch_bounds__(kThreads) void quantize_kernel(
    const uint16_t *__restrict__ x, int64_t rows, int64_t cols, int64_t ldx,
    uint8_t *__restrict__ codes, uint8_t *__restrict__ scales, uint16_t *__restrict__ y,
    int64_t ldy, float *gptr, int gsrc, const uint32_t *__restrict__ partials, int nparts) {
    constexpr int B = FMT == kMX ? 32 : 16;
    constexpr int NV4 = B / 8;                          // 16-byte vectors per block

    // ---- global scale (NVFP4)
    float g = 1.0f;
    if (FMT == kNV) {
        if (gsrc == kGComputed) {
            __shared__ float g_sh;
            if (threadIdx.x < 64) {
                uint32_t m = 0;
                for (int i = threadIdx.x; i < nparts; i += 64) {
                    uint32_t p = partials[i];
                    m = m > p ? m : p;
                }
                m = wave_max_u32(m);
                if (threadIdx.x == 0) g_sh = nv_global_scale(m);
            }
            __syncthreads();
            g = g_sh;
            if (blockIdx.x == 0 && threadIdx.x == 0) *gptr = g;
        } else {
            g = *gptr;
        }
    }
    const uint32_t gb = bits_from_f32(g);
    const bool g_pow2 = (gb & 0x807FFFFFu) == 0u && (gb >> 23) != 0u;
    const int kg = (int)(gb >> 23) - 127;               // g = 2^kg when g_pow2

    const int64_t nb = cols / B;
    const int64_t total = rows * nb;
    const bool contiguous = ldx == cols;
    const bool narrow = total < (int64_t(1) << 32);
    const int64_t stride = (int64_t)gridDim.x * kThreads;

    // Blocks are walked from the end of the tensor: the absmax pass that
    // precedes an NVFP4 call with a computed g walks it from the start, so the
    // tail it read last is still in the Infinity Cache.
    for (int64_t it = (int64_t)blockIdx.x * kThreads + threadIdx.x; it < total; it += stride) {
        const int64_t blk = total - 1 - it;
        int64_t xoff, yoff;
        if (contiguous) {
            xoff = blk * B;
        } else {
            int64_t r = narrow ? (int64_t)((uint32_t)blk / (uint32_t)nb) : blk / nb;
            xoff = r * ldx + (blk - r * nb) * B;
        }
        if (OUT == kFakeQuant) {
            if (ldy == cols) {
                yoff = blk * B;
            } else {
                int64_t r = narrow ? (int64_t)((uint32_t)blk / (uint32_t)nb) : blk / nb;
                yoff = r * ldy + (blk - r * nb) * B;
            }
        }

        // ---- load the block and its absmax (packed 16-bit max of magnitudes)
        uint32_t w[B / 2];
        const uint4 *src = reinterpret_cast<const uint4 *>(x + xoff);
#pragma unroll
        for (int i = 0; i < NV4; ++i) {
            uint4 d = src[i];
            w[4 * i + 0] = d.x; w[4 * i + 1] = d.y; w[4 * i + 2] = d.z; w[4 * i + 3] = d.w;
        }
        us2 mx2 = __builtin_bit_cast(us2, w[0] & 0x7FFF7FFFu);
#pragma unroll
        for (int i = 1; i < B / 2; ++i)
            mx2 = __builtin_elementwise_max(mx2, __builtin_bit_cast(us2, w[i] & 0x7FFF7FFFu));
        const uint32_t am = mx2[0] > mx2[1] ? mx2[0] : mx2[1];
        const bool bad = am >= 0x7F80u;                  // NaN or Inf somewhere in the block

        // ---- scale, path choice
        uint32_t sbyte;
        bool fast;
        float p2 = 1.0f, mant = 1.0f;
        double Sd = 0.0;
        if (FMT == kMX) {
            sbyte = bad ? 0xFFu : mx_scale_byte(am);
            fast = !bad && sbyte >= (OUT == kCodes ? 1u : 3u);
            p2 = f32_from_bits(sbyte << 23);
            Sd = __builtin_ldexp(1.0, (int)sbyte - 127);
        } else {
            // g = 2^kg and a normal bfloat16 amax = A * 2^(Ef - 134) (A = 128..255):
            // the smallest 4-significant-bit value >= amax / 6 is
            // Q(A) * 2^(Ef - 134), Q(A) = 2*ceil(A/12) (A <= 180) or 4*ceil(A/24),
            // = (1 + f/8) * 2^j; when amax / (6g) rounded that way is a normal E4M3
            // value it is the scale (dividing by g only moves the exponent), and
            // s * g = Q(A) * 2^(Ef - 134) exactly.
            fast = false;
            const uint32_t Ef = am >> 7;
            if (!bad && g_pow2 && Ef != 0u) {
                const uint32_t A = 128u + (am & 0x7Fu);
                const uint32_t j = A <= 180u ? 4u : 5u;
                const uint32_t f = (A <= 180u ? (A + 11u) / 12u : (A + 23u) / 24u) - 8u;
                const int ef = (int)(j + Ef) - 127 - kg;
                const int eS = (int)(j + Ef) - 134;
                if (ef >= 1 && (ef < 15 || (ef == 15 && f < 7u)) && eS >= -123 && eS <= 125) {
                    sbyte = ((uint32_t)ef << 3) | f;
                    p2 = f32_from_bits((uint32_t)(eS + 127) << 23);
                    mant = f32_from_bits(0x3F800000u | (f << 20));
                    fast = true;
                }
            }
            if (!fast) {
                sbyte = bad ? 0x7Fu : nv_scale_byte(bf16_mag_value(am), g);
                const float s = e4m3_value(sbyte);
                const float S = s * g;
                fast = !bad && sbyte != 0u && g_pow2 && S >= 0x1p-123f && S <= 0x1p125f;
                p2 = f32_from_bits(bits_from_f32(S) & 0x7F800000u);
                mant = f32_from_bits((bits_from_f32(S) & 0x007FFFFFu) | 0x3F800000u);
                Sd = (double)s * (double)g;
            }
        }

        if (OUT == kCodes) {
            uint32_t out[B / 8];
            if (fast) {
                if (FMT == kMX) codes_fast_mx<B>(w, p2, out);
                else codes_fast_nv<B>(w, p2, __builtin_amdgcn_rcpf(mant), out);
            } else {
                uint32_t U[7], P[8];
                general_plan<false>(Sd, bad || (FMT == kNV && sbyte == 0u), U, P);
                codes_general<B>(w, U, bad, out);
            }
            uint8_t *dst = codes + blk * (B / 2);
            if constexpr (B == 16) *reinterpret_cast<uint2 *>(dst) = make_uint2(out[0], out[1]);
            else *reinterpret_cast<uint4 *>(dst) = make_uint4(out[0], out[1], out[2], out[3]);
            scales[blk] = (uint8_t)sbyte;
        } else {
            uint32_t outw[B / 2];
            if (fast) {
                uint32_t cw[B / 8];
                if (FMT == kMX) codes_fast_mx<B>(w, p2, cw);
                else codes_fast_nv<B>(w, p2, __builtin_amdgcn_rcpf(mant), cw);
#pragma unroll
                for (int q = 0; q < B / 8; ++q) {
                    if (FMT == kMX) fq_fast_mx(cw[q], p2, &outw[4 * q]);
                    else fq_fast_nv(cw[q], p2, mant, &outw[4 * q]);
                }
            } else {
                uint32_t U[7], P[8];
                general_plan<true>(Sd, bad || (FMT == kNV && sbyte == 0u), U, P);
                fq_general<B>(w, U, P, bad, outw);
            }
            uint4 *dst = reinterpret_cast<uint4 *>(y + yoff);
#pragma unroll
            for (int i = 0; i < NV4; ++i)
                dst[i] = make_uint4(outw[4 * i], outw[4 * i + 1], outw[4 * i + 2], outw[4 * i + 3]);
        }
    }
}

// Writes g = 1 (the global scale of a tensor with no elements).
__global__ void unit_scale_kernel(float *gptr) { *gptr = 1.0f; }

}  // namespace

hipError_t launch_unit_scale(float *gptr, hipStream_t stream) {
    hipLaunchKernelGGL(unit_scale_kernel, dim3(1), dim3(1), 0, stream, gptr);
    return hipGetLastError();
}

hipError_t launch_absmax(const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                         uint32_t *partials, int *nparts_out, hipStream_t stream) {
    const int64_t total = rows * (cols / 8);
    int64_t want = (total + kThreads * 16 - 1) / (kThreads * 16);   // >= 16 vectors per lane
    int grid = (int)(want < 1 ? 1 : (want > kMaxPartials ? kMaxPartials : want));
    hipLaunchKernelGGL(absmax_kernel, dim3(grid), dim3(kThreads), 0, stream, x, rows, cols, ldx,
                       partials);
    *nparts_out = grid;
    return hipGetLastError();
}

hipError_t launch_quantize(Fmt fmt, QuantOut out, const uint16_t *x, int64_t rows, int64_t cols,
                           int64_t ldx, uint8_t *codes, uint8_t *scales, uint16_t *y, int64_t ldy,
                           float *gptr, GSrc gsrc, const uint32_t *partials, int nparts,
                           hipStream_t stream) {
    const int B = fmt == kMX ? 32 : 16;
    const int64_t blocks = rows * (cols / B);
    if (blocks == 0) return hipSuccess;
    int64_t grid = (blocks + kThreads - 1) / kThreads;
    if (grid > kMaxGroups) grid = kMaxGroups;
    dim3 g((unsigned)grid), t(kThreads);
    if (fmt == kMX) {
        if (out == kCodes)
            hipLaunchKernelGGL((quantize_kernel<kMX, kCodes>), g, t, 0, stream, x, rows, cols, ldx,
                               codes, scales, y, ldy, gptr, (int)gsrc, partials, nparts);
        else
            hipLaunchKernelGGL((quantize_kernel<kMX, kFakeQuant>), g, t, 0, stream, x, rows, cols,
                               ldx, codes, scales, y, ldy, gptr, (int)gsrc, partials, nparts);
    } else {
        if (out == kCodes)
            hipLaunchKernelGGL((quantize_kernel<kNV, kCodes>), g, t, 0, stream, x, rows, cols, ldx,
                               codes, scales, y, ldy, gptr, (int)gsrc, partials, nparts);
        else
            hipLaunchKernelGGL((quantize_kernel<kNV, kFakeQuant>), g, t, 0, stream, x, rows, cols,
                               ldx, codes, scales, y, ldy, gptr, (int)gsrc, partials, nparts);
    }
    return hipGetLastError();
}

}  // namespace reqat
