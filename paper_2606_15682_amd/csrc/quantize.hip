// Block quantizer, fake-quant and tensor absmax kernels for gfx950.
//
// Quantize: one lane owns one scale block (16 bfloat16 = 32 B for NVFP4, 32 =
// 64 B for MXFP4), so the block absmax, the scale and the rounding thresholds
// are computed once per block with no cross-lane traffic; consecutive lanes
// own consecutive blocks of a row, so each wave-wide 16-byte load instruction
// covers whole 128-byte lines.  Codes leave as one 8-byte (NV) or 16-byte (MX)
// store per lane, scales as one byte per lane (contiguous across the wave).
//
// NVFP4 computed global scale: a first pass writes one partial absmax per
// workgroup into the workspace; every quantize workgroup folds the partials
// (<= 1024 words, L2-resident) before it starts, and workgroup 0 publishes g.
#include "fp4_device.h"
#include "internal.h"

namespace reqat {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        uint32_t o = __shfl_xor(v, off, 64);
        v = v > o ? v : o;
    }
    return v;
}

// One partial maximum of the finite bfloat16 magnitudes per workgroup.
__global__ __launch_bounds__(kThreads) void absmax_kernel(const uint16_t *__restrict__ x,
                                                          int64_t rows, int64_t cols, int64_t ldx,
                                                          uint32_t *__restrict__ partials) {
    const int64_t vpr = cols / 8;                       // 16-byte vectors per row
    const int64_t total = rows * vpr;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    uint32_t m = 0;
    for (int64_t v = (int64_t)blockIdx.x * kThreads + threadIdx.x; v < total; v += stride) {
        int64_t r = v / vpr, c = v - r * vpr;
        uint4 d = *reinterpret_cast<const uint4 *>(x + r * ldx + c * 8);
        uint32_t w[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            uint32_t lo = w[i] & 0x7FFFu, hi = (w[i] >> 16) & 0x7FFFu;
            lo = lo >= 0x7F80u ? 0u : lo;               // non-finite values are excluded
            hi = hi >= 0x7F80u ? 0u : hi;
            m = m > lo ? m : lo;
            m = m > hi ? m : hi;
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

// Grid values of the E2M1 magnitudes 0..7, for fake-quant outputs.
__device__ __forceinline__ float e2m1_mag_value(int m) {
    constexpr float v[8] = {0.0f, 0.5f, 1.0f, 1.5f, 2.0f, 3.0f, 4.0f, 6.0f};
    return v[m];
}

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
    const bool g_pow2 = (FMT == kMX) || ((bits_from_f32(g) & 0x807FFFFFu) == 0u &&
                                         (bits_from_f32(g) >> 23) != 0u);

    const int64_t nb = cols / B;
    const int64_t blk = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (blk >= rows * nb) return;
    const int64_t r = blk / nb, b = blk - r * nb;

    // ---- load the block and its absmax
    uint32_t w[B / 2];
    const uint4 *src = reinterpret_cast<const uint4 *>(x + r * ldx + b * B);
#pragma unroll
    for (int i = 0; i < NV4; ++i) {
        uint4 d = src[i];
        w[4 * i + 0] = d.x; w[4 * i + 1] = d.y; w[4 * i + 2] = d.z; w[4 * i + 3] = d.w;
    }
    uint32_t am = 0;
#pragma unroll
    for (int i = 0; i < B / 2; ++i) {
        uint32_t lo = bf16_mag_or_bad(w[i] & 0xFFFFu), hi = bf16_mag_or_bad(w[i] >> 16);
        am = am > lo ? am : lo;
        am = am > hi ? am : hi;
    }

    // ---- scale and thresholds
    uint32_t U[7];
    uint32_t sbyte;
    bool bad = am >= kBadBlock;
    bool fast = true;
    float Sf = 0.0f;
    double Sd = 0.0;
    if (bad) {
        sbyte = FMT == kMX ? 0xFFu : 0x7Fu;
#pragma unroll
        for (int i = 0; i < 7; ++i) U[i] = kNever;
    } else if (FMT == kMX) {
        sbyte = mx_scale_byte(am);
        int e = (int)sbyte - 127;
        fast = e >= -124 && e <= 125;
        if (fast) {
            Sf = f32_from_bits((uint32_t)(e + 127) << 23);
            thresholds_fast(Sf, U);
        } else {
            Sd = __builtin_ldexp(1.0, e);
            thresholds_exact(Sd, U);
        }
    } else {
        sbyte = nv_scale_byte(bf16_mag_value(am), g);
        if (sbyte == 0u) {                               // all-zero block: sign-only codes
#pragma unroll
            for (int i = 0; i < 7; ++i) U[i] = kNever;
            Sf = 0.0f;
        } else {
            float s = e4m3_value(sbyte);
            Sf = s * g;
            fast = fast_ok(Sf, g_pow2);
            if (fast) {
                thresholds_fast(Sf, U);
            } else {
                Sd = (double)s * (double)g;
                thresholds_exact(Sd, U);
            }
        }
    }

    if (OUT == kCodes) {
        uint32_t out[B / 8];
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
        uint8_t *dst = codes + r * (cols / 2) + b * (B / 2);
        if constexpr (B == 16) {
            *reinterpret_cast<uint2 *>(dst) = make_uint2(out[0], out[1]);
        } else {
            *reinterpret_cast<uint4 *>(dst) = make_uint4(out[0], out[1], out[2], out[3]);
        }
        scales[r * nb + b] = (uint8_t)sbyte;
    } else {
        // output patterns of the 8 grid magnitudes for this block
        uint32_t P[8];
        if (bad) {
#pragma unroll
            for (int m = 0; m < 8; ++m) P[m] = 0x7FC0u;
        } else if (fast) {
#pragma unroll
            for (int m = 0; m < 8; ++m) P[m] = bits_from_f32(e2m1_mag_value(m) * Sf) >> 16;
        } else {
#pragma unroll
            for (int m = 0; m < 8; ++m) P[m] = bf16_rne_from_double((double)e2m1_mag_value(m) * Sd);
        }
        uint32_t outw[B / 2];
#pragma unroll
        for (int i = 0; i < B / 2; ++i) {
            uint32_t res[2];
#pragma unroll
            for (int hlf = 0; hlf < 2; ++hlf) {
                uint32_t h = hlf ? (w[i] >> 16) : (w[i] & 0xFFFFu);
                uint32_t mag = h & 0x7FFFu;
                uint32_t v = P[0];
#pragma unroll
                for (int t = 0; t < 7; ++t) v = (mag >= U[t]) ? P[t + 1] : v;
                res[hlf] = bad ? 0x7FC0u : (v | (h & 0x8000u));
            }
            outw[i] = res[0] | (res[1] << 16);
        }
        uint4 *dst = reinterpret_cast<uint4 *>(y + r * ldy + b * B);
#pragma unroll
        for (int i = 0; i < NV4; ++i)
            dst[i] = make_uint4(outw[4 * i], outw[4 * i + 1], outw[4 * i + 2], outw[4 * i + 3]);
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
    int64_t want = (total + kThreads * 8 - 1) / (kThreads * 8);   // >= 8 vectors per lane
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
    const int64_t grid = (blocks + kThreads - 1) / kThreads;
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
