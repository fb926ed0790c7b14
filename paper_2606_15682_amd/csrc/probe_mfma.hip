// Rate probes for gfx950 (measurement context, not part of the product path;
// built into their own library, libreqat_probe.so): the matrix-core rate
// (reqat_probe_mfma) and the read-only HBM stream rate (reqat_probe_read).
//
// The products' rooflines are quoted against the nominal MFMA peaks, but the
// rate the chip sustains depends on the operand bits: under random-looking
// data the matrix cores draw more power and the chip lowers its clock.  This
// kernel issues only MFMAs, from registers, at one wave per SIMD (the
// products' occupancy): 256 workgroups of four waves, sixteen independent
// 32 x 32 accumulators per wave, operand words taken from a caller buffer
// (e.g. a workload's own packed codes), so its rate is the ceiling a product
// on that data could reach with no memory traffic at all.
//   kind 0: v_mfma_scale_f32_32x32x64_f8f6f4 on E2M1 x E2M1 (E8M0 scales 1.0)
//   kind 1: v_mfma_f32_32x32x16_f16 (operand words read as FP16 pairs)
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kAcc = 16;
constexpr int kWords = 1024;                    // operand words per operand (4 KB)

// ops[0 .. kWords) feed A, ops[kWords .. 2 kWords) feed B; lane l takes four
// consecutive words at 4 (l + 64 i) for tile i (wrapping), so lanes and tiles
// see different data.
template <int KIND>
__global__ __launch_bounds__(kThreads, 1) void probe_mfma_kernel(const uint32_t *__restrict__ ops,
                                                                 float *__restrict__ out, int iters) {
    const int lane = threadIdx.x & 63;
    v4u a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int o = (4 * (lane + 64 * i)) & (kWords - 1);
        a[i] = v4u{ops[o], ops[o + 1], ops[o + 2], ops[o + 3]};
        b[i] = v4u{ops[kWords + o], ops[kWords + o + 1], ops[kWords + o + 2], ops[kWords + o + 3]};
    }
    v16f acc[kAcc];
#pragma unroll
    for (int i = 0; i < kAcc; ++i) acc[i] = v16f{};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < kAcc; ++i) {
            const v4u x = a[i & 3], y = b[i >> 2];
            if constexpr (KIND == 0) {
                const v8i xa = v8i{(int)x[0], (int)x[1], (int)x[2], (int)x[3], 0, 0, 0, 0};
                const v8i yb = v8i{(int)y[0], (int)y[1], (int)y[2], (int)y[3], 0, 0, 0, 0};
                acc[i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(xa, yb, acc[i], 4, 4, 0, 0x7F7F7F7F, 0,
                                                                         0x7F7F7F7F);
            } else {
                acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(v8h, x),
                                                                __builtin_bit_cast(v8h, y), acc[i], 0, 0, 0);
            }
        }
    }
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kAcc; ++i)
#pragma unroll
        for (int k = 0; k < 16; ++k) s += acc[i][k];
    out[blockIdx.x * kThreads + threadIdx.x] = s;
}

// Read-only stream: one 16-byte load per thread per iteration of a
// grid-stride loop, folded by XOR so that no load is dead; each thread writes
// its fold.  (Four loads per iteration a grid-stride apart measured 19% slower
// on gfx950, four consecutive 1 KB wave pieces 4% slower.)
__global__ __launch_bounds__(kThreads) void probe_read_kernel(const uint4 *__restrict__ p, int64_t n16,
                                                              uint32_t *__restrict__ out) {
    uint32_t acc = 0u;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n16; i += (int64_t)gridDim.x * kThreads) {
        const uint4 a = p[i];
        acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc;
}

}  // namespace

extern "C" {

// Enqueues one read of `bytes` bytes (a multiple of 16; p 16-byte aligned)
// by `blocks` workgroups of 256 threads on `stream`; out: blocks * 256
// uint32 of device memory, whose XOR is the XOR of every 32-bit word read.
// Returns 0, or the HIP error code of the launch (1 for a bad argument).
int reqat_probe_read(const void *p, int64_t bytes, void *out, int blocks, void *stream) {
    if (!p || !out || bytes <= 0 || bytes % 16 || blocks <= 0 || (reinterpret_cast<uintptr_t>(p) & 15u)) return 1;
    hipLaunchKernelGGL(probe_read_kernel, dim3(blocks), dim3(kThreads), 0, reinterpret_cast<hipStream_t>(stream),
                       static_cast<const uint4 *>(p), bytes / 16, static_cast<uint32_t *>(out));
    return (int)hipGetLastError();
}


// Enqueues one probe launch of `blocks` workgroups (256 threads each) running
// `iters` rounds of 16 MFMAs per wave on `stream`.  ops: 8 KB of device
// operand words (A then B); out: blocks * 256 floats of device memory.
// FLOPs per launch: blocks * 4 * iters * 16 * (kind 0: 131072, kind 1: 32768).
// Returns 0, or the HIP error code of the launch (1 for a bad argument).
int reqat_probe_mfma(int kind, const void *ops, void *out, int blocks, int iters, void *stream) {
    if ((kind != 0 && kind != 1) || !ops || !out || blocks <= 0 || iters <= 0) return 1;
    const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    if (kind == 0)
        hipLaunchKernelGGL(probe_mfma_kernel<0>, dim3(blocks), dim3(kThreads), 0, st,
                           static_cast<const uint32_t *>(ops), static_cast<float *>(out), iters);
    else
        hipLaunchKernelGGL(probe_mfma_kernel<1>, dim3(blocks), dim3(kThreads), 0, st,
                           static_cast<const uint32_t *>(ops), static_cast<float *>(out), iters);
    return (int)hipGetLastError();
}

}  // extern "C"
