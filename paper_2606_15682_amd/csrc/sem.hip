// SEM loss for gfx950 (selective entropy minimization, Sec. 4.2):
//   per token t (a row of bfloat16 logits over the vocabulary, p = softmax):
//     H_t = -sum_j p_j log p_j,  NLL_t = -log p_{y_t},  lse_t = log sum_j exp(z_j)
//   over the minibatch: H_min = min_t H_t, tau = 75th percentile of H (linear
//   interpolation between order statistics at 0.75 (T - 1)),
//     w_t = max(0, 1 - (H_t - H_min) / (tau - H_min + eps)),
//     L = (1/T) sum_t NLL_t + lambda (1/T) sum_t w_t H_t.
//   Backward (the weights held fixed):
//     dL/dz_tj = (scale / T) [(p_j - [j == y_t]) - lambda w_t p_j (log p_j + H_t)].
//
// sem_rows_kernel: one 256-thread workgroup per row, one pass over the row with
// a running maximum m and, in base-2 units (mb = m log2 e, t = z log2 e - mb
// in one fused multiply-add, 2^t by v_exp_f32), S = sum 2^t and
// A = sum 2^t t per thread (rescaled when m grows), merged in a fixed tree
// order; then H = ln 2 (log2 S - A / S), lse = ln 2 (mb + log2 S),
// NLL = lse - z_y.  The logits are read once.
// sem_batch_kernel: one workgroup; H_min by reduction, the two order
// statistics by radix selection on the FP32 patterns (exact, deterministic;
// up to 8192 tokens the keys stay in registers and the second statistic
// follows from the first in one counting pass), the weights and the three
// loss sums (FP64, fixed order).
// sem_backward_kernel: one workgroup per row, logits read once more, gradient
// written as bfloat16 (round to nearest even) or FP32.
#include "fp4_device.h"
#include "internal.h"

namespace reqat {

namespace {

constexpr int kThreads = 256;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float exp_fast(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }

// Running softmax state of a slice of a row, in base-2 units: mb = RN(m log2 e)
// for the largest logit m seen so far, S = sum 2^t and A = sum 2^t t over the
// slice with t = RN(z log2 e - mb) (one fused multiply-add per logit), so that
// 2^t = exp(z - mb / log2 e).  Then ln sum exp(z) = ln 2 (mb + log2 S) and the
// entropy H = ln 2 (log2 S - A / S), whatever mb is.
struct Online {
    float m, mb, S, A;
};

// Merge two partial states.
__device__ __forceinline__ Online merge(Online a, Online b) {
    if (b.m > a.m) { Online t = a; a = b; b = t; }
    if (b.S == 0.0f) return a;                     // b empty (m = -inf)
    const float d = b.mb - a.mb;                   // <= 0
    const float f = __builtin_amdgcn_exp2f(d);
    a.A = a.A + f * (b.A + d * b.S);
    a.S = a.S + f * b.S;
    return a;
}

// Adds eight finite logits (the header requires finite logits).
__device__ __forceinline__ void add8(Online &o, const float (&z)[8]) {
    const float mx = __builtin_fmaxf(__builtin_fmaxf(__builtin_fmaxf(z[0], z[1]), __builtin_fmaxf(z[2], z[3])),
                                     __builtin_fmaxf(__builtin_fmaxf(z[4], z[5]), __builtin_fmaxf(z[6], z[7])));
    if (mx > o.m) {
        const float mxb = mx * kLog2e;
        if (o.S != 0.0f) {
            const float d = o.mb - mxb;
            const float f = __builtin_amdgcn_exp2f(d);
            o.A = f * (o.A + d * o.S);
            o.S = f * o.S;
        }
        o.m = mx;
        o.mb = mxb;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float t = __builtin_fmaf(z[i], kLog2e, -o.mb);
        const float e = __builtin_amdgcn_exp2f(t);
        o.S += e;
        o.A = __builtin_fmaf(e, t, o.A);
    }
}

__device__ __forceinline__ void unpack8(uint4 v, float (&z)[8]) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        z[2 * i] = f32_from_bits(w[i] << 16);
        z[2 * i + 1] = f32_from_bits(w[i] & 0xFFFF0000u);
    }
}

__global__ __launch_bounds__(kThreads) void sem_rows_kernel(const uint16_t *__restrict__ logits, int64_t V,
                                                            int64_t ld, const int32_t *__restrict__ targets,
                                                            float *__restrict__ stats) {
    const int64_t t = blockIdx.x;
    const uint4 *row = reinterpret_cast<const uint4 *>(logits + t * ld);
    const int64_t nv = V / 8;
    Online o{-__builtin_inff(), -__builtin_inff(), 0.0f, 0.0f};
    int64_t i = threadIdx.x;
    for (; i + 3 * kThreads < nv; i += 4 * kThreads) {
        uint4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = row[i + u * kThreads];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            float z[8];
            unpack8(v[u], z);
            add8(o, z);
        }
    }
    for (; i < nv; i += kThreads) {
        float z[8];
        unpack8(row[i], z);
        add8(o, z);
    }
    // fixed-order tree: within the wave by xor shuffles, then the four waves in LDS
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        Online b{__shfl_xor(o.m, off, 64), __shfl_xor(o.mb, off, 64), __shfl_xor(o.S, off, 64),
                 __shfl_xor(o.A, off, 64)};
        o = merge(o, b);
    }
    __shared__ float red[4][kThreads / 64];
    if ((threadIdx.x & 63) == 0) {
        red[0][threadIdx.x >> 6] = o.m;
        red[1][threadIdx.x >> 6] = o.mb;
        red[2][threadIdx.x >> 6] = o.S;
        red[3][threadIdx.x >> 6] = o.A;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        Online r{red[0][0], red[1][0], red[2][0], red[3][0]};
        for (int w = 1; w < kThreads / 64; ++w) r = merge(r, Online{red[0][w], red[1][w], red[2][w], red[3][w]});
        const float log2S = __builtin_amdgcn_logf(r.S);
        const float lse = (r.mb + log2S) * kLn2;
        const int32_t y = targets[t];
        const bool ok = y >= 0 && (int64_t)y < V;  // a target outside [0, V) gives NaN, reads nothing
        const float zy = ok ? f32_from_bits((uint32_t)logits[t * ld + y] << 16) : __builtin_nanf("");
        stats[4 * t + 0] = (log2S - r.A / r.S) * kLn2;   // H
        stats[4 * t + 1] = lse - zy;                      // NLL
        stats[4 * t + 2] = lse;
        stats[4 * t + 3] = 0.0f;
    }
}

// Order-preserving key of an FP32 pattern.
__device__ __forceinline__ uint32_t fkey(float f) {
    const uint32_t b = bits_from_f32(f);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

constexpr int kBatchThreads = 1024;

// Adds one to hist[bin] for each active lane.  Entropies cluster, so in the
// high-digit passes most lanes of a wave share a bin: the lanes with the first
// active lane's bin are counted with one atomic, the others add theirs alone
// (a 64-way same-address atomic serialises in the LDS).
__device__ __forceinline__ void hist_add(uint32_t *hist, bool active, uint32_t bin) {
    const uint64_t act = __ballot(active);
    if (act == 0) return;
    const int first = __builtin_ctzll(act);
    const uint32_t lb = (uint32_t)__shfl((int)bin, first, 64);
    const bool same = active && bin == lb;
    const uint64_t group = __ballot(same);
    if (same) {
        if ((int)(threadIdx.x & 63) == first) atomicAdd(&hist[lb], (uint32_t)__builtin_popcountll(group));
    } else if (active) {
        atomicAdd(&hist[bin], 1u);
    }
}

// k-th smallest (0-based) of the T entropies, by 4 passes of 8-bit radix selection.
__device__ uint32_t select_key(const float *__restrict__ stats, int64_t T, int64_t k, uint32_t *hist,
                               uint32_t *scan, uint32_t *sel) {
    uint32_t prefix = 0, mask = 0;
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        for (int i = threadIdx.x; i < 256; i += kBatchThreads) hist[i] = 0;
        __syncthreads();
        for (int64_t t0 = 0; t0 < T; t0 += kBatchThreads) {      // whole waves, so the ballots see every lane
            const int64_t t = t0 + threadIdx.x;
            const uint32_t key = t < T ? fkey(stats[4 * t]) : 0u;
            hist_add(hist, t < T && (key & mask) == prefix, (key >> shift) & 0xFFu);
        }
        __syncthreads();
        // exclusive prefix sums of the 256 counts (Hillis-Steele in LDS, the
        // first 256 threads); the bin holding rank k publishes its digit
        uint32_t c = 0, incl = 0;
        if (threadIdx.x < 256) {
            incl = c = hist[threadIdx.x];
            scan[threadIdx.x] = c;
        }
        for (int off = 1; off < 256; off <<= 1) {
            __syncthreads();                       // the previous step's sums are written
            const uint32_t add = (threadIdx.x < 256 && (int)threadIdx.x >= off) ? scan[threadIdx.x - off] : 0u;
            __syncthreads();                       // every read done before the next writes
            if (threadIdx.x < 256) {
                incl += add;
                scan[threadIdx.x] = incl;
            }
        }
        __syncthreads();
        if (threadIdx.x < 256) {
            const int64_t below = (int64_t)(incl - c);
            if (c != 0 && k >= below && k < below + (int64_t)c) {
                sel[0] = threadIdx.x;
                sel[1] = (uint32_t)below;
            }
        }
        __syncthreads();
        const uint32_t digit = sel[0];
        k -= (int64_t)sel[1];
        prefix |= digit << shift;
        mask |= 0xFFu << shift;
        __syncthreads();
    }
    return prefix;
}

// Entropies a thread holds in registers for the batch kernel: a batch of up
// to kBatchThreads * kKeyCache tokens is read from memory once; larger ones
// take select_key above, which re-reads the keys in every pass.
constexpr int kKeyCache = 8;

// Inclusive prefix sum over threads 0..255 of c (the 256 bin counts), four
// waves of 64: shuffles within each wave, then the totals of the waves
// before it (one barrier).  Threads past 255 pass 0 and get unused values.
__device__ __forceinline__ uint32_t bins_inclusive_scan(uint32_t c, uint32_t *wsum) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    uint32_t v = c;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t u = __shfl_up(v, off, 64);
        if (lane >= off) v += u;
    }
    if (w < 4 && lane == 63) wsum[w] = v;
    __syncthreads();
    uint32_t base = 0;
    for (int i = 0; i < w && i < 4; ++i) base += wsum[i];
    return v + base;
}

// k-th smallest (0-based) of the n keys held kKeyCache per thread (key j of
// thread t is entry t + j * kBatchThreads), by 4 passes of 8-bit radix
// selection: the same key select_key finds, without re-reading memory.
__device__ uint32_t select_key_cached(const uint32_t (&keys)[kKeyCache], int64_t n, int64_t k, uint32_t *hist,
                                      uint32_t *wsum, uint32_t *sel) {
    uint32_t prefix = 0, mask = 0;
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        if (threadIdx.x < 256) hist[threadIdx.x] = 0;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kKeyCache; ++j) {
            const int64_t t = threadIdx.x + (int64_t)j * kBatchThreads;
            hist_add(hist, t < n && (keys[j] & mask) == prefix, (keys[j] >> shift) & 0xFFu);
        }
        __syncthreads();
        const uint32_t c = threadIdx.x < 256 ? hist[threadIdx.x] : 0u;
        const uint32_t incl = bins_inclusive_scan(c, wsum);
        if (threadIdx.x < 256) {
            const int64_t below = (int64_t)(incl - c);
            if (c != 0 && k >= below && k < below + (int64_t)c) {
                sel[0] = threadIdx.x;
                sel[1] = (uint32_t)below;
            }
        }
        __syncthreads();
        const uint32_t digit = sel[0];
        k -= (int64_t)sel[1];
        prefix |= digit << shift;
        mask |= 0xFFu << shift;
        __syncthreads();                           // sel, wsum and hist are reused
    }
    return prefix;
}

// The (k+1)-th smallest key given the k-th, klo: klo again when at least k + 2
// keys are <= klo, else the smallest key above klo (one pass: a count and a
// minimum over the cached keys).
__device__ uint32_t next_key_cached(const uint32_t (&keys)[kKeyCache], int64_t n, int64_t k, uint32_t klo,
                                    uint32_t *wsum) {
    uint32_t cnt = 0, mn = 0xFFFFFFFFu;
#pragma unroll
    for (int j = 0; j < kKeyCache; ++j) {
        const int64_t t = threadIdx.x + (int64_t)j * kBatchThreads;
        if (t < n) {
            cnt += keys[j] <= klo ? 1u : 0u;
            if (keys[j] > klo && keys[j] < mn) mn = keys[j];
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        cnt += __shfl_xor(cnt, off, 64);
        const uint32_t o = __shfl_xor(mn, off, 64);
        mn = o < mn ? o : mn;
    }
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (lane == 0) {
        wsum[w] = cnt;
        wsum[kBatchThreads / 64 + w] = mn;
    }
    __syncthreads();
    uint64_t total = 0;
    uint32_t m = 0xFFFFFFFFu;
    for (int i = 0; i < kBatchThreads / 64; ++i) {
        total += wsum[i];
        m = wsum[kBatchThreads / 64 + i] < m ? wsum[kBatchThreads / 64 + i] : m;
    }
    __syncthreads();
    return (int64_t)total >= k + 2 ? klo : m;
}

__device__ __forceinline__ float unkey(uint32_t key) {
    return f32_from_bits((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

__global__ __launch_bounds__(kBatchThreads) void sem_batch_kernel(const float *__restrict__ stats, int64_t T,
                                                                  float lambda, float eps,
                                                                  float *__restrict__ weights,
                                                                  float *__restrict__ loss) {
    __shared__ uint32_t hist[256], scan[256], sel[2], wsum[2 * (kBatchThreads / 64)];
    __shared__ double dred[2][kBatchThreads / 64];
    __shared__ float fred[kBatchThreads / 64];

    // H_min; a batch of at most kBatchThreads * kKeyCache tokens keeps its
    // entropies' keys in registers for the selection below
    const bool cached = T <= (int64_t)kBatchThreads * kKeyCache;
    uint32_t keys[kKeyCache];
    float hmin = __builtin_inff();
    if (cached) {
        float h[kKeyCache];
#pragma unroll
        for (int j = 0; j < kKeyCache; ++j) {
            const int64_t t = threadIdx.x + (int64_t)j * kBatchThreads;
            h[j] = t < T ? stats[4 * t] : __builtin_inff();
        }
#pragma unroll
        for (int j = 0; j < kKeyCache; ++j) {
            hmin = fminf(hmin, h[j]);
            keys[j] = fkey(h[j]);
        }
    } else {
        for (int64_t t = threadIdx.x; t < T; t += kBatchThreads) hmin = fminf(hmin, stats[4 * t]);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) hmin = fminf(hmin, __shfl_xor(hmin, off, 64));
    if ((threadIdx.x & 63) == 0) fred[threadIdx.x >> 6] = hmin;
    __syncthreads();
    hmin = fred[0];
    for (int w = 1; w < kBatchThreads / 64; ++w) hmin = fminf(hmin, fred[w]);
    __syncthreads();

    // tau: linear interpolation at position q = 0.75 (T - 1), computed in FP64
    const double q = 0.75 * (double)(T - 1);
    const int64_t lo = (int64_t)q;
    const int64_t hi = lo + 1 < T ? lo + 1 : T - 1;
    double hlo, hhi;
    if (cached) {
        const uint32_t klo = select_key_cached(keys, T, lo, hist, wsum, sel);
        hlo = (double)unkey(klo);
        hhi = hi == lo ? hlo : (double)unkey(next_key_cached(keys, T, lo, klo, wsum));
    } else {
        hlo = (double)unkey(select_key(stats, T, lo, hist, scan, sel));
        hhi = hi == lo ? hlo : (double)unkey(select_key(stats, T, hi, hist, scan, sel));
    }
    const double tau = hlo + (q - (double)lo) * (hhi - hlo);
    const double denom = tau - (double)hmin + (double)eps;

    double s_nll = 0.0, s_ent = 0.0;
    for (int64_t t = threadIdx.x; t < T; t += kBatchThreads) {
        const double H = (double)stats[4 * t];
        double w = 1.0 - (H - (double)hmin) / denom;
        w = w > 0.0 ? w : 0.0;
        weights[t] = (float)w;
        s_nll += (double)stats[4 * t + 1];
        s_ent += w * H;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        s_nll += __shfl_xor(s_nll, off, 64);
        s_ent += __shfl_xor(s_ent, off, 64);
    }
    if ((threadIdx.x & 63) == 0) {
        dred[0][threadIdx.x >> 6] = s_nll;
        dred[1][threadIdx.x >> 6] = s_ent;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double a = 0.0, b = 0.0;
        for (int w = 0; w < kBatchThreads / 64; ++w) { a += dred[0][w]; b += dred[1][w]; }
        const double l_sft = a / (double)T, l_ent = b / (double)T;
        loss[0] = (float)(l_sft + (double)lambda * l_ent);
        loss[1] = (float)l_sft;
        loss[2] = (float)l_ent;
        loss[3] = (float)tau;
    }
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void sem_backward_kernel(const uint16_t *__restrict__ logits, int64_t V,
                                                                int64_t ld, const int32_t *__restrict__ targets,
                                                                const float *__restrict__ stats,
                                                                const float *__restrict__ weights, float lambda,
                                                                float scale, void *__restrict__ grad,
                                                                int64_t ldg, int64_t T) {
    const int64_t t = blockIdx.x;
    const float H = stats[4 * t], lse = stats[4 * t + 2];
    const float c = scale / (float)T;
    const float lw = lambda * weights[t];
    const int32_t y = targets[t];
    const uint4 *row = reinterpret_cast<const uint4 *>(logits + t * ld);
    const int64_t nv = V / 8;
    for (int64_t i = threadIdx.x; i < nv; i += kThreads) {
        float z[8];
        unpack8(row[i], z);
        float g[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const float lp = z[k] - lse;
            const float p = exp_fast(lp);
            float v = p - lw * p * (lp + H);
            if (8 * i + k == y) v -= 1.0f;
            g[k] = c * v;
        }
        if (BF16) {
            uint32_t o[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const __bf16 a = (__bf16)g[2 * k], b = (__bf16)g[2 * k + 1];
                o[k] = (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
            }
            reinterpret_cast<uint4 *>(reinterpret_cast<uint16_t *>(grad) + t * ldg)[i] =
                make_uint4(o[0], o[1], o[2], o[3]);
        } else {
            float4 *dst = reinterpret_cast<float4 *>(reinterpret_cast<float *>(grad) + t * ldg) + 2 * i;
            dst[0] = make_float4(g[0], g[1], g[2], g[3]);
            dst[1] = make_float4(g[4], g[5], g[6], g[7]);
        }
    }
}

}  // namespace

hipError_t launch_sem_forward(const uint16_t *logits, int64_t T, int64_t V, int64_t ld, const int32_t *targets,
                              float lambda, float eps, float *stats, float *weights, float *loss,
                              hipStream_t stream) {
    if (T == 0) return hipSuccess;
    hipLaunchKernelGGL(sem_rows_kernel, dim3((unsigned)T), dim3(kThreads), 0, stream, logits, V, ld, targets, stats);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sem_batch_kernel, dim3(1), dim3(kBatchThreads), 0, stream, stats, T, lambda, eps, weights,
                       loss);
    return hipGetLastError();
}

hipError_t launch_sem_backward(const uint16_t *logits, int64_t T, int64_t V, int64_t ld, const int32_t *targets,
                               const float *stats, const float *weights, float lambda, float scale, void *grad,
                               bool grad_bf16, int64_t ldg, hipStream_t stream) {
    if (T == 0) return hipSuccess;
    if (grad_bf16)
        hipLaunchKernelGGL(sem_backward_kernel<true>, dim3((unsigned)T), dim3(kThreads), 0, stream, logits, V, ld,
                           targets, stats, weights, lambda, scale, grad, ldg, T);
    else
        hipLaunchKernelGGL(sem_backward_kernel<false>, dim3((unsigned)T), dim3(kThreads), 0, stream, logits, V, ld,
                           targets, stats, weights, lambda, scale, grad, ldg, T);
    return hipGetLastError();
}

}  // namespace reqat
