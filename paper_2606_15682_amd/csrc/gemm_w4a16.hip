// W4A16 product for gfx950 (the MXFP4 W4A16 deployment setting: MXFP4 weights,
// bfloat16 activations):
//   Y[m][n] = sum_k x[m][k] * w^[n][k],   w^ = RN_bf16(E2M1(c) * 2^e),
// FP32 accumulation.  The weight is dequantized to the activation type in
// registers: v_cvt_scalef32_pk_bf16_fp4 returns exactly RN_bf16(code * 2^e) for
// every E8M0 scale byte 0..254 (overflow to Inf and bfloat16 subnormals
// included; checked on gfx950 for all 255 x 16 cases), and
// v_mfma_f32_16x16x32_bf16 multiplies exactly (it keeps subnormal inputs) and
// sums in FP32.  A NaN scale byte (0xFF) makes its 32 weights NaN.
//
// Decode-shaped work streams W once and is bound by how the activations reach
// the matrix cores: a workgroup owns 64 weight rows (16 per wave) and loads
// each 128-element chunk of its activation rows once into LDS, where all four
// waves read it, so every activation byte read from L2 serves 64 weight rows
// (reading it per wave, for 16 rows, made the L2 reads four times the weight
// bytes and capped the rate near 1 TB/s).  With few weight rows the K range
// is split over more workgroups (about two per CU, spread evenly, else up to
// 1024 in total; at most 12 splits) whose FP32 partial sums a second kernel
// adds in split order (deterministic).
//
// The weights come row-major (codes [N][K/2], scales [N][K/32]) or as the
// packed image of w4a16_pack_kernel: per 16-row group and 128-element chunk,
// the 1 KB of codes in the order the lanes below load them, then (after all
// code units) the 64 scale bytes, so that a wave's chunk is one contiguous
// 1 KB load instead of 64 bytes from each of 16 rows.  The two layouts differ
// only in the load addresses (kPacked); the arithmetic is the same.
//
// In a chunk, lane l takes the 32-element MX block kg = l / 16 of weight row
// l % 16 (16 code bytes + its scale byte) and the same 32 K positions of
// activation row l % 16 from LDS; MFMA step s uses the lane's elements
// 8s .. 8s+7, so A and B agree on which K each lane holds.  Rows past M or N
// re-read the last real row and are never stored.
#include <type_traits>

#include "fp4_device.h"
#include "internal.h"

namespace reqat {

namespace {

typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

#ifndef REQAT_W16_NT
#define REQAT_W16_NT 1
#endif
#ifndef REQAT_W16_KSMAX
#define REQAT_W16_KSMAX 12
#endif

#ifndef REQAT_W16_DEPTH1
#define REQAT_W16_DEPTH1 4
#endif
#ifndef REQAT_W16_TARGET
#define REQAT_W16_TARGET 1024
#endif
#ifndef REQAT_W16_XG
#define REQAT_W16_XG 2
#endif

constexpr int kThreads = 256;          // four waves
constexpr int kMaxSplits = REQAT_W16_KSMAX;

// Calls f(integral_constant<int, J>) for J = B .. E-1, unrolled at compile time.
template <int B, int E, typename F> __device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

__device__ __forceinline__ uint32_t pick4(const v4u &q, int s) {
    return s == 0 ? q.x : s == 1 ? q.y : s == 2 ? q.z : q.w;
}

// Bfloat16 weights of MFMA step s: the lane's elements 8s .. 8s+7, RN_bf16(code * 2^e)
// for the block's E8M0 byte sb.  The NaN byte 0xFF gives the FP32 scale +Inf,
// which the conversion turns into NaN for every code, zero included (checked
// on gfx950 for all 256 code pairs and the four byte selects).
__device__ __forceinline__ v8bf decode_step(const v4u &w, uint32_t sb, int s) {
    const float p2 = __builtin_bit_cast(float, sb << 23);
    const uint32_t word = pick4(w, s);
    const v2bf d0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 0);
    const v2bf d1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 1);
    const v2bf d2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 2);
    const v2bf d3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, p2, 3);
    return v8bf{d0[0], d0[1], d1[0], d1[1], d2[0], d2[1], d3[0], d3[1]};
}

// A workgroup owns 64*NT weight rows (16*NT per wave, NT MFMA column tiles)
// and 16*MT activation rows and walks the K chunks of its split ks =
// blockIdx.y (whole chunk pairs, balanced over the splits).  Each 128-element
// chunk of the activation rows is loaded once per workgroup (16 bytes per
// thread per 16-row tile), stored to LDS and read by all four waves; each LDS
// fragment feeds NT MFMAs.  With one split the results go to y; otherwise to the FP32 partial
// sums part[ks][m][n], added in split order by gemm_w4a16_reduce.
template <int MT, int NT, int kDepth, int XG, bool kPacked>
__global__ __launch_bounds__(kThreads) void gemm_w4a16_kernel(
    int64_t M, int64_t N, int64_t K, const uint16_t *__restrict__ x, int64_t ldx,
    const uint8_t *__restrict__ w_codes, const uint8_t *__restrict__ w_scales, void *__restrict__ y,
    int y_bf16, int64_t ldy, int KS, float *__restrict__ part) {
    constexpr int XP = XG * 128 + 8;                    // LDS row pitch of an x group (bfloat16 elements)
    __shared__ __attribute__((aligned(16))) uint16_t xs[2][MT * 16][XP];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, kg = lane >> 4;
    const int64_t n0 = (int64_t)blockIdx.x * (64 * NT) + 16 * NT * wave;
    int64_t nrow[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) nrow[t] = (n0 + 16 * t + r) < N ? (n0 + 16 * t + r) : N - 1;
    // packed image: 16-row group of each tile (past the last group: the last, never stored)
    const int64_t ngrp = (N + 15) / 16;
    int64_t grp[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) grp[t] = (n0 / 16 + t) < ngrp ? (n0 / 16 + t) : ngrp - 1;
    const int ks = blockIdx.y;
    const int64_t m0 = (int64_t)blockIdx.z * 16 * MT;
    const int64_t nch = K / 128;
    // splits start at even chunks: a pair of chunks is a whole 128-byte line
    // of each weight row (when K % 256 == 0)
    const int64_t npair = nch / 2;
    const int64_t c0 = 2 * (npair * ks / KS);
    const int64_t nc = (ks + 1 == KS ? nch : 2 * (npair * (ks + 1) / KS)) - c0;

    // activation chunk loader: thread t takes row t / 16 of each 16-row tile, elements 8 (t % 16) ..
    const int xr = tid >> 4, xc = (tid & 15) * 8;
    auto load_x = [&](int64_t c, v4u (&v)[MT]) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int64_t row = (m0 + 16 * mt + xr) < M ? (m0 + 16 * mt + xr) : M - 1;
            v[mt] = *reinterpret_cast<const v4u *>(x + row * ldx + c * 128 + xc);
        }
    };
    auto store_x = [&](int buf, int u, const v4u (&v)[MT]) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) *reinterpret_cast<v4u *>(&xs[buf][16 * mt + xr][128 * u + xc]) = v[mt];
    };
    // the lane's 32 codes (MX block kg of the chunk) of each of its weight rows
    // (packed: the 1 KB of group grp, chunk c, in lane order)
    auto load_w = [&](int64_t c, v4u (&v)[NT]) {
#pragma unroll
        for (int t = 0; t < NT; ++t)
            v[t] = kPacked ? *reinterpret_cast<const v4u *>(w_codes + ((grp[t] * nch + c) << 10) + lane * 16)
                           : *reinterpret_cast<const v4u *>(w_codes + nrow[t] * (K / 2) + (c * 4 + kg) * 16);
    };
    // Scale bytes of four chunks in one load: lane (r, kg) takes the dword of
    // chunk c + kg (its four blocks' E8M0 bytes; K % 128 == 0 keeps it
    // aligned); the lanes of chunk c + u read it from lane r + 16u.
    // (packed: the 64 scale bytes of group grp, chunk c, four per row)
    auto load_s = [&](int64_t c, uint32_t (&v)[NT]) {
#pragma unroll
        for (int t = 0; t < NT; ++t)
            v[t] = kPacked ? *reinterpret_cast<const uint32_t *>(w_scales + ((grp[t] * nch + c) << 6) + r * 4)
                           : *reinterpret_cast<const uint32_t *>(w_scales + nrow[t] * (K / 32) + c * 4);
    };

    v4f acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[mt][t] = v4f{};

    // Activations move in groups of XG chunks: group q travels global ->
    // registers (issued at the start of group q - 2) -> LDS (buffer q & 1,
    // stored at the start of group q - 1), so the workgroup meets at one
    // barrier per group, not per chunk.  A chunk's codes go to registers
    // kDepth chunks ahead (in pairs, below) and its scale bytes with those of
    // three neighbours, kDepth chunks ahead.  The loop is unrolled by
    // templates so every ring slot is a constant, and loads past the last
    // chunk re-read it (clamped, never used), so the main loop has no
    // branches and the compiler waits on each load alone.
    if (nc > 0) {
        constexpr int kTurn = 2 * kDepth;                      // steps per unrolled loop turn
        constexpr int kGroups = kTurn / 4;                      // scale-group ring slots
        static_assert(kTurn % XG == 0 && kDepth % 2 == 0, "loop turn of whole x groups and code pairs");
        static_assert(kDepth % 4 == 0, "scale dwords cover four chunks: the prologue loads kDepth / 4 of them");
        v4u xv[XG][MT];                                         // the next x group in flight
        v4u wq[kDepth][NT];
        uint32_t sq[kGroups][NT];                               // scale dwords of 4-chunk groups
        auto clamp = [&](int64_t i) { return c0 + (i < nc ? i : nc - 1); };
        static_for<0, kDepth / 4>([&](auto G) {                 // first: the oldest loads at the loop entry
            load_s(clamp(4 * decltype(G)::value + kg), sq[decltype(G)::value]);
        });
        static_for<0, XG>([&](auto U) { load_x(clamp(decltype(U)::value), xv[decltype(U)::value]); });
        static_for<0, kDepth>([&](auto J) { load_w(clamp(decltype(J)::value), wq[decltype(J)::value]); });
        static_for<0, XG>([&](auto U) { store_x(0, decltype(U)::value, xv[decltype(U)::value]); });
        static_for<0, XG>([&](auto U) { load_x(clamp(XG + decltype(U)::value), xv[decltype(U)::value]); });
        // step i = i0 + j of a loop turn (j static)
        auto step = [&](int64_t i, auto J) {
            constexpr int j = decltype(J)::value;
            constexpr int slot = j % kDepth, grp = (j / 4) % kGroups, u = j % XG;
            // keep each chunk's decode in its own step: hoisted, it would wait
            // on weights still in flight and shorten the prefetch
            __builtin_amdgcn_sched_barrier(0);
            const int64_t xgrp = i / XG;
            if constexpr (u == 0) {
                __syncthreads();                                // group xgrp in LDS; the other buffer free
                static_for<0, XG>([&](auto U) {                 // group xgrp + 1 (unused past the end)
                    store_x((int)((xgrp + 1) & 1), decltype(U)::value, xv[decltype(U)::value]);
                });
                static_for<0, XG>([&](auto U) {
                    load_x(clamp((xgrp + 2) * XG + decltype(U)::value), xv[decltype(U)::value]);
                });
            }
            if constexpr (j % 4 == 0)                           // the group kDepth chunks ahead
                load_s(clamp(i + kDepth + kg), sq[((j + kDepth) / 4) % kGroups]);
            uint32_t sb[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t)
                sb[t] = ((uint32_t)__builtin_amdgcn_ds_bpermute(4 * (r + 16 * (j % 4)), (int)sq[grp][t]) >>
                         (8 * kg)) & 0xFFu;
            const int buf = (int)(xgrp & 1);
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                v8bf wb[NT];
#pragma unroll
                for (int t = 0; t < NT; ++t) wb[t] = decode_step(wq[slot][t], sb[t], s);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const v4u xa = *reinterpret_cast<const v4u *>(&xs[buf][16 * mt + r][128 * u + 32 * kg + 8 * s]);
#pragma unroll
                    for (int t = 0; t < NT; ++t)
                        acc[mt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, xa), wb[t],
                                                                            acc[mt][t], 0, 0, 0);
                }
            }
            // codes go out in pairs of chunks once the odd chunk of a pair is
            // consumed: chunks 2p and 2p+1 are the two 64-byte halves of each
            // row's 128-byte line, requested back to back (one chunk at a time,
            // the halves went out a step apart: 12% slower from HBM)
            if constexpr (j % 2 == 1) {
                load_w(clamp(i - 1 + kDepth), wq[(slot + kDepth - 1) % kDepth]);
                load_w(clamp(i + kDepth), wq[slot]);
            }
        };
        int64_t i0 = 0;
        for (; i0 + kTurn <= nc; i0 += kTurn)
            static_for<0, kTurn>([&](auto J) { step(i0 + decltype(J)::value, J); });
        static_for<0, kTurn - 1>([&](auto J) {
            if (i0 + decltype(J)::value < nc) step(i0 + decltype(J)::value, J);   // uniform
        });
    }

    // D[m][n] of a 16 x 16 tile sits in lane n + 16 * (m / 4), register m % 4
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int64_t col = n0 + 16 * t + r;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t row = m0 + 16 * mt + 4 * kg + i;
                if (row < M && col < N) {
                    const float v = acc[mt][t][i];
                    if (KS > 1) part[((int64_t)ks * M + row) * N + col] = v;
                    else if (y_bf16) reinterpret_cast<__bf16 *>(y)[row * ldy + col] = (__bf16)v;
                    else reinterpret_cast<float *>(y)[row * ldy + col] = v;
                }
            }
    }
}

// y[m][n] = sum over splits, in split order, of part[ks][m][n].
__global__ __launch_bounds__(kThreads) void gemm_w4a16_reduce(int64_t M, int64_t N, int KS,
                                                              const float *__restrict__ part, void *__restrict__ y,
                                                              int y_bf16, int64_t ldy) {
    const int64_t total = M * N;
    for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < total; e += (int64_t)gridDim.x * kThreads) {
        float p[kMaxSplits];
#pragma unroll
        for (int k = 0; k < kMaxSplits; ++k) p[k] = k < KS ? part[(int64_t)k * total + e] : 0.0f;
        float v = p[0];
#pragma unroll
        for (int k = 1; k < kMaxSplits; ++k)
            if (k < KS) v += p[k];
        const int64_t row = e / N, col = e - row * N;
        if (y_bf16) reinterpret_cast<__bf16 *>(y)[row * ldy + col] = (__bf16)v;
        else reinterpret_cast<float *>(y)[row * ldy + col] = v;
    }
}

template <int MT>
hipError_t launch_mt(int64_t M, int64_t N, int64_t K, const uint16_t *x, int64_t ldx, const uint8_t *w_codes,
                     const uint8_t *w_scales, bool packed, void *y, bool y_bf16, int64_t ldy, int KS, float *part,
                     hipStream_t stream) {
    constexpr int NT = REQAT_W16_NT;
    const dim3 grid((unsigned)((N + 64 * NT - 1) / (64 * NT)), (unsigned)KS,
                    (unsigned)((M + 16 * MT - 1) / (16 * MT)));
    // chunks in flight per wave (8 measured no faster than 4)
    constexpr int kDepth = MT == 1 ? REQAT_W16_DEPTH1 : 4;
    constexpr int XG = MT == 1 ? REQAT_W16_XG : 1;
    if (packed)
        hipLaunchKernelGGL((gemm_w4a16_kernel<MT, NT, kDepth, XG, true>), grid, dim3(kThreads), 0, stream, M, N, K, x,
                           ldx, w_codes, w_scales, y, (int)y_bf16, ldy, KS, part);
    else
        hipLaunchKernelGGL((gemm_w4a16_kernel<MT, NT, kDepth, XG, false>), grid, dim3(kThreads), 0, stream, M, N, K,
                           x, ldx, w_codes, w_scales, y, (int)y_bf16, ldy, KS, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || KS == 1) return e;
    int64_t rgrid = (M * N + kThreads - 1) / kThreads;
    if (rgrid > 4096) rgrid = 4096;
    hipLaunchKernelGGL(gemm_w4a16_reduce, dim3((unsigned)rgrid), dim3(kThreads), 0, stream, M, N, KS, part, y,
                       (int)y_bf16, ldy);
    return hipGetLastError();
}

int row_tile(int64_t M) { return M <= 16 ? 1 : (M <= 32 ? 2 : 4); }

// Packed weight image (one thread per 16 code bytes, and per scale dword):
// unit (G, c) of 16-row group G and 128-element chunk c holds 1024 code bytes,
// piece q (bytes 16q .. 16q+15 of the chunk) of row 16G + r at byte
// 16 (r + 16 q), then, in the scale part, that row's four E8M0 bytes of the
// chunk at byte 4 r.  Rows past N are zero.
__global__ __launch_bounds__(kThreads) void w4a16_pack_kernel(const uint8_t *__restrict__ codes,
                                                              const uint8_t *__restrict__ scales, int64_t N,
                                                              int64_t K, uint8_t *__restrict__ packed) {
    const int64_t nch = K / 128, units = (N + 15) / 16 * nch;
    uint8_t *pscales = packed + (units << 10);
    for (int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x; p < units * 64;
         p += (int64_t)gridDim.x * kThreads) {
        const int64_t u = p >> 6, g = u / nch, c = u - g * nch;
        const int l = (int)(p & 63), r = l & 15, q = l >> 4;
        const int64_t row = 16 * g + r;
        v4u v = v4u{0u, 0u, 0u, 0u};
        uint32_t sc = 0u;
        if (row < N) {
            v = *reinterpret_cast<const v4u *>(codes + row * (K / 2) + c * 64 + q * 16);
            sc = *reinterpret_cast<const uint32_t *>(scales + row * (K / 32) + c * 4);
        }
        *reinterpret_cast<v4u *>(packed + (u << 10) + l * 16) = v;
        if (q == 0) *reinterpret_cast<uint32_t *>(pscales + (u << 6) + r * 4) = sc;
    }
}

}  // namespace

size_t w4a16_packed_bytes(int64_t N, int64_t K) { return (size_t)((N + 15) / 16) * (size_t)(K / 128) * 1088u; }

hipError_t launch_w4a16_pack(const uint8_t *codes, const uint8_t *scales, int64_t N, int64_t K, uint8_t *packed,
                             hipStream_t stream) {
    const int64_t pieces = (N + 15) / 16 * (K / 128) * 64;
    if (pieces == 0) return hipSuccess;
    int64_t grid = (pieces + kThreads - 1) / kThreads;
    if (grid > 8192) grid = 8192;
    hipLaunchKernelGGL(w4a16_pack_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream, codes, scales, N, K,
                       packed);
    return hipGetLastError();
}

// K splits, when the weight rows alone give fewer workgroups than CUs: the
// fewest splits (fewest FP32 partials to add) that give about two workgroups
// per CU, spread evenly (the average CU has at least 90% of the busiest CU's
// count, so no CU runs a round alone); when no split count up to
// REQAT_W16_KSMAX does, enough to reach REQAT_W16_TARGET workgroups.  At most
// REQAT_W16_KSMAX splits and one pair of chunks each (splits start at even
// chunks).  On 16 x 5120 x 27648 (80 row groups) the first rule picks 6:
// 20.3 us against 21.6 for 12 and 24.5 for 4, which leaves a quarter of the
// CUs with one workgroup more than the rest.  The split depends on the shape
// alone, never on the device, so results are deterministic.
int gemm_w4a16_splits(int64_t M, int64_t N, int64_t K) {
    constexpr int64_t kCUs = 256;
    const int64_t rows = 64 * REQAT_W16_NT;
    const int64_t base = ((N + rows - 1) / rows) * ((M + 16 * row_tile(M) - 1) / (16 * row_tile(M)));
    const int64_t npair = K / 256;
    if (base >= kCUs || npair <= 1) return 1;
    const int64_t kmax = REQAT_W16_KSMAX < npair ? REQAT_W16_KSMAX : npair;
    for (int64_t ks = 2; ks <= kmax; ++ks) {
        const int64_t wg = base * ks, busiest = (wg + kCUs - 1) / kCUs;
        if (10 * wg >= 18 * kCUs && 10 * wg >= 9 * busiest * kCUs) return (int)ks;
    }
    int64_t ks = (REQAT_W16_TARGET + base - 1) / base;
    return (int)(ks < kmax ? ks : kmax);
}

size_t gemm_w4a16_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    const int ks = gemm_w4a16_splits(M, N, K);
    return ks > 1 ? sizeof(float) * (size_t)ks * (size_t)M * (size_t)N : 0;
}

hipError_t launch_gemm_w4a16(int64_t M, int64_t N, int64_t K, const uint16_t *x, int64_t ldx,
                             const uint8_t *w_codes, const uint8_t *w_scales, bool packed, void *y, bool y_bf16,
                             int64_t ldy, float *workspace, hipStream_t stream) {
    if (M == 0 || N == 0) return hipSuccess;
    const int ks = gemm_w4a16_splits(M, N, K);
    switch (row_tile(M)) {
    case 1: return launch_mt<1>(M, N, K, x, ldx, w_codes, w_scales, packed, y, y_bf16, ldy, ks, workspace, stream);
    case 2: return launch_mt<2>(M, N, K, x, ldx, w_codes, w_scales, packed, y, y_bf16, ldy, ks, workspace, stream);
    default: return launch_mt<4>(M, N, K, x, ldx, w_codes, w_scales, packed, y, y_bf16, ldy, ks, workspace, stream);
    }
}

}  // namespace reqat
