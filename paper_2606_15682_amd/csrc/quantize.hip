// Block quantizer, fake-quant and tensor absmax kernels for gfx950.
//
// Quantize: a lane owns one scale block at a time (16 bfloat16 = 32 B for
// NVFP4, 32 = 64 B for MXFP4); a wave takes U adjacent segments of 64 blocks
// per step and the grid's waves sweep the tensor front to back, so the block
// absmax, the scale and the rounding are computed once per block with no
// cross-lane traffic, and per-thread set-up (global scale) is paid once.  Consecutive lanes own consecutive blocks, so every wave-wide 16-byte
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
// NVFP4 computed global scale, by tensor size:
//   up to 2^16 elements: one launch; each workgroup reads the whole tensor for
//     its amax before its block loop (kGLocal);
//   up to 2^19 segments of 64 blocks: one pass over x under per-segment
//     reference scales, then a fix-up kernel (kGDeferred, nv_fixup_kernel);
//   beyond: a first pass writes one partial absmax per workgroup into the
//     workspace; each quantize workgroup folds the partials (<= 4096 words,
//     L2-resident) before its block loop (kGFold).
// Workgroup 0 publishes g in every case.
#include <type_traits>

#include "fp4_device.h"
#include "internal.h"
#include "quant_block.h"
#include "rht_exact.h"

namespace reqat {

namespace {

constexpr int kThreads = 256;
#ifndef REQAT_Q_GROUPS
#define REQAT_Q_GROUPS 4096
#endif
// blocks per lane per step: codes output / fake-quant output / both
#ifndef REQAT_Q_UCODES
#define REQAT_Q_UCODES 1
#endif
#ifndef REQAT_Q_UFQ
#define REQAT_Q_UFQ 2
#endif
#ifndef REQAT_Q_UBOTH
#define REQAT_Q_UBOTH 2
#endif
#ifndef REQAT_Q_BLOCKED
#define REQAT_Q_BLOCKED 0
#endif
#ifndef REQAT_Q_SPW
#define REQAT_Q_SPW 2
#endif
// grid cap of the block loop (one partial maximum per workgroup)
constexpr int kMaxGroups = REQAT_Q_GROUPS < kMaxPartials ? REQAT_Q_GROUPS : kMaxPartials;
constexpr int kMaxDeferredFqGroups = 1024;  // grid cap of the one-pass fake-quant passes (launch_quantize)
constexpr int kSeg = 64;                    // blocks per segment: one per lane of a wave
constexpr int kSegPerWave = REQAT_Q_SPW;    // segments per wave the grid size aims at

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

// ---------------------------------------------------------------- block loop

// How the NVFP4 global scale is obtained.
enum GMode : int {
    kGFixed = 0,      // read from *gptr (NVFP4 given g), or none (MXFP4)
    kGFold = 1,       // folded from the partial maxima of a preceding absmax pass
    kGDeferred = 2,   // per-segment reference, corrected by nv_fixup_kernel
    kGLocal = 3,      // small tensor: every workgroup reads all of x for the amax first
};


__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        uint32_t o = __shfl_xor(v, off, 64);
        v = v < o ? v : o;
    }
    return v;
}

// Global scale from the partial maxima.  Every thread issues its (at most
// kMaxPartials / kThreads) loads at once, so the fold costs one L2 round trip.
__device__ __forceinline__ float fold_partials(const uint32_t *__restrict__ partials, int nparts) {
    __shared__ uint32_t red[kThreads / 64];
    constexpr int kPer = (kMaxPartials + kThreads - 1) / kThreads;
    uint32_t p[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int i = (int)threadIdx.x + j * kThreads;
        p[j] = i < nparts ? partials[i] : 0u;
    }
    uint32_t m = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) m = m > p[j] ? m : p[j];
    m = wave_max_u32(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    uint32_t r = red[0];
#pragma unroll
    for (int i = 1; i < kThreads / 64; ++i) r = r > red[i] ? r : red[i];
    return nv_global_scale(r);
}

// Blocks are grouped in segments of kSeg = 64 consecutive blocks, one per lane
// of a wave.  Each step of a wave takes U adjacent segments (loads of all U
// issued before any is used): wave w of workgroup b starts at segment
// (4 b + w) U, and steps advance by all the grid's waves (4 G U segments), so
// the grid sweeps x front to back.  The U segments of a step are adjacent
// rather than a grid apart: on gfx950 a stream whose concurrent loads sit a
// grid stride apart reads 19% slower than one sweeping contiguous memory.
//
// kGDeferred (NVFP4, computed g, one pass over x): the final g needs the tensor
// amax, which is only known once every block has been read.  Each segment is
// therefore quantized under its own reference g_r = the power-of-two global
// scale rule applied to the segment's amax (g_r <= g, both powers of two).
// Dividing g by a power of two only moves the exponent of s, so codes, s*g
// and fake-quant values under g_r equal those under g for every block whose
// scale under g is still a normal E4M3 value; nv_fixup_kernel then lowers the
// scale exponents by log2(g/g_r) and re-quantizes from x only the blocks whose
// scale would leave the normal range.  The segment table records, per
// segment, log2(g_r) + 127 (0 when the segment holds no non-zero finite block,
// whose outputs do not depend on g) and the smallest scale exponent field among
// its non-zero finite blocks; each workgroup also writes the maximum finite
// magnitude of its elements to partials[blockIdx.x].
template <int FMT, int OUT, int GM, int U>
__global__ __launch_bounds__(kThreads) void quantize_kernel(
    const uint16_t *__restrict__ x, int64_t rows, int64_t cols, int64_t ldx,
    uint8_t *__restrict__ codes, uint8_t *__restrict__ scales, uint16_t *__restrict__ y,
    int64_t ldy, float *gptr, uint32_t *__restrict__ partials, int nparts,
    uint16_t *__restrict__ seg_table) {
    constexpr int B = FMT == kMX ? 32 : 16;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nb = cols / B;
    const int64_t total = rows * nb;
    const int64_t nseg = (total + kSeg - 1) / kSeg;
    const bool narrow = total < (int64_t(1) << 32);
#if REQAT_Q_BLOCKED
    // workgroup i owns the contiguous segments [nseg i / G, nseg (i + 1) / G),
    // its four waves every fourth one
    const int64_t s_begin = nseg * blockIdx.x / gridDim.x + wave;
    const int64_t s_end = nseg * (blockIdx.x + 1) / gridDim.x;
    const int64_t useg = 4, sstride = 4 * U;
#else
    const int64_t s_begin = ((int64_t)blockIdx.x * 4 + wave) * U;
    const int64_t s_end = nseg;
    const int64_t useg = 1, sstride = (int64_t)gridDim.x * 4 * U;
#endif

    // Loads the U blocks of the step starting at segment s.  A lane without a
    // block there loads the tensor's last block instead (always valid, never
    // used), so the loads need no branch.
    auto load_step = [&](int64_t s, uint32_t (&wd)[U][B / 2]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            int64_t b = (s + useg * u) * kSeg + lane;
            b = (s + useg * u < s_end && b < total) ? b : total - 1;
            load_block<B>(x + block_offset(b, nb, cols, ldx, B, narrow), wd[u]);
        }
    };

    // kGLocal: the first step's blocks are requested together with the amax
    // pass (the grid gives each wave at most one segment, launched with U = 1,
    // so this is the wave's only step): one memory round trip for both.
    uint32_t wfirst[U][B / 2];
    if (GM == kGLocal && s_begin < s_end) load_step(s_begin, wfirst);

    GScale G = make_gscale(1.0f);
    if (FMT == kNV && GM == kGFold) {
        G = make_gscale(fold_partials(partials, nparts));
        if (blockIdx.x == 0 && threadIdx.x == 0) *gptr = G.g;
    } else if (FMT == kNV && GM == kGLocal) {
        G = make_gscale(local_global_scale<kThreads>(x, rows, cols, ldx));
        if (blockIdx.x == 0 && threadIdx.x == 0) *gptr = G.g;
    } else if (FMT == kNV && GM == kGFixed) {
        G = make_gscale(*gptr);
    }

    uint32_t mloc = 0;                                  // kGDeferred: finite max of this lane's elements
    auto run_step = [&](int64_t s, const uint32_t (&wc)[U][B / 2]) {
        uint32_t am[U];
        int64_t blk[U];
        bool act[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            blk[u] = (s + useg * u) * kSeg + lane;
            act[u] = s + useg * u < s_end && blk[u] < total;
            am[u] = act[u] ? block_mag_max<B>(wc[u]) : 0u;
        }

        GScale Gs[U];
        uint32_t segmax[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            Gs[u] = G;
            if (GM == kGDeferred) {
                const bool bad = am[u] >= 0x7F80u;
                const uint32_t fm = bad ? block_finite_max<B>(wc[u]) : am[u];
                mloc = mloc > fm ? mloc : fm;
                segmax[u] = wave_max_u32(bad ? 0u : am[u]);
                Gs[u] = make_gscale(nv_global_scale(segmax[u]));
            }
        }

        bool general[U];
        uint32_t sbyte[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            sbyte[u] = 0u;
            general[u] = false;
            if (act[u]) {
                const BlockPlan pl = plan_block<FMT, OUT, false>(am[u], Gs[u]);
                sbyte[u] = pl.sbyte;
                general[u] = !pl.fast;
                if (pl.fast) {
                    uint16_t *ydst = OUT != kCodes ? y + block_offset(blk[u], nb, cols, ldy, B, narrow) : nullptr;
                    emit_fast<FMT, OUT>(wc[u], pl, blk[u], codes, scales, ydst);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (general[u]) {
                uint16_t *ydst = OUT != kCodes ? y + block_offset(blk[u], nb, cols, ldy, B, narrow) : nullptr;
                sbyte[u] = emit_general<FMT, OUT>(x + block_offset(blk[u], nb, cols, ldx, B, narrow), Gs[u], blk[u],
                                                  codes, scales, ydst);
            }
            if (GM == kGDeferred && s + useg * u < s_end) {
                const bool live = act[u] && am[u] != 0u && am[u] < 0x7F80u;
                const uint32_t emin = wave_min_u32(live ? sbyte[u] >> 3 : 0xFFu);
                if (lane == 0)
                    seg_table[s + useg * u] =
                        segmax[u] ? (uint16_t)((uint32_t)(Gs[u].kg + 127) | (emin << 8)) : (uint16_t)0;
            }
        }
    };
    int64_t s = s_begin;
    if (GM == kGLocal && s < s_end) {
        run_step(s, wfirst);
        s += sstride;
    }
    for (; s < s_end; s += sstride) {
        uint32_t wc[U][B / 2];
        load_step(s, wc);
        run_step(s, wc);
    }

    if (GM == kGDeferred) {
        __shared__ uint32_t red[kThreads / 64];
        mloc = wave_max_u32(mloc);
        if (lane == 0) red[wave] = mloc;
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t r = red[0];
            for (int i = 1; i < kThreads / 64; ++i) r = r > red[i] ? r : red[i];
            partials[blockIdx.x] = r;
        }
    }
}

// Subtracts sub (= sh << 3 < 128, a lowering of the exponent field by sh) from
// each of the four scale bytes in v except 0x00 (zero block) and 0x7F (NaN
// block), whose meaning does not depend on g.  Every other byte must have an
// exponent field > sh, so no byte borrows from its neighbour.
__device__ __forceinline__ uint32_t lower_scale_bytes(uint32_t v, uint32_t sub) {
    const uint32_t z = ~(((v & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | v | 0x7F7F7F7Fu);   // 0x80 where a byte is 0x00
    const uint32_t t = v ^ 0x7F7F7F7Fu;
    const uint32_t n = ~(((t & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | t | 0x7F7F7F7Fu);   // 0x80 where a byte is 0x7F
    const uint32_t mask = 0x01010101u & ~((z | n) >> 7);
    return v - mask * sub;
}

// Second kernel of the one-pass NVFP4 quantizer (see quantize_kernel): folds
// the partial maxima into g, publishes it, and corrects every segment whose
// reference scale differs from g by the factor 2^sh.  One lane per segment:
// when the segment's smallest scale exponent field exceeds sh, every block
// keeps a normal scale, so codes and fake-quant values stand and only the
// segment's 64 scale bytes are lowered (codes outputs).  Otherwise the wave
// walks such segments together, one lane per block, lowering the bytes that
// stay normal and re-quantizing the other blocks from x under g (fake-quant
// alone, with no scale bytes to tell them apart: every block of the segment).
// The lane's first table entry and scale bytes are requested before the fold,
// so their latency overlaps it.
template <int OUT>
__global__ __launch_bounds__(kThreads) void nv_fixup_kernel(
    const uint16_t *__restrict__ x, int64_t rows, int64_t cols, int64_t ldx,
    uint8_t *__restrict__ codes, uint8_t *__restrict__ scales, uint16_t *__restrict__ y,
    int64_t ldy, float *gptr, const uint32_t *__restrict__ partials, int nparts,
    const uint16_t *__restrict__ seg_table) {
    const int lane = threadIdx.x & 63;
    const int64_t nb = cols / 16;
    const int64_t total = rows * nb;
    const int64_t nseg = (total + kSeg - 1) / kSeg;
    const bool narrow = total < (int64_t(1) << 32);
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    const int64_t first = (int64_t)blockIdx.x * kThreads + (threadIdx.x & ~63);

    auto fetch = [&](int64_t seg, uint32_t &m, uint4 (&v)[4]) {
        m = 0u;
        if (seg < nseg) {
            m = seg_table[seg];
            if (OUT != kFakeQuant && total - seg * kSeg >= kSeg) {
                const uint4 *p = reinterpret_cast<const uint4 *>(scales + seg * kSeg);
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = p[i];
            }
        }
    };
    uint32_t m;
    uint4 v[4] = {};
    fetch(first + lane, m, v);

    const GScale G = make_gscale(fold_partials(partials, nparts));
    if (blockIdx.x == 0 && threadIdx.x == 0) *gptr = G.g;

    for (int64_t s0 = first; s0 < nseg; s0 += stride) {
        if (s0 != first) fetch(s0 + lane, m, v);
        const int64_t seg = s0 + lane;
        int sh = 0;
        bool redo = false;
        if (m != 0u) sh = G.kg - ((int)(m & 0xFFu) - 127);
        if (sh > 0) {
            redo = (int)(m >> 8) <= sh;
            if (OUT != kFakeQuant && !redo) {
                const uint32_t sub = (uint32_t)sh << 3;
                const int64_t n = total - seg * kSeg;
                if (n >= kSeg) {
                    uint4 *p = reinterpret_cast<uint4 *>(scales + seg * kSeg);
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        p[i] = make_uint4(lower_scale_bytes(v[i].x, sub), lower_scale_bytes(v[i].y, sub),
                                          lower_scale_bytes(v[i].z, sub), lower_scale_bytes(v[i].w, sub));
                } else {
                    for (int64_t i = 0; i < n; ++i) {
                        const uint32_t b = scales[seg * kSeg + i];
                        scales[seg * kSeg + i] = (uint8_t)lower_scale_bytes(b, sub);
                    }
                }
            }
        }

        uint64_t flags = __ballot(redo);
        while (flags) {
            const int l = __builtin_ctzll(flags);
            flags &= flags - 1;
            const int lsh = __shfl(sh, l, 64);
            const int64_t blk = (s0 + l) * kSeg + lane;
            if (blk < total) {
                bool requant = true;
                if (OUT != kFakeQuant) {
                    const uint32_t b = scales[blk];
                    if (b == 0u || b == 0x7Fu) {
                        requant = false;
                    } else if ((int)(b >> 3) > lsh) {
                        scales[blk] = (uint8_t)(b - ((uint32_t)lsh << 3));
                        requant = false;
                    }
                }
                if (requant) {
                    const uint16_t *xsrc = x + block_offset(blk, nb, cols, ldx, 16, narrow);
                    uint16_t *ydst = OUT != kCodes ? y + block_offset(blk, nb, cols, ldy, 16, narrow) : nullptr;
                    uint32_t w[8];
                    load_block<16>(xsrc, w);
                    const BlockPlan pl = plan_block<kNV, OUT, false>(block_mag_max<16>(w), G);
                    if (pl.fast) emit_fast<kNV, OUT>(w, pl, blk, codes, scales, ydst);
                    else emit_general<kNV, OUT>(xsrc, G, blk, codes, scales, ydst);
                }
            }
        }
    }
}

// ---------------------------------------------------------------- block rotation

// MXFP4 activations may be rotated block by block before quantization (a
// randomized Hadamard transform per 32-element block, Sec. 4.3 and App. C.2):
// y = H_32 D x / sqrt(32), D = diag(d), d_j = -1 where bit j of `signs` is set,
// H_32 the Sylvester Hadamard matrix.  The codes and the scale are those of
// the exact real y (see rht_exact.h).
//
// Fast path: y^ = s^ * RN(1/sqrt(32)) with s^ = H D x in FP32 (the fast
// Walsh-Hadamard transform in five stages of sums and differences).  Its error
// is at most (7u + O(u^2)) / sqrt(32) * sum|x| + 2^-150 (u = 2^-24: one
// rounding per stage on each input's path, one in the constant, one in the
// product; sums of bfloat16 inputs are exact where they are subnormal).  With
//     err = 2.5 u sum|x| + 2^-149
// (about 1.8 times that, which also covers the FP32 sum|x|), the exact y_i lies
// strictly between the two ends y^_i -+ copysign(err, y^_i) (each one FP32
// rounding of an exact product-sum, within the margin).  A decision is kept
// when it comes out the same at both ends: the scale byte of max|y^| -+ err,
// and the code (sign included) of each element's ends; an end of -0 or of the
// wrong sign gives a different code.  A block where any of them differs, or
// with sum|x| >= 2^127 (where the FP32 sums could overflow), is decided
// exactly instead, by the whole wave (rotated_exact_wave).  About one block in
// a thousand of Gaussian or Student-t activations takes that path.

constexpr uint32_t kInvSqrt32 = 0x3E3504F3u;   // 1/sqrt(32) rounded to nearest FP32
constexpr float kRotErr = 2.5f * 0x1p-24f;      // err = kRotErr * sum|x| + 2^-149

// The unnormalized FP32 transform s^ = H D x of one block (y^ = s^ / sqrt(32));
// returns the FP32 sum of |x|.
__device__ __forceinline__ float rotate32(const uint32_t (&w)[16], uint32_t signs, float (&t)[32]) {
    float sabs = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const uint32_t lo = (w[i] << 16) ^ (((signs >> (2 * i)) & 1u) << 31);
        const uint32_t hi = (w[i] & 0xFFFF0000u) ^ (((signs >> (2 * i + 1)) & 1u) << 31);
        t[2 * i] = f32_from_bits(lo);
        t[2 * i + 1] = f32_from_bits(hi);
        sabs += __builtin_fabsf(t[2 * i]) + __builtin_fabsf(t[2 * i + 1]);
    }
#pragma unroll
    for (int h = 1; h < 32; h *= 2)
#pragma unroll
        for (int i = 0; i < 32; i += 2 * h)
#pragma unroll
            for (int j = i; j < i + h; ++j) {
                const float a = t[j], b = t[j + h];
                t[j] = a + b;
                t[j + h] = a - b;
            }
    return sabs;
}

// E8M0 byte of the smallest e in [-127, 127] with amax <= 6 * 2^e, for an FP32
// magnitude pattern: with amax = 1.f * 2^E that is E - 2 when 1.f <= 1.5, else E - 1.
__device__ __forceinline__ uint32_t mx_scale_byte_f32(uint32_t am) {
    if (am == 0u) return 0u;
    int E;
    uint32_t frac;
    if ((am >> 23) != 0u) {
        E = (int)(am >> 23) - 127;
        frac = am & 0x7FFFFFu;
    } else {                                   // FP32 subnormal: normalize
        const int p = 31 - __builtin_clz(am);
        E = p - 149;
        frac = (am << (23 - p)) & 0x7FFFFFu;
    }
    int e = frac <= 0x400000u ? E - 2 : E - 1;
    e = e < -127 ? -127 : (e > 127 ? 127 : e);
    return (uint32_t)(e + 127);
}

// Codes of 8 FP32 values at scale p2 (one packed word).
__device__ __forceinline__ uint32_t cvt8(const float *v, float p2) {
    uint32_t word = 0;
    word = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word, v[0], v[1], p2, 0);
    word = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word, v[2], v[3], p2, 1);
    word = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word, v[4], v[5], p2, 2);
    word = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word, v[6], v[7], p2, 3);
    return word;
}

// The fast path's decisions: true (and sbyte, cw) when every one is proven.
// t holds s^ (unnormalized); the ends y^ -+ copysign(err, y^) are formed as
// single fused products with the FP32 constant RN(1/sqrt(32)), so y^ itself is
// never rounded (the bound above covers this form too).
// v_cvt_scalef32_pk_fp4_f32 rounds an FP32 value v to the nearest E2M1 value
// of v / 2^e with ties to the even code (checked on gfx950 for every scale
// 2^-126..2^127 at each midpoint and its neighbouring FP32 values).
__device__ __forceinline__ bool rotated_certified(const float (&t)[32], float sabs, uint32_t &sbyte,
                                                  uint32_t (&cw)[4]) {
    const float c = f32_from_bits(kInvSqrt32);
    float ams = 0.0f;
#pragma unroll
    for (int j = 0; j < 32; j += 2)
        ams = __builtin_fmaxf(ams, __builtin_fmaxf(__builtin_fabsf(t[j]), __builtin_fabsf(t[j + 1])));
    const float err = __builtin_fmaf(sabs, kRotErr, 0x1p-149f);
    const float amf = ams * c;
    const float alo = amf - err, ahi = amf + err;
    // no partial sum can overflow while sum|x| < 2^127 (and then y^, err and ahi are finite)
    bool ok = sabs < 0x1p127f;
    const uint32_t slo = alo > 0.0f ? mx_scale_byte_f32(bits_from_f32(alo)) : 0u;
    sbyte = mx_scale_byte_f32(bits_from_f32(ahi));
    ok = ok && slo == sbyte && sbyte >= 1u;         // scale byte 0 has no FP32 scale operand
    const float p2 = f32_from_bits(sbyte << 23);
    uint32_t diff = 0u;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        float lo[8], hi[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const float v = t[8 * q + k];
            const float se = f32_from_bits(bits_from_f32(err) | (bits_from_f32(v) & 0x80000000u));
            lo[k] = __builtin_fmaf(v, c, -se);
            hi[k] = __builtin_fmaf(v, c, se);
        }
        const uint32_t wl = cvt8(lo, p2), wh = cvt8(hi, p2);
        diff |= wl ^ wh;
        cw[q] = wh;
    }
    return ok && diff == 0u;
}

// Stores one rotated block: codes and scale byte, or the fake-quant values
// code * 2^e (exact in bfloat16; a NaN block is 0x7FC0).
template <int OUT>
__device__ __forceinline__ void store_rotated(uint32_t sbyte, const uint32_t (&cw)[4], bool bad, int64_t blk,
                                              uint8_t *codes, uint8_t *scales, uint16_t *ydst) {
    if (OUT == kCodes) {
        *reinterpret_cast<uint4 *>(codes + blk * 16) = make_uint4(cw[0], cw[1], cw[2], cw[3]);
        scales[blk] = (uint8_t)sbyte;
        return;
    }
    uint4 *dst = reinterpret_cast<uint4 *>(ydst);
    if (!bad && sbyte >= 3u) {
        const float p2 = f32_from_bits(sbyte << 23);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            uint32_t o[4];
            fq_fast_mx(cw[q], p2, o);
            dst[q] = make_uint4(o[0], o[1], o[2], o[3]);
        }
        return;
    }
    const double S = __builtin_ldexp(1.0, (int)sbyte - 127);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        uint32_t o[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            uint32_t h2[2];
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                const uint32_t c = (cw[q] >> (8 * k + 4 * hf)) & 0xFu;
                const double v = (double)e2m1_mag_value((int)(c & 7u)) * S;
                h2[hf] = bad ? 0x7FC0u : (bf16_rne_from_double(v) | ((c & 8u) << 12));
            }
            o[k] = h2[0] | (h2[1] << 16);
        }
        dst[q] = make_uint4(o[0], o[1], o[2], o[3]);
    }
}

// Exact decisions for the block at `bsrc` (32 finite bfloat16 values), with
// the whole wave taking part (every lane must be active): lane j (and j + 32)
// holds input j; in units of 2^(min sh) the inputs are integers, and with an
// exponent spread of at most 40 the five butterfly stages across lanes compute
// the sums S_i exactly in FP64, lane i ending with S_i.  The scale and the
// codes then follow from signs of fused multiply-adds (rht_exact.h).  Wider
// spreads go to the wide-integer path on lane 0, its words in `wide` (LDS).
// Returns the scale byte; cw (the same in every lane) gets the packed codes.
__device__ __forceinline__ uint32_t rotated_exact_wave(const uint16_t *bsrc, uint32_t signs, int lane,
                                                       uint32_t (&cw)[4], uint32_t *wide) {
    const int j = lane & 31;
    const uint32_t h = bsrc[j];
    bool neg;
    uint32_t m;
    int sh;
    rht::int_parts(h, ((signs >> j) & 1u) != 0u, neg, m, sh);
    int lo = m ? sh : 1 << 20, hi = m ? sh : -1;
#pragma unroll
    for (int off = 16; off > 0; off >>= 1) {            // lanes 32..63 mirror 0..31
        const int lo2 = __shfl_xor(lo, off, 64), hi2 = __shfl_xor(hi, off, 64);
        lo = lo < lo2 ? lo : lo2;
        hi = hi > hi2 ? hi : hi2;
    }
    const int shmin = __builtin_amdgcn_readfirstlane(lo), shmax = __builtin_amdgcn_readfirstlane(hi);
#pragma unroll
    for (int q = 0; q < 4; ++q) cw[q] = 0u;
    if (shmax < 0) return 0u;                           // every input is +-0: y == 0
    if (shmax - shmin > 40) {
        uint32_t sb = 0u;
        if (lane == 0) {
#pragma unroll 1
            for (int k = 0; k < 16; ++k) wide[k] = (uint32_t)bsrc[2 * k] | ((uint32_t)bsrc[2 * k + 1] << 16);
            uint32_t c4[4];
            rht::block_wide(signs, sb, c4, wide);
#pragma unroll
            for (int q = 0; q < 4; ++q) wide[q] = c4[q];
        }
        sb = (uint32_t)__builtin_amdgcn_readfirstlane((int)sb);
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
#pragma unroll
        for (int q = 0; q < 4; ++q) cw[q] = (uint32_t)__builtin_amdgcn_readfirstlane((int)wide[q]);
        __builtin_amdgcn_wave_barrier();
        return sb;
    }
    const double v0 = m ? __builtin_ldexp((double)m, sh - shmin) : 0.0;   // <= 255 * 2^40: exact
    double v = neg ? -v0 : v0;
#pragma unroll
    for (int off = 1; off < 32; off <<= 1) {            // integers below 2^53: exact
        const double o = __shfl_xor(v, off, 64);
        v = (j & off) ? o - v : v + o;
    }
    double amax = __builtin_fabs(v);
#pragma unroll
    for (int off = 16; off > 0; off >>= 1) amax = __builtin_fmax(amax, __shfl_xor(amax, off, 64));
    {
        const uint64_t ab = __builtin_bit_cast(uint64_t, amax);
        const uint32_t alo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)ab);
        const uint32_t ahi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(ab >> 32));
        amax = __builtin_bit_cast(double, (uint64_t)alo | ((uint64_t)ahi << 32));
    }
    if (amax == 0.0) return 0u;
    // smallest e with S_max^2 <= 1152 * 2^P, P = 2e + 266 - 2 shmin: with S_max in
    // [2^L, 2^(L+1)) it is L + shmin - 138 or one above
    const int L = (int)((__builtin_bit_cast(uint64_t, amax) >> 52) & 0x7FFu) - 1023;
    int e = L + shmin - 138;
    e = e < -127 ? -127 : (e > 127 ? 127 : e);
    while (e > -127 && __builtin_fma(amax, amax, -__builtin_ldexp(1152.0, 2 * e - 2 + 266 - 2 * shmin)) < 0.0) --e;
    while (e < 127 && !(__builtin_fma(amax, amax, -__builtin_ldexp(1152.0, 2 * e + 266 - 2 * shmin)) < 0.0)) ++e;
    const int P = 2 * e + 266 - 2 * shmin;
    uint32_t m3 = 0u;
#pragma unroll
    for (int k = 0; k < 7; ++k) {
        const double bound = __builtin_ldexp((double)(2u * rht::mid_k(k) * rht::mid_k(k)), P);
        m3 += __builtin_fma(v, v, -bound) > 0.0 ? 1u : 0u;
    }
    // code of output j in nibble j % 8 of word j / 8: OR over groups of 8 lanes
    uint32_t word = (m3 | (v < 0.0 ? 8u : 0u)) << (4 * (j & 7));
#pragma unroll
    for (int off = 1; off < 8; off <<= 1) word |= __shfl_xor(word, off, 64);
#pragma unroll
    for (int q = 0; q < 4; ++q) cw[q] = (uint32_t)__builtin_amdgcn_readlane((int)word, 8 * q);
    return (uint32_t)(e + 127);
}

// One lane per 32-element block, blocks in segments of 64 (one per lane of a
// wave), wave w of workgroup b taking segments b*4 + w + k*(4*grid).  After
// the wave's fast stores, the blocks the fast path could not decide are
// decided exactly one at a time by the whole wave (about one wave in ten
// has one, for Gaussian or Student-t activations).
template <int OUT>
__global__ __launch_bounds__(kThreads) void quantize_rht_kernel(
    const uint16_t *__restrict__ x, int64_t rows, int64_t cols, int64_t ldx, uint32_t signs,
    uint8_t *__restrict__ codes, uint8_t *__restrict__ scales, uint16_t *__restrict__ y, int64_t ldy) {
    __shared__ uint32_t wide_buf[4][rht::kWideWords];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nb = cols / 32;
    const int64_t total = rows * nb;
    const int64_t nseg = (total + kSeg - 1) / kSeg;
    const bool narrow = total < (int64_t(1) << 32);
    const int64_t step = (int64_t)gridDim.x * 4;
    for (int64_t s = (int64_t)blockIdx.x * 4 + wave; s < nseg; s += step) {
        const int64_t blk = s * kSeg + lane;
        const int64_t b = blk < total ? blk : total - 1;       // branch-free load, result unused
        const uint16_t *src = x + block_offset(b, nb, cols, ldx, 32, narrow);
        uint32_t w[16];
        load_block<32>(src, w);
        float t[32];
        const float sabs = rotate32(w, signs, t);
        // a NaN or Inf input makes sum|x| NaN or Inf
        const bool bad = !(sabs < 0x1p127f) && block_mag_max<32>(w) >= 0x7F80u;
        uint32_t sbyte, cw[4];
        bool done = rotated_certified(t, sabs, sbyte, cw);
        if (bad || sabs == 0.0f) {                             // NaN block, or every input +-0 (y == 0)
            sbyte = bad ? 0xFFu : 0u;
#pragma unroll
            for (int q = 0; q < 4; ++q) cw[q] = 0u;
            done = true;
        }
        uint16_t *ydst = nullptr;
        if (OUT == kFakeQuant && blk < total) ydst = y + block_offset(blk, nb, cols, ldy, 32, narrow);
        if (blk < total && done) store_rotated<OUT>(sbyte, cw, bad, blk, codes, scales, ydst);
        uint64_t pend = __ballot(blk < total && !done);
        while (pend) {                                         // wave-uniform
            const int L = __builtin_ctzll(pend);
            pend &= pend - 1;
            const uint64_t pa = (uint64_t)(uintptr_t)src;
            const uint16_t *bsrc = (const uint16_t *)(uintptr_t)(
                (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)pa, L) |
                ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(pa >> 32), L) << 32));
            uint32_t ecw[4];
            const uint32_t esb = rotated_exact_wave(bsrc, signs, lane, ecw, wide_buf[wave]);
            if (lane == L) store_rotated<OUT>(esb, ecw, false, blk, codes, scales, ydst);
        }
    }
}

// Writes g = 1 (the global scale of a tensor with no elements).
__global__ void unit_scale_kernel(float *gptr) { *gptr = 1.0f; }

template <int FMT, int OUT, int GM, int U>
hipError_t launch_loop(int grid, const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx, uint8_t *codes,
                       uint8_t *scales, uint16_t *y, int64_t ldy, float *gptr, uint32_t *partials, int nparts,
                       uint16_t *seg_table, hipStream_t stream) {
    hipLaunchKernelGGL((quantize_kernel<FMT, OUT, GM, U>), dim3(grid), dim3(kThreads), 0, stream, x, rows, cols,
                       ldx, codes, scales, y, ldy, gptr, partials, nparts, seg_table);
    return hipGetLastError();
}

template <int FMT, int OUT>
hipError_t launch_fmt_out(GSrc gsrc, bool local, bool deferred, int grid, const uint16_t *x, int64_t rows,
                          int64_t cols, int64_t ldx, uint8_t *codes, uint8_t *scales, uint16_t *y, int64_t ldy,
                          float *gptr, uint32_t *partials, int nparts, uint16_t *seg_table, hipStream_t stream) {
    constexpr int U = OUT == kCodes ? REQAT_Q_UCODES : OUT == kFakeQuant ? REQAT_Q_UFQ : REQAT_Q_UBOTH;
    if (FMT == kNV && local)   // one segment per wave, one step (see quantize_kernel)
        return launch_loop<FMT, OUT, kGLocal, 1>(grid, x, rows, cols, ldx, codes, scales, y, ldy, gptr, partials,
                                                nparts, seg_table, stream);
    if (FMT == kNV && deferred)
        return launch_loop<FMT, OUT, kGDeferred, U>(grid, x, rows, cols, ldx, codes, scales, y, ldy, gptr,
                                                   partials, nparts, seg_table, stream);
    if (FMT == kNV && gsrc == kGComputed)
        return launch_loop<FMT, OUT, kGFold, U>(grid, x, rows, cols, ldx, codes, scales, y, ldy, gptr, partials,
                                               nparts, seg_table, stream);
    return launch_loop<FMT, OUT, kGFixed, U>(grid, x, rows, cols, ldx, codes, scales, y, ldy, gptr, partials,
                                            nparts, seg_table, stream);
}

}  // namespace

hipError_t launch_unit_scale(float *gptr, hipStream_t stream) {
    hipLaunchKernelGGL(unit_scale_kernel, dim3(1), dim3(1), 0, stream, gptr);
    return hipGetLastError();
}

hipError_t launch_quantize_rht(QuantOut out, const uint16_t *x, int64_t rows, int64_t cols, int64_t ldx,
                               uint32_t signs, uint8_t *codes, uint8_t *scales, uint16_t *y, int64_t ldy,
                               hipStream_t stream) {
    const int64_t total = rows * (cols / 32);
    if (total == 0) return hipSuccess;
    const int64_t nseg = (total + kSeg - 1) / kSeg;
    int64_t grid = (nseg + 4 * kSegPerWave - 1) / (4 * kSegPerWave);
    if (grid > kMaxGroups) grid = kMaxGroups;
    if (out == kCodes)
        hipLaunchKernelGGL(quantize_rht_kernel<kCodes>, dim3((unsigned)grid), dim3(kThreads), 0, stream, x, rows,
                           cols, ldx, signs, codes, scales, y, ldy);
    else
        hipLaunchKernelGGL(quantize_rht_kernel<kFakeQuant>, dim3((unsigned)grid), dim3(kThreads), 0, stream, x,
                           rows, cols, ldx, signs, codes, scales, y, ldy);
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
                           float *gptr, GSrc gsrc, uint32_t *partials, uint16_t *seg_table,
                           int64_t seg_capacity, hipStream_t stream) {
    const int B = fmt == kMX ? 32 : 16;
    const int64_t total = rows * (cols / B);
    if (total == 0) return hipSuccess;
    const int64_t nseg = (total + kSeg - 1) / kSeg;
    const bool nv = fmt == kNV;
    const bool local = nv && gsrc == kGComputed && total * B <= kLocalMaxElems;
    const bool deferred = !local && nv && gsrc == kGComputed && seg_table != nullptr && nseg <= seg_capacity;
    int nparts = 0;
    if (nv && gsrc == kGComputed && !deferred && !local) {
        hipError_t e = launch_absmax(x, rows, cols, ldx, partials, &nparts, stream);
        if (e != hipSuccess) return e;
    }
    // about kSegPerWave segments per wave, at most kMaxGroups workgroups
    int64_t grid = (nseg + 4 * kSegPerWave - 1) / (4 * kSegPerWave);
    if (grid > kMaxGroups) grid = kMaxGroups;
    if (grid < 1) grid = 1;
    // small tensor: one segment per wave (at most 16 workgroups, each reading
    // all of x for the amax) keeps each wave's chain of block arithmetic short
    if (local) grid = (nseg + 3) / 4;
    // one pass with a computed g writing fake-quant values (two segments per
    // step): four workgroups per CU, so each wave takes several steps and the
    // fix-up folds fewer partial maxima (21M-element X, codes and fake-quant:
    // 25.9 -> 23.2 us; the 141M-element W: 130.1 -> 129.2 us, fake-quant alone
    // 113.5 -> 112.1 us).  The codes-only pass keeps the larger grid (its
    // steps hold one segment, and fewer waves measured slower there).
    if (deferred && out != kCodes && grid > kMaxDeferredFqGroups) grid = kMaxDeferredFqGroups;
    if (deferred) nparts = (int)grid;
    hipError_t e;
    auto run = [&](auto fmt_c, auto out_c) {
        return launch_fmt_out<decltype(fmt_c)::value, decltype(out_c)::value>(
            gsrc, local, deferred, (int)grid, x, rows, cols, ldx, codes, scales, y, ldy, gptr, partials, nparts,
            seg_table, stream);
    };
    using MXc = std::integral_constant<int, kMX>;
    using NVc = std::integral_constant<int, kNV>;
    using Cc = std::integral_constant<int, kCodes>;
    using Fc = std::integral_constant<int, kFakeQuant>;
    using Bc = std::integral_constant<int, kBoth>;
    if (fmt == kMX)
        e = out == kCodes ? run(MXc{}, Cc{}) : out == kFakeQuant ? run(MXc{}, Fc{}) : run(MXc{}, Bc{});
    else
        e = out == kCodes ? run(NVc{}, Cc{}) : out == kFakeQuant ? run(NVc{}, Fc{}) : run(NVc{}, Bc{});
    if (e != hipSuccess || !deferred) return e;
    int64_t fgrid = (nseg + kThreads - 1) / kThreads;
    if (fgrid > kMaxGroups) fgrid = kMaxGroups;
    if (out == kCodes)
        hipLaunchKernelGGL(nv_fixup_kernel<kCodes>, dim3((unsigned)fgrid), dim3(kThreads), 0, stream, x, rows,
                           cols, ldx, codes, scales, y, ldy, gptr, partials, nparts, seg_table);
    else if (out == kFakeQuant)
        hipLaunchKernelGGL(nv_fixup_kernel<kFakeQuant>, dim3((unsigned)fgrid), dim3(kThreads), 0, stream, x, rows,
                           cols, ldx, codes, scales, y, ldy, gptr, partials, nparts, seg_table);
    else
        hipLaunchKernelGGL(nv_fixup_kernel<kBoth>, dim3((unsigned)fgrid), dim3(kThreads), 0, stream, x, rows,
                           cols, ldx, codes, scales, y, ldy, gptr, partials, nparts, seg_table);
    return hipGetLastError();
}

}  // namespace reqat
