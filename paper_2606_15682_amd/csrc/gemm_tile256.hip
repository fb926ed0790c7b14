// Large-tile W4A4 GEMM for gfx950.
//
// Workgroup tile 256 x 256, four waves of 128 x 128 (4 x 4 MFMA tiles of 32 x 32,
// 256 FP32 accumulators per lane, one wave per SIMD).  K advances KS elements
// per stage; each stage's packed codes (KS/2 bytes per row) and scale bytes go
// global -> LDS with direct-to-LDS loads (global_load_lds_dwordx4 / _dword)
// into a ring of NBUF stage buffers: the loads of stage st + NBUF - 1 are
// issued while stage st is multiplied, and the wait at the top of each stage
// counts only the loads of the stages still in flight behind it (vmcnt) and is
// followed by a bare s_barrier (no fence that would drain those loads).
//
// LDS code layout: one row = CH chunks of 16 B (32 E2M1 codes each); chunk c of
// row r is stored at chunk position c ^ f(r).  A wave's 16-byte operand read
// puts consecutive rows at the same logical chunk on consecutive lanes, and f
// spreads them: any 8 aligned consecutive rows land in 8 distinct 16-byte
// slots of a 128-byte bank window and any 16 aligned rows in 16 distinct slots
// of a 256-byte window, so the reads are free of bank conflicts for either 32
// or 64 four-byte banks.
//   CH = 8 (128-byte rows): f(r) = (r & 7) ^ ((r >> 3) & 1)
//   CH = 4 ( 64-byte rows): f(r) = ((r >> 1) & 3) ^ ((r >> 3) & 1)
// One direct-to-LDS instruction writes 1 KB contiguous, and each lane fetches
// whichever 16 global bytes belong at its LDS slot.
//
// MXFP4 (v_mfma_scale_f32_32x32x64_f8f6f4, E2M1 x E2M1): in substep s of a
// stage, lanes 0-31 feed 32-block s and lanes 32-63 feed 32-block KS/64 + s of
// their row; the lane's scale bytes for the stage sit in one dword and the
// instruction's op_sel picks byte s.  A and B use the same K assignment, so
// the sum over K is unchanged.  The next substep's operands are read from LDS
// before the current substep's MFMAs are issued.
//
// NVFP4 (v_mfma_f32_32x32x16_f16): per 64-element chunk a lane loads 32 codes
// (16 B) and the two E4M3 scale bytes of its two 16-blocks (one 16-bit LDS
// read).  v_cvt_scalef32_pk_f16_fp8 turns the two scale bytes into FP16 (every
// E4M3 value, subnormals and NaN included, is exact in FP16), and each step
// decodes 8 codes with v_cvt_scalef32_pk_f16_fp4 (unit scale) and multiplies
// them by their block's scale with v_pk_mul_f16 (op_sel picks the half).
// code * scale has <= 6 significant bits and lies in [2^-10, 2688], so the
// product is exact and the FP16 MFMA sums exactly the terms of the definition.
//
// Tile order: workgroups are dealt round-robin to the 8 XCDs, so workgroup b
// is mapped to the (b % 8)-th contiguous range of tiles, and tiles are walked
// in groups of 8 tile-rows, keeping the A and B panels a group reuses in the
// L2 of the XCD that owns it.
#include "fp4_device.h"
#include "internal.h"

#ifndef REQAT_MX_KS
#define REQAT_MX_KS 128
#endif
#ifndef REQAT_MX_NBUF
#define REQAT_MX_NBUF 4
#endif
#ifndef REQAT_NV_KS
#define REQAT_NV_KS 256
#endif
#ifndef REQAT_NV_NBUF
#define REQAT_NV_NBUF 2
#endif

namespace reqat {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kThreads = 256;
constexpr int TM = 256, TN = 256;
constexpr int GROUP_M = 8;

template <int FMT, int KS, int NBUF>
struct Cfg {
    static constexpr int B = FMT == kMX ? 32 : 16;
    static constexpr int ROW = KS / 2;                  // code bytes per row per stage
    static constexpr int CH = ROW / 16;                 // 16-byte chunks per row
    static constexpr int RPI = 1024 / ROW;              // rows per 1 KB load instruction
    static constexpr int CODE = TM * ROW;               // code bytes per operand per stage
    static constexpr int SB = KS / B;                   // scale bytes per row per stage
    static constexpr int SCALE = TM * SB;
    static constexpr int LS = SB >= 16 ? 16 : 4;        // bytes per lane of a scale load
    static constexpr int SRPI = 64 * LS / SB;           // rows per scale load instruction
    static constexpr int SINS = TM / SRPI;              // scale load instructions per operand
    static constexpr int A_CODES = 0, B_CODES = CODE;
    static constexpr int A_SC = 2 * CODE, B_SC = 2 * CODE + SCALE;
    static constexpr int STAGE = 2 * CODE + 2 * SCALE;
    static constexpr int TOTAL = NBUF * STAGE;
    static constexpr int CODE_LPW = (CODE / 1024) / 4;  // code loads per operand per wave
    static constexpr int SCALE_LPW = SINS / 4;          // scale loads per operand per wave
    static constexpr int LPS = 2 * CODE_LPW + 2 * SCALE_LPW;   // loads per wave per stage
    static_assert(CH == 4 || CH == 8, "row must be 4 or 8 chunks");
    static_assert(SINS % 4 == 0 && (CODE / 1024) % 4 == 0, "loads must split over 4 waves");
    static_assert(TOTAL <= 160 * 1024, "LDS budget");
};

__device__ __forceinline__ void g2l16(const void *g, uint8_t *l) {
    __builtin_amdgcn_global_load_lds(g, (lds_void *)l, 16, 0, 0);
}
__device__ __forceinline__ void g2l4(const void *g, uint8_t *l) {
    __builtin_amdgcn_global_load_lds(g, (lds_void *)l, 4, 0, 0);
}

__device__ __forceinline__ uint4 lds16(const uint8_t *p) { return *reinterpret_cast<const uint4 *>(p); }
__device__ __forceinline__ uint32_t lds4(const uint8_t *p) { return *reinterpret_cast<const uint32_t *>(p); }

template <int CH>
__device__ __forceinline__ int swz(int r) {
    return CH == 8 ? ((r & 7) ^ ((r >> 3) & 1)) : (((r >> 1) & 3) ^ ((r >> 3) & 1));
}

// Byte offset of logical 16-byte chunk c of tile row r.
template <int ROW>
__device__ __forceinline__ int code_off(int r, int c) {
    return r * ROW + ((c ^ swz<ROW / 16>(r)) << 4);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Load number IDX (0 .. LPS-1) of this wave's share of one stage.  a/b point at
// the first row of the tile and at the stage's first column; edge tiles clamp
// rows to the last valid one (those rows are loaded but never stored).
template <class C, int IDX>
__device__ __forceinline__ void load_one(uint8_t *buf, int wave, int lane, int rows_a, int rows_b,
                                         int64_t cpr, int64_t spr, const uint8_t *a_codes,
                                         const uint8_t *b_codes, const uint8_t *a_scales,
                                         const uint8_t *b_scales) {
    if constexpr (IDX < 2 * C::CODE_LPW) {
        constexpr bool isA = IDX < C::CODE_LPW;
        const int j = wave * C::CODE_LPW + (isA ? IDX : IDX - C::CODE_LPW);
        const int row = C::RPI * j + lane / C::CH;
        const int c = (lane % C::CH) ^ swz<C::CH>(row);
        const int lim = isA ? rows_a : rows_b;
        const int r = row < lim ? row : lim - 1;
        // 32-bit lane offset from a wave-uniform base (the launcher bounds 256 * K / 2 below 2^32)
        g2l16((isA ? a_codes : b_codes) + (uint32_t)(r * (uint32_t)cpr + c * 16),
              buf + (isA ? C::A_CODES : C::B_CODES) + j * 1024);
    } else {
        constexpr int k = IDX - 2 * C::CODE_LPW;
        constexpr bool isA = k < C::SCALE_LPW;
        const int j = wave * C::SCALE_LPW + (isA ? k : k - C::SCALE_LPW);
        constexpr int PPR = C::SB / C::LS;              // lanes per row
        const int row = C::SRPI * j + lane / PPR;
        const int piece = lane % PPR;
        const int lim = isA ? rows_a : rows_b;
        const int r = row < lim ? row : lim - 1;
        const uint8_t *src = (isA ? a_scales : b_scales) + (uint32_t)(r * (uint32_t)spr + piece * C::LS);
        uint8_t *dst = buf + (isA ? C::A_SC : C::B_SC) + j * (64 * C::LS);
        if constexpr (C::LS == 16) g2l16(src, dst);
        else g2l4(src, dst);
    }
}

// Loads [LO, HI) of this wave's share of one stage.
template <class C, int LO, int HI>
__device__ __forceinline__ void load_range(uint8_t *buf, int wave, int lane, int rows_a, int rows_b,
                                           int64_t cpr, int64_t spr, const uint8_t *ac,
                                           const uint8_t *bc, const uint8_t *as_, const uint8_t *bs_) {
    if constexpr (LO < HI) {
        load_one<C, LO>(buf, wave, lane, rows_a, rows_b, cpr, spr, ac, bc, as_, bs_);
        load_range<C, LO + 1, HI>(buf, wave, lane, rows_a, rows_b, cpr, spr, ac, bc, as_, bs_);
    }
}

// Issues the loads of one later stage in four parts (part P covers loads
// [P*LPS/4, (P+1)*LPS/4) of this wave's share), or nothing when no stage is left.
template <class C>
struct StageIssue {
    uint8_t *buf;
    bool active;
    int wave, lane, rows_a, rows_b;
    int64_t cpr, spr;
    const uint8_t *ac, *bc, *as_, *bs_;
    template <int P>
    __device__ __forceinline__ void part() { region<P, 4>(); }
    // Region R of NR: loads [R*LPS/NR, (R+1)*LPS/NR).
    template <int R, int NR>
    __device__ __forceinline__ void region() {
        if (active)
            load_range<C, R * C::LPS / NR, (R + 1) * C::LPS / NR>(buf, wave, lane, rows_a, rows_b, cpr,
                                                                   spr, ac, bc, as_, bs_);
    }
    template <int R, int NR>
    static constexpr int count() { return (R + 1) * C::LPS / NR - R * C::LPS / NR; }
};

__device__ __forceinline__ v8i as_v8i(uint4 q) {
    return v8i{(int)q.x, (int)q.y, (int)q.z, (int)q.w, 0, 0, 0, 0};
}

template <int S>
__device__ __forceinline__ void mx_mfma16(v16f (&acc)[4][4], const uint4 (&a)[4], const uint4 (&b)[4],
                                          const uint32_t (&sa)[4], const uint32_t (&sb)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                as_v8i(a[i]), as_v8i(b[j]), acc[i][j], 4, 4, S, (int)sa[i], S, (int)sb[j]);
}

// Eight codes (one dword) times an NVFP4 block scale (FP16, in both halves) -> FP16 (exact).
__device__ __forceinline__ v8h nv_decode8(uint32_t c, v2h s) {
    v2h p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 0) * s;
    v2h p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 1) * s;
    v2h p2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 2) * s;
    v2h p3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 3) * s;
    return v8h{p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

__device__ __forceinline__ uint32_t pick(const uint4 &q, int s) {
    return s == 0 ? q.x : s == 1 ? q.y : s == 2 ? q.z : q.w;
}

// MXFP4: one stage from LDS buffer `buf`, with the loads of a later stage
// issued in parts between the substeps.
template <class C, class Issue>
__device__ __forceinline__ void mx_stage(v16f (&acc)[4][4], const uint8_t *buf, int rA0, int rB0,
                                         int h, Issue &issue) {
    constexpr int NSUB = C::CH / 2;                     // K=64 substeps per stage
    uint32_t sa[4], sb[4];
    uint4 a0[4], b0[4], a1[4], b1[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int ra = rA0 + 32 * i, rb = rB0 + 32 * i;
        if constexpr (C::SB == 8) {
            sa[i] = lds4(buf + C::A_SC + ra * 8 + 4 * h);
            sb[i] = lds4(buf + C::B_SC + rb * 8 + 4 * h);
        } else {
            sa[i] = lds4(buf + C::A_SC + ra * 4) >> (16 * h);
            sb[i] = lds4(buf + C::B_SC + rb * 4) >> (16 * h);
        }
        a0[i] = lds16(buf + C::A_CODES + code_off<C::ROW>(ra, NSUB * h));
        b0[i] = lds16(buf + C::B_CODES + code_off<C::ROW>(rb, NSUB * h));
    }
#define REQAT_MX_READ(A, B, S)                                                           \
    _Pragma("unroll") for (int i = 0; i < 4; ++i) {                                      \
        A[i] = lds16(buf + C::A_CODES + code_off<C::ROW>(rA0 + 32 * i, NSUB * h + (S))); \
        B[i] = lds16(buf + C::B_CODES + code_off<C::ROW>(rB0 + 32 * i, NSUB * h + (S))); \
    }
    REQAT_MX_READ(a1, b1, 1);
    issue.template part<0>();
    __builtin_amdgcn_sched_barrier(0);
    mx_mfma16<0>(acc, a0, b0, sa, sb);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (NSUB == 4) {
        REQAT_MX_READ(a0, b0, 2);
        issue.template part<1>();
        __builtin_amdgcn_sched_barrier(0);
        mx_mfma16<1>(acc, a1, b1, sa, sb);
        __builtin_amdgcn_sched_barrier(0);
        REQAT_MX_READ(a1, b1, 3);
        issue.template part<2>();
        __builtin_amdgcn_sched_barrier(0);
        mx_mfma16<2>(acc, a0, b0, sa, sb);
        __builtin_amdgcn_sched_barrier(0);
        issue.template part<3>();
        __builtin_amdgcn_sched_barrier(0);
        mx_mfma16<3>(acc, a1, b1, sa, sb);
    } else {
        issue.template part<1>();
        issue.template part<2>();
        issue.template part<3>();
        __builtin_amdgcn_sched_barrier(0);
        mx_mfma16<1>(acc, a1, b1, sa, sb);
    }
#undef REQAT_MX_READ
}

// NVFP4: one stage from LDS buffer `buf`, software-pipelined by MFMA step.
// K assignment: a stage's row holds 2*NQ units of 32 codes (16 B, two
// 16-blocks each); in chunk q (64 elements) lane half h takes unit NQ*h + q,
// so over the stage a lane half covers one contiguous half of the row and
// its 2*NQ scale bytes are contiguous too (one 4- or 8-byte LDS read per tile
// and stage; chunk q's pair is 16-bit word q of them).  A and B use the same
// assignment, so the sum over K is unchanged.
// A step is one 16-element slice of K for all 4 x 4 tiles of the wave: 16
// MFMAs fed by 8 decoded operands (4 A tiles, 4 B tiles; 8 VALU each).  The
// operands of step t+1 are decoded while the MFMAs of step t run, and
// sched_group_barrier interleaves them as one MFMA then four VALU, so the
// decode hides under the matrix pipe.  Chunk q+1's codes are read from LDS in
// the first step of chunk q and its scales converted in the third.
template <class C>
struct NvLane {
    static constexpr int NQ = C::CH / 2;
    int codeA[NQ], codeB[NQ];                           // byte offset of this lane's unit in chunk q (tile 0)
    int scA, scB;                                       // byte offset of this lane's scale bytes (tile 0)
    __device__ __forceinline__ NvLane(int rA0, int rB0, int h) {
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            codeA[q] = C::A_CODES + code_off<C::ROW>(rA0, NQ * h + q);
            codeB[q] = C::B_CODES + code_off<C::ROW>(rB0, NQ * h + q);
        }
        scA = C::A_SC + rA0 * C::SB + NQ * 2 * h;
        scB = C::B_SC + rB0 * C::SB + NQ * 2 * h;
    }
};

template <class C>
struct NvState {
    static constexpr int NW = C::CH / 4;                // scale dwords per tile and stage
    uint4 ca[2][4], cb[2][4];                           // codes of chunks q (even/odd)
    uint32_t wa[4][NW], wb[4][NW];                      // this stage's scale bytes
    v2h sa[2][4], sb[2][4];                             // FP16 scales of chunk q's two 16-blocks
    v8h av[2][4], bv[2][4];                             // decoded operands of steps t (even/odd)
};

template <class C, int Q, int D>
__device__ __forceinline__ void nv_read_codes(NvState<C> &st, const uint8_t *buf, const NvLane<C> &ln) {
    const uint8_t *pa = buf + ln.codeA[Q], *pb = buf + ln.codeB[Q];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        st.ca[D][i] = lds16(pa + 32 * C::ROW * i);
        st.cb[D][i] = lds16(pb + 32 * C::ROW * i);
    }
}

template <class C>
__device__ __forceinline__ void nv_read_scales(NvState<C> &st, const uint8_t *buf, const NvLane<C> &ln) {
    const uint8_t *pa = buf + ln.scA, *pb = buf + ln.scB;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if constexpr (NvState<C>::NW == 2) {
            const uint2 x = *reinterpret_cast<const uint2 *>(pa + 32 * C::SB * i);
            const uint2 y = *reinterpret_cast<const uint2 *>(pb + 32 * C::SB * i);
            st.wa[i][0] = x.x; st.wa[i][1] = x.y;
            st.wb[i][0] = y.x; st.wb[i][1] = y.y;
        } else {
            st.wa[i][0] = lds4(pa + 32 * C::SB * i);
            st.wb[i][0] = lds4(pb + 32 * C::SB * i);
        }
    }
}

template <class C, int Q, int D>
__device__ __forceinline__ void nv_scales(NvState<C> &st) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        st.sa[D][i] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(st.wa[i][Q >> 1], 1.0f, (Q & 1) != 0);
        st.sb[D][i] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(st.wb[i][Q >> 1], 1.0f, (Q & 1) != 0);
    }
}

template <class C, int T>
__device__ __forceinline__ void nv_decode(NvState<C> &st) {
    constexpr int D = (T >> 2) & 1, S = T & 3, HB = S >> 1, E = T & 1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        st.av[E][i] = nv_decode8(pick(st.ca[D][i], S), __builtin_shufflevector(st.sa[D][i], st.sa[D][i], HB, HB));
        st.bv[E][i] = nv_decode8(pick(st.cb[D][i], S), __builtin_shufflevector(st.sb[D][i], st.sb[D][i], HB, HB));
    }
}

template <class C, int T, int NT, class Issue>
__device__ __forceinline__ void nv_region(v16f (&acc)[4][4], NvState<C> &st, const uint8_t *buf,
                                          const NvLane<C> &ln, Issue &issue) {
    constexpr int NQ = NT / 4, Q = T >> 2, S = T & 3, E = T & 1;
    constexpr bool READ = S == 0 && Q + 1 < NQ;
    constexpr int ND = READ ? 8 : 0;                    // LDS reads in this region
    // the next stage's loads go out in the first half of the stage
    constexpr int NG = T < NT / 2 ? Issue::template count<T, NT / 2>() : 0;
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (READ) nv_read_codes<C, Q + 1, (Q + 1) & 1>(st, buf, ln);
    if constexpr (S == 2 && Q + 1 < NQ) nv_scales<C, Q + 1, (Q + 1) & 1>(st);
    if constexpr (T < NT / 2) issue.template region<T, NT / 2>();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(st.av[E][i], st.bv[E][j], acc[i][j], 0, 0, 0);
    if constexpr (T + 1 < NT) nv_decode<C, T + 1>(st);
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // one MFMA
        if (T + 1 < NT) __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);   // four VALU
        if (k < ND) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);       // one LDS read
        if (k < NG) __builtin_amdgcn_sched_group_barrier(0x010, 1, 0);       // one global load
    }
    if constexpr (T + 1 < NT) {
        // pin the decoded operands to this region (otherwise they are sunk next to their MFMAs)
#pragma unroll
        for (int i = 0; i < 4; ++i) asm volatile("" : "+v"(st.av[E ^ 1][i]), "+v"(st.bv[E ^ 1][i]));
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (T + 1 < NT) nv_region<C, T + 1, NT>(acc, st, buf, ln, issue);
}

template <class C, class Issue>
__device__ __forceinline__ void nv_stage(v16f (&acc)[4][4], const uint8_t *buf, const NvLane<C> &ln,
                                         Issue &issue) {
    constexpr int NT = 2 * C::CH;                       // 16-element steps per stage
    NvState<C> st;
    nv_read_codes<C, 0, 0>(st, buf, ln);
    nv_read_scales<C>(st, buf, ln);
    nv_scales<C, 0, 0>(st);
    nv_decode<C, 0>(st);
    nv_region<C, 0, NT>(acc, st, buf, ln, issue);
}

template <int FMT, int KS, int NBUF>
__global__ __launch_bounds__(kThreads, 1) void gemm_tile256_kernel(
    int64_t M, int64_t N, int64_t K, const uint8_t *__restrict__ a_codes,
    const uint8_t *__restrict__ a_scales, const float *__restrict__ ga,
    const uint8_t *__restrict__ b_codes, const uint8_t *__restrict__ b_scales,
    const float *__restrict__ gb, void *__restrict__ y, int y_bf16, int64_t ldy) {
    using C = Cfg<FMT, KS, NBUF>;
    extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int h = lane >> 5;
    const int wm = wave >> 1, wn = wave & 1;

    // ---- tile order: XCD-contiguous ranges, then groups of GROUP_M tile-rows
    const int64_t tm_n = (M + TM - 1) / TM, tn_n = (N + TN - 1) / TN, T = tm_n * tn_n;
    const int64_t bid = blockIdx.x;
    const int64_t xcd = bid % 8, local = bid / 8, per = T / 8, rem = T % 8;
    const int64_t t = xcd * per + (xcd < rem ? xcd : rem) + local;
    const int64_t width = GROUP_M * tn_n;
    const int64_t first_m = (t / width) * GROUP_M;
    const int64_t gsz = (tm_n - first_m) < GROUP_M ? (tm_n - first_m) : GROUP_M;
    const int64_t tm = first_m + (t % width) % gsz, tn = (t % width) / gsz;
    const int64_t m0 = tm * TM, n0 = tn * TN;
    const int64_t cpr = K / 2, spr = K / C::B;

    v16f acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    const int nst = (int)(K / KS);
    const int rows_a = (int)(M - m0 < TM ? M - m0 : TM), rows_b = (int)(N - n0 < TN ? N - n0 : TN);
    const uint8_t *ac = a_codes + m0 * cpr, *bc = b_codes + n0 * cpr;
    const uint8_t *as_ = a_scales + m0 * spr, *bs_ = b_scales + n0 * spr;

    // prologue: the first NBUF - 1 stages
#pragma unroll
    for (int p = 0; p < NBUF - 1; ++p) {
        if (p < nst)
            load_range<C, 0, C::LPS>(smem + p * C::STAGE, wave, lane, rows_a, rows_b, cpr, spr,
                                     ac + (int64_t)p * KS / 2, bc + (int64_t)p * KS / 2,
                                     as_ + (int64_t)p * KS / C::B, bs_ + (int64_t)p * KS / C::B);
    }

    const int rA0 = wm * 128 + (lane & 31);               // this lane's A row in tile i: rA0 + 32 i
    const int rB0 = wn * 128 + (lane & 31);
    const NvLane<C> nvl(rA0, rB0, h);

    for (int st = 0; st < nst; ++st) {
        // stage st has landed once no more than (stages issued after it) x LPS loads remain
        const int behind = (nst - 1 - st) < (NBUF - 2) ? (nst - 1 - st) : (NBUF - 2);
        if (NBUF >= 3 && behind == NBUF - 2) wait_vmcnt<(NBUF >= 3 ? NBUF - 2 : 0) * C::LPS>();
        else if (NBUF >= 4 && behind == 1) wait_vmcnt<C::LPS>();
        else wait_vmcnt<0>();
        // A bare barrier: __syncthreads() would also drain every load still in
        // flight for later stages.  This wave's loads of stage st are done (vmcnt
        // above) and its LDS reads of the buffer about to be refilled are done
        // (lgkmcnt), so after the barrier stage st is complete for every wave.
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");

        const uint8_t *buf = smem + (st % NBUF) * C::STAGE;
        const int nx = st + NBUF - 1;                      // stage whose loads go out now
        const int64_t kx = (int64_t)nx * KS;
        StageIssue<C> issue{smem + (nx % NBUF) * C::STAGE, nx < nst, wave, lane, rows_a, rows_b,
                            cpr, spr, ac + kx / 2, bc + kx / 2, as_ + kx / C::B, bs_ + kx / C::B};
        if constexpr (FMT == kMX) {
            mx_stage<C>(acc, buf, rA0, rB0, h, issue);
        } else {
            nv_stage<C>(acc, buf, nvl, issue);
        }
    }

    // ---- epilogue: D[i][j] of a 32 x 32 tile is in lane j + 32*((i/4)%2), register (i/8)*4 + i%4
    float scale = 1.0f;
    if (FMT == kNV) scale = (*ga) * (*gb);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t gn = n0 + wn * 128 + j * 32 + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t gm = m0 + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
                if (gm < M && gn < N) {
                    const float v = acc[i][j][r] * scale;
                    if (y_bf16)
                        reinterpret_cast<uint16_t *>(y)[gm * ldy + gn] = (uint16_t)bf16_rne_from_float(v);
                    else
                        reinterpret_cast<float *>(y)[gm * ldy + gn] = v;
                }
            }
        }
}

template <int FMT, int KS, int NBUF>
hipError_t launch_cfg(int64_t M, int64_t N, int64_t K, const uint8_t *a_codes, const uint8_t *a_scales,
                      const float *ga, const uint8_t *b_codes, const uint8_t *b_scales,
                      const float *gb, void *y, bool y_bf16, int64_t ldy, hipStream_t stream) {
    const int64_t tiles = ((M + TM - 1) / TM) * ((N + TN - 1) / TN);
    const size_t lds = Cfg<FMT, KS, NBUF>::TOTAL;
    hipError_t e = hipFuncSetAttribute((const void *)gemm_tile256_kernel<FMT, KS, NBUF>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((gemm_tile256_kernel<FMT, KS, NBUF>), dim3((unsigned)tiles), dim3(kThreads), lds,
                       stream, M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, (int)y_bf16,
                       ldy);
    return hipGetLastError();
}

}  // namespace

bool gemm_tile256_supported(Fmt fmt, int64_t M, int64_t N, int64_t K) {
    const int ks = fmt == kMX ? REQAT_MX_KS : REQAT_NV_KS;
    // lane offsets into a tile's rows are 32-bit: 256 rows * K/2 bytes < 2^32
    return K > 0 && K % ks == 0 && M > 0 && N > 0 && K <= (int64_t(1) << 24);
}

hipError_t launch_gemm_tile256(Fmt fmt, int64_t M, int64_t N, int64_t K, const uint8_t *a_codes,
                               const uint8_t *a_scales, const float *ga, const uint8_t *b_codes,
                               const uint8_t *b_scales, const float *gb, void *y, bool y_bf16,
                               int64_t ldy, hipStream_t stream) {
    if (fmt == kMX)
        return launch_cfg<kMX, REQAT_MX_KS, REQAT_MX_NBUF>(M, N, K, a_codes, a_scales, ga, b_codes,
                                                           b_scales, gb, y, y_bf16, ldy, stream);
    return launch_cfg<kNV, REQAT_NV_KS, REQAT_NV_NBUF>(M, N, K, a_codes, a_scales, ga, b_codes,
                                                       b_scales, gb, y, y_bf16, ldy, stream);
}

}  // namespace reqat
