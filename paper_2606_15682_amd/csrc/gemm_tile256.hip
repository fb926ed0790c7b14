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
// The direct-to-LDS loads of a CU are bound by how many distinct cache lines
// they touch, not by their bytes (measured on gfx950: sixteen 64-byte row
// pieces per instruction ran at about 60% of the rate of eight whole 128-byte
// lines).  So MXFP4 with K % 512 == 0 (and 16-byte aligned scales) runs
// K = 256 per stage in two buffers, each code row a whole line per stage, and
// keeps its scale bytes out of the stages: 16 bytes per row (two stages) go
// to LDS in one 1 KB load per 64 rows, into a ring of two group buffers
// (loaded per stage, 4 bytes per row, they touched one line per 4 bytes).
// Other MXFP4 shapes run K = 128 per stage in four buffers.
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
#include <type_traits>

#include "fp4_device.h"
#include "internal.h"

// MXFP4 stages: with scale groups (K % 512 == 0), K = 256 per stage in two
// buffers (each code row a whole 128-byte line per stage); otherwise K = 128
// in four buffers.
#ifndef REQAT_MX_KS
#define REQAT_MX_KS 128
#endif
#ifndef REQAT_MX_NBUF
#define REQAT_MX_NBUF 4
#endif
#ifndef REQAT_MX_GS_KS
#define REQAT_MX_GS_KS 256
#endif
#ifndef REQAT_MX_GS_NBUF
#define REQAT_MX_GS_NBUF 2
#endif
#ifndef REQAT_NV_KS
#define REQAT_NV_KS 256
#endif
#ifndef REQAT_NV_NBUF
#define REQAT_NV_NBUF 2
#endif
#ifndef REQAT_NV_LEAD
#define REQAT_NV_LEAD 3
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

// Calls f(integral_constant<int, J>) for J = B .. E-1, unrolled at compile time.
template <int B, int E, typename F> __device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}
constexpr int GROUP_M = 8;

// GS (MXFP4 with K % 512 == 0 and 16-byte aligned scales): the scale bytes
// are not part of the stage; they go to LDS 16 bytes per row at a time (two
// stages of K = 256: one 1 KB load per 64 rows), into a ring of two group
// buffers.  Loading a stage's 8 bytes per row would touch one cache line per
// row for every 8 bytes, and the vector memory path of a CU is bound by the
// number of distinct cache lines its loads touch, not by their bytes.
template <int FMT, int KS, int NBUF, bool GS = false>
struct Cfg {
    static constexpr bool kGS = GS;
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
    static constexpr int STAGE = GS ? 2 * CODE : 2 * CODE + 2 * SCALE;
    static constexpr int GSTAGES = SB <= 16 ? 16 / SB : 1;   // stages per scale group: 16 bytes per row (GS)
    static constexpr int GROW = GSTAGES * SB;           // scale bytes per row per group (GS)
    static constexpr int GROUP = 2 * TM * GROW;         // bytes of a scale group buffer: A rows, then B rows
    static constexpr int SC_RING = NBUF * STAGE;        // offset of the two scale group buffers (GS)
    static constexpr int TOTAL = NBUF * STAGE + (GS ? 2 * GROUP : 0);
    static constexpr int CODE_LPW = (CODE / 1024) / 4;  // code loads per operand per wave
    static constexpr int SCALE_LPW = SINS / 4;          // scale loads per operand per wave
    static constexpr int LPS = 2 * CODE_LPW + (GS ? 0 : 2 * SCALE_LPW);   // loads per wave per stage
    static constexpr int GLPW = GS ? (GROUP / 1024) / 4 : 0;              // scale-group loads per wave
    static_assert(CH == 4 || CH == 8, "row must be 4 or 8 chunks");
    static_assert(SINS % 4 == 0 && (CODE / 1024) % 4 == 0, "loads must split over 4 waves");
    static_assert(TOTAL <= 160 * 1024, "LDS budget");
    static_assert(!GS || (FMT == kMX && GROW == 16 && GLPW == 2 && GSTAGES >= 2),
                  "scale groups: 16 bytes per row, 2 loads per wave");
};

// Direct-to-LDS loads: lane i's 16 (4) bytes at base + voff land at LDS
// address l + 16 i (4 i); base and l are wave-uniform.  Written as inline asm
// so the compiler does not track them: it would otherwise wait for every
// such load in flight (vmcnt(0)) before any later LDS read, since it cannot
// tell which stage buffer a read touches.  The kernels order these writes
// against their LDS reads themselves (vmcnt waits and barriers).
__device__ __forceinline__ void g2l16(const uint8_t *base, uint32_t voff, uint8_t *l) {
    asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "{m0}"((uint32_t)(uintptr_t)l));
}
__device__ __forceinline__ void g2l4(const uint8_t *base, uint32_t voff, uint8_t *l) {
    asm volatile("global_load_lds_dword %0, %1" ::"v"(voff), "s"(base), "{m0}"((uint32_t)(uintptr_t)l));
}

// A float read through the scalar cache (the pointer is uniform).
__device__ __forceinline__ float uniform_load(const float *p) {
    return *(const __attribute__((address_space(4))) float *)p;
}

__device__ __forceinline__ uint4 lds16(const uint8_t *p) { return *reinterpret_cast<const uint4 *>(p); }

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
        g2l16(isA ? a_codes : b_codes, (uint32_t)(r * (uint32_t)cpr + c * 16),
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
        const uint8_t *src = isA ? a_scales : b_scales;
        const uint32_t off = (uint32_t)(r * (uint32_t)spr + piece * C::LS);
        uint8_t *dst = buf + (isA ? C::A_SC : C::B_SC) + j * (64 * C::LS);
        if constexpr (C::LS == 16) g2l16(src, off, dst);
        else g2l4(src, off, dst);
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
__device__ __forceinline__ void nv_read_codes1(NvState<C> &st, const uint8_t *buf, const NvLane<C> &ln, int i) {
    st.ca[D][i] = lds16(buf + ln.codeA[Q] + 32 * C::ROW * i);
    st.cb[D][i] = lds16(buf + ln.codeB[Q] + 32 * C::ROW * i);
}

template <class C>
__device__ __forceinline__ void nv_read_scales1(NvState<C> &st, const uint8_t *buf, const NvLane<C> &ln, int i) {
    if constexpr (NvState<C>::NW == 2) {
        const uint2 x = *reinterpret_cast<const uint2 *>(buf + ln.scA + 32 * C::SB * i);
        const uint2 y = *reinterpret_cast<const uint2 *>(buf + ln.scB + 32 * C::SB * i);
        st.wa[i][0] = x.x; st.wa[i][1] = x.y;
        st.wb[i][0] = y.x; st.wb[i][1] = y.y;
    } else {
        st.wa[i][0] = lds4(buf + ln.scA + 32 * C::SB * i);
        st.wb[i][0] = lds4(buf + ln.scB + 32 * C::SB * i);
    }
}

template <class C, int Q, int D>
__device__ __forceinline__ void nv_scales1(NvState<C> &st, int i) {
    st.sa[D][i] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(st.wa[i][Q >> 1], 1.0f, (Q & 1) != 0);
    st.sb[D][i] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(st.wb[i][Q >> 1], 1.0f, (Q & 1) != 0);
}

// Decodes step T's operands of A tile i and B tile i.
template <class C, int T>
__device__ __forceinline__ void nv_decode1(NvState<C> &st, int i) {
    constexpr int D = (T >> 2) & 1, S = T & 3, HB = S >> 1, E = T & 1;
    st.av[E][i] = nv_decode8(pick(st.ca[D][i], S), __builtin_shufflevector(st.sa[D][i], st.sa[D][i], HB, HB));
    st.bv[E][i] = nv_decode8(pick(st.cb[D][i], S), __builtin_shufflevector(st.sb[D][i], st.sb[D][i], HB, HB));
}

// Region T of a stage (NT regions; buffer `buf`, next stage in `nbuf`), in
// four fenced parts: part k issues the MFMAs of A tile k (4) and decodes A
// tile k and B tile k for step T + 1 (16 VALU), one MFMA to four VALU, plus
// its share of LDS reads and loads.  The stage's LDS reads all happen by
// region NT-4; at its end the wave waits for its loads of the next stage and
// meets the others at a barrier.  Past that point every wave is done with
// `buf`, so regions NT-3 .. NT-1 issue the loads of stage + 2 into it, read
// the next stage's first chunk and scales from `nbuf`, and decode its first
// step: the next stage starts with its operands ready.
template <class C, int T, int NT, int K, class Issue>
__device__ __forceinline__ void nv_part(v16f (&acc)[4][4], NvState<C> &st, const uint8_t *buf,
                                        const uint8_t *nbuf, const NvLane<C> &ln, Issue &issue) {
    constexpr int NQ = NT / 4, Q = T >> 2, S = T & 3, E = T & 1;
    constexpr bool READ = S == 0 && Q + 1 < NQ;
    constexpr int L = REQAT_NV_LEAD;                    // regions after the stage's barrier
    static_assert(L >= 3 && L <= 5, "the barrier follows chunk NQ-1's reads and conversions");
    constexpr bool NEXT_READ = T == NT - L, NEXT_CVT = T == NT - L + 1;
    constexpr int LP = (T - (NT - L)) * 4 + K;          // load part (0..4L-1) in the last L regions
    constexpr int NG = LP >= 0 ? Issue::template count<(LP >= 0 ? LP : 0), 4 * L>() : 0;
    constexpr int ND = READ ? 2 : NEXT_READ ? 4 : 0;    // LDS reads in this part
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (READ) nv_read_codes1<C, Q + 1, (Q + 1) & 1>(st, buf, ln, K);
    if constexpr (S == 2 && Q + 1 < NQ) nv_scales1<C, Q + 1, (Q + 1) & 1>(st, K);
    if constexpr (NEXT_READ) {
        nv_read_codes1<C, 0, 0>(st, nbuf, ln, K);
        nv_read_scales1<C>(st, nbuf, ln, K);
    }
    if constexpr (NEXT_CVT) nv_scales1<C, 0, 0>(st, K);
    if constexpr (LP >= 0) issue.template region<(LP >= 0 ? LP : 0), 4 * L>();
#pragma unroll
    for (int j = 0; j < 4; ++j)
        acc[K][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(st.av[E][K], st.bv[E][j], acc[K][j], 0, 0, 0);
    nv_decode1<C, T + 1>(st, K);                        // T + 1 == NT: the next stage's step 0
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);     // four VALU
        if (k < ND) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);       // one LDS read
    }
    if (NG > 0) __builtin_amdgcn_sched_group_barrier(0x010, NG, 0);          // the part's loads
    // pin the decoded operands to this part (otherwise they are sunk next to their MFMAs)
    asm volatile("" : "+v"(st.av[E ^ 1][K]), "+v"(st.bv[E ^ 1][K]));
    __builtin_amdgcn_sched_barrier(0);
}

template <class C, int T, int NT, class Issue>
__device__ __forceinline__ void nv_region(v16f (&acc)[4][4], NvState<C> &st, const uint8_t *buf,
                                          const uint8_t *nbuf, const NvLane<C> &ln, Issue &issue) {
    nv_part<C, T, NT, 0>(acc, st, buf, nbuf, ln, issue);
    nv_part<C, T, NT, 1>(acc, st, buf, nbuf, ln, issue);
    nv_part<C, T, NT, 2>(acc, st, buf, nbuf, ln, issue);
    nv_part<C, T, NT, 3>(acc, st, buf, nbuf, ln, issue);
    if constexpr (T == NT - REQAT_NV_LEAD - 1) {
        // this wave's loads of the next stage have landed and its reads of `buf`
        // are done; after the barrier both hold for every wave
        asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    }
    if constexpr (T + 1 < NT) nv_region<C, T + 1, NT>(acc, st, buf, nbuf, ln, issue);
}

// Output tile of virtual tile id v: workgroups are dealt round-robin to the 8
// XCDs, so id v is mapped into the (v % 8)-th contiguous range of tiles, and
// tiles are walked in groups of GROUP_M tile-rows, keeping the A and B panels
// a group reuses in the L2 of the XCD that owns it.  With a persistent grid
// of G workgroups (G a multiple of 8), workgroup w takes ids w, w + G, ...,
// which stay on its XCD and walk that XCD's range in order.
struct TileGeo {
    int64_t m0, n0;
    int rows_a, rows_b;
};

__device__ __forceinline__ TileGeo tile_geo(int64_t v, int64_t M, int64_t N) {
    const int64_t tm_n = (M + TM - 1) / TM, tn_n = (N + TN - 1) / TN, T = tm_n * tn_n;
    const int64_t xcd = v % 8, local = v / 8, per = T / 8, rem = T % 8;
    const int64_t t = xcd * per + (xcd < rem ? xcd : rem) + local;
    const int64_t width = GROUP_M * tn_n;
    const int64_t first_m = (t / width) * GROUP_M;
    const int64_t gsz = (tm_n - first_m) < GROUP_M ? (tm_n - first_m) : GROUP_M;
    const int64_t tm = first_m + (t % width) % gsz, tn = (t % width) / gsz;
    TileGeo g;
    g.m0 = tm * TM;
    g.n0 = tn * TN;
    g.rows_a = (int)(M - g.m0 < TM ? M - g.m0 : TM);
    g.rows_b = (int)(N - g.n0 < TN ? N - g.n0 : TN);
    return g;
}

// Stores the wave's 128 x 128 block of a finished tile (times `scale`).
// D[i][j] of a 32 x 32 MFMA tile is in lane j + 32*((i/4)%2), register (i/8)*4 + i%4:
// a row base per (i, register) is wave-uniform and the lane adds a 32-bit
// offset (the launcher bounds ldy), so each store needs no address VALU.
template <bool BF16, bool FULL>
__device__ __forceinline__ void store_tile_as(const v16f (&acc)[4][4], const TileGeo &g, int64_t M, int64_t N,
                                              int wm, int wn, int lane, float scale, void *y, int64_t ldy) {
    typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
    constexpr int ES = BF16 ? 2 : 4;
    const int h = lane >> 5;
    const int64_t row0 = g.m0 + wm * 128, col0 = g.n0 + wn * 128;
    const uint32_t voff = (uint32_t)((4 * h) * ldy + (lane & 31)) * ES;
    const int lrow = 4 * h, lcol = lane & 31;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
            // registers r and r + 1 are consecutive rows of the same column
            const int ro = i * 32 + 8 * (r >> 2) + (r & 3);
            uint8_t *p0 = reinterpret_cast<uint8_t *>(y) + ((row0 + ro) * ldy + col0) * ES;
            uint8_t *p1 = p0 + ldy * ES;
            const bool r0 = FULL || row0 + ro + lrow < M, r1 = FULL || row0 + ro + lrow + 1 < M;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                float v0 = acc[i][j][r], v1 = acc[i][j][r + 1];
                // keep each pair's copy out of the accumulators next to its store
                asm volatile("" : "+v"(v0), "+v"(v1));
                v0 *= scale;
                v1 *= scale;
                const bool c = FULL || col0 + 32 * j + lcol < N;
                if (BF16) {
                    const v2bf b = {(__bf16)v0, (__bf16)v1};
                    const uint32_t u = __builtin_bit_cast(uint32_t, b);
                    if (r0 && c) *reinterpret_cast<uint16_t *>(p0 + voff + 32 * ES * j) = (uint16_t)u;
                    if (r1 && c) *reinterpret_cast<uint16_t *>(p1 + voff + 32 * ES * j) = (uint16_t)(u >> 16);
                } else {
                    if (r0 && c) *reinterpret_cast<float *>(p0 + voff + 32 * ES * j) = v0;
                    if (r1 && c) *reinterpret_cast<float *>(p1 + voff + 32 * ES * j) = v1;
                }
            }
        }
}

__device__ __forceinline__ void store_tile(const v16f (&acc)[4][4], const TileGeo &g, int64_t M, int64_t N,
                                           int wm, int wn, int lane, float scale, void *y, int y_bf16,
                                           int64_t ldy) {
    const bool full = g.rows_a == TM && g.rows_b == TN;
    if (y_bf16) {
        if (full) store_tile_as<true, true>(acc, g, M, N, wm, wn, lane, scale, y, ldy);
        else store_tile_as<true, false>(acc, g, M, N, wm, wn, lane, scale, y, ldy);
    } else {
        if (full) store_tile_as<false, true>(acc, g, M, N, wm, wn, lane, scale, y, ldy);
        else store_tile_as<false, false>(acc, g, M, N, wm, wn, lane, scale, y, ldy);
    }
}

// Position of the load stream: stage s of virtual tile v (the mapping is
// evaluated only for tiles that exist: past the last one its group size
// would be zero).
template <class C>
struct LoadPos {
    int64_t v;
    int s;
    TileGeo g;
    __device__ __forceinline__ void advance(int nst, int64_t G, int64_t M, int64_t N, int64_t T) {
        if (++s == nst) {
            s = 0;
            v += G;
            if (v < T) g = tile_geo(v, M, N);
        }
    }
};

// NVFP4, persistent: the workgroup runs the stages of all its tiles as one
// stream over two stage buffers (stage g in buffer g % 2; stages 0 and 1 are
// loaded up front and stage g + 2 during stage g), so the next tile's first
// stages are loaded, and its first step decoded, while the current tile ends;
// a finished tile is stored and its accumulators cleared between two stages.
template <class C>
__device__ __forceinline__ void nv_persistent(uint8_t *smem, int64_t M, int64_t N, int64_t K,
                                              const uint8_t *a_codes, const uint8_t *a_scales, float scale,
                                              const uint8_t *b_codes, const uint8_t *b_scales, void *y,
                                              int y_bf16, int64_t ldy, int wave, int lane) {
    constexpr int KS = 2 * C::ROW, NT = 2 * C::CH;
    static_assert(C::TOTAL == 2 * C::STAGE, "two stage buffers");
    const int h = lane >> 5, wm = wave >> 1, wn = wave & 1;
    const int64_t tm_n = (M + TM - 1) / TM, tn_n = (N + TN - 1) / TN, T = tm_n * tn_n;
    const int64_t G = gridDim.x, w = blockIdx.x;
    const int nst = (int)(K / KS);
    const int64_t cpr = K / 2, spr = K / C::B;
    const int64_t total = ((T - w + G - 1) / G) * nst;  // stages this workgroup runs (grid <= T)

    auto issue_at = [&](const LoadPos<C> &p, uint8_t *buf) {
        const int64_t k0 = (int64_t)p.s * KS;
        return StageIssue<C>{buf, p.v < T, wave, lane, p.g.rows_a, p.g.rows_b, cpr, spr,
                             a_codes + p.g.m0 * cpr + k0 / 2, b_codes + p.g.n0 * cpr + k0 / 2,
                             a_scales + p.g.m0 * spr + k0 / C::B, b_scales + p.g.n0 * spr + k0 / C::B};
    };

    LoadPos<C> ld{w, 0, tile_geo(w, M, N)};
    {
        StageIssue<C> i0 = issue_at(ld, smem);
        i0.template region<0, 1>();
        ld.advance(nst, G, M, N, T);
        StageIssue<C> i1 = issue_at(ld, smem + C::STAGE);
        i1.template region<0, 1>();
        ld.advance(nst, G, M, N, T);
        if (total > 1) wait_vmcnt<C::LPS>();
        else wait_vmcnt<0>();
    }
    asm volatile("s_barrier" ::: "memory");

    const NvLane<C> ln(wm * 128 + (lane & 31), wn * 128 + (lane & 31), h);
    NvState<C> st;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        nv_read_codes1<C, 0, 0>(st, smem, ln, i);
        nv_read_scales1<C>(st, smem, ln, i);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        nv_scales1<C, 0, 0>(st, i);
        nv_decode1<C, 0>(st, i);
    }

    int64_t gs = 0;                                     // stream position (stage buffer gs % 2)
    for (int64_t v = w; v < T; v += G) {
        v16f acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = v16f{};
        for (int s = 0; s < nst; ++s, ++gs) {
            uint8_t *buf = smem + (gs & 1) * C::STAGE;
            const uint8_t *nbuf = smem + ((gs + 1) & 1) * C::STAGE;
            StageIssue<C> issue = issue_at(ld, buf);    // stage gs + 2
            nv_region<C, 0, NT>(acc, st, buf, nbuf, ln, issue);
            ld.advance(nst, G, M, N, T);
        }
        store_tile(acc, tile_geo(v, M, N), M, N, wm, wn, lane, scale, y, y_bf16, ldy);
    }
}

// MXFP4, persistent, over a ring of NBUF stage buffers (stage g in buffer
// g % NBUF).  A stage has NS = KS/64 substeps of 16 scaled MFMAs; the operands
// of substep s + 1 are read during substep s, and during the last substep the
// next stage's first operands and scale bytes are read, so stages follow each
// other without a bubble.  The barrier of stage g sits before its last
// substep: by then this wave's reads of buffer g % NBUF are done and its loads
// of stage g + 1 have landed (vmcnt counts only the later stages still in
// flight); after it, stage g + 1 is readable and buffer g % NBUF is refilled
// with stage g + NBUF during the last substep.  The first barrier after a
// tile's stores waits for everything (vmcnt(0)), since the counter is only
// ordered among loads.
template <class C>
struct MxLane {
    static constexpr int NS = C::CH / 2;
    int codeA[NS], codeB[NS];                           // byte offset of this lane's unit in substep s (tile 0)
    int scA, scB;                                       // byte offset of this lane's NS scale bytes (tile 0)
    // tile i's scale bytes sit SCSTEP * i bytes further (32 rows)
    static constexpr int SCSTEP = 32 * (C::kGS ? C::GROW : C::SB);
    __device__ __forceinline__ MxLane(int rA0, int rB0, int h) {
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            codeA[q] = C::A_CODES + code_off<C::ROW>(rA0, NS * h + q);
            codeB[q] = C::B_CODES + code_off<C::ROW>(rB0, NS * h + q);
        }
        if constexpr (C::kGS) {                         // within a group buffer, at the stage's 4-byte column
            scA = rA0 * C::GROW + NS * h;
            scB = TM * C::GROW + rB0 * C::GROW + NS * h;
        } else {
            scA = C::A_SC + rA0 * C::SB + NS * h;
            scB = C::B_SC + rB0 * C::SB + NS * h;
        }
    }
};

template <class C>
struct MxState {
    uint4 a[2][4], b[2][4];                             // operands of substeps (even/odd)
    uint32_t sa[4], sb[4];                              // scale bytes of the current stage (byte s: substep s)
    uint32_t na[4], nb[4];                              // scale bytes of the next stage
};

template <class C>
__device__ __forceinline__ uint32_t mx_scale_read(const uint8_t *p) {
    if constexpr (C::CH / 2 == 4) return *reinterpret_cast<const uint32_t *>(p);
    else return *reinterpret_cast<const uint16_t *>(p);
}

// Part K of substep S of a stage: the 4 MFMAs of A tile K, reads of operands
// for the next substep (in the last substep, of the next stage's first one,
// with its scale bytes), and, in the last substep, a quarter of the loads of
// the stage NB later: they go out right after the barrier that frees its
// buffer, one per MFMA, which leaves them the most time.
// The next substep's first part multiplies A tile 0 by all four B tiles, so
// the B tiles are read first (parts 0 and 1, two each, with A tiles 0 and 1)
// and A tiles 2 and 3 after them: every operand is read at least 15 MFMAs
// (about 480 cycles) before its use.  Reading B tile K in part K left B tile
// 3 only 4 MFMAs ahead of its first use, under the LDS latency.
template <class C, int S, int NS, int K, class Issue>
__device__ __forceinline__ void mx_part(v16f (&acc)[4][4], MxState<C> &st, const uint8_t *buf,
                                        const uint8_t *nbuf, const uint8_t *nsc, const MxLane<C> &ln,
                                        Issue &next) {
    constexpr int E = S & 1, LAST = S == NS - 1;
    constexpr int NB_ = K < 2 ? 2 : 0;                  // B tiles read in this part: 2K, 2K + 1
    constexpr int ND = (1 + NB_) * (LAST ? 2 : 1);      // LDS reads in this part (operands, scale words)
    constexpr int NG = LAST ? Issue::template count<K, 4>() : 0;
    const uint8_t *src = LAST ? nbuf : buf;
    const int q = LAST ? 0 : (S + 1 < NS ? S + 1 : 0);
    __builtin_amdgcn_sched_barrier(0);
    st.a[E ^ 1][K] = lds16(src + ln.codeA[q] + 32 * C::ROW * K);
    if constexpr (NB_) {
        st.b[E ^ 1][2 * K] = lds16(src + ln.codeB[q] + 32 * C::ROW * (2 * K));
        st.b[E ^ 1][2 * K + 1] = lds16(src + ln.codeB[q] + 32 * C::ROW * (2 * K + 1));
    }
    if constexpr (LAST) {
        st.na[K] = mx_scale_read<C>(nsc + ln.scA + MxLane<C>::SCSTEP * K);
        if constexpr (NB_) {
            st.nb[2 * K] = mx_scale_read<C>(nsc + ln.scB + MxLane<C>::SCSTEP * (2 * K));
            st.nb[2 * K + 1] = mx_scale_read<C>(nsc + ln.scB + MxLane<C>::SCSTEP * (2 * K + 1));
        }
    }
    if constexpr (LAST) next.template region<K, 4>();
#pragma unroll
    for (int j = 0; j < 4; ++j)
        acc[K][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            as_v8i(st.a[E][K]), as_v8i(st.b[E][j]), acc[K][j], 4, 4, S, (int)st.sa[K], S, (int)st.sb[j]);
    static_for<0, 4>([&](auto KK) {
        constexpr int k = decltype(KK)::value;
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // one MFMA
        // the part's LDS reads spread over its four MFMAs, the earliest first
        constexpr int per = (ND + 3) / 4;
        constexpr int nr = (k + 1) * per <= ND ? per : (k * per < ND ? ND - k * per : 0);
        if constexpr (nr > 0) __builtin_amdgcn_sched_group_barrier(0x100, nr, 0);
        if constexpr (k < NG) __builtin_amdgcn_sched_group_barrier(0x010, 1, 0);       // one load
    });
    // keep the part's MFMAs in it (they would otherwise be sunk past the
    // stage's barrier and branches)
#pragma unroll
    for (int j = 0; j < 4; ++j) asm volatile("" : "+a"(acc[K][j]));
    __builtin_amdgcn_sched_barrier(0);
}

template <class C, int S, int NS, class Issue>
__device__ __forceinline__ void mx_substep(v16f (&acc)[4][4], MxState<C> &st, const uint8_t *buf,
                                           const uint8_t *nbuf, const uint8_t *nsc, const MxLane<C> &ln,
                                           Issue &next) {
    mx_part<C, S, NS, 0>(acc, st, buf, nbuf, nsc, ln, next);
    mx_part<C, S, NS, 1>(acc, st, buf, nbuf, nsc, ln, next);
    mx_part<C, S, NS, 2>(acc, st, buf, nbuf, nsc, ln, next);
    mx_part<C, S, NS, 3>(acc, st, buf, nbuf, nsc, ln, next);
}

// Scale-group loads issued after the last code load of stage g + 1 and before
// the wait in stage g (phase PH = g % GS_): stage g + 1's loads go out in the
// last substep of stage g + 1 - NB, and a group at the start of each stage j
// with j % GS_ == 0, so the groups of stages j in [g + 2 - NB, g] count.
template <int NB, int GS_, int PH>
constexpr int groups_after() {
    int n = 0;
    for (int d = 0; d <= NB - 2; ++d)
        if (((PH - d) % GS_ + GS_) % GS_ == 0) ++n;
    return n;
}

// One stage of the MXFP4 stream.  Past the end of the workgroup's stages the
// loads still go out (re-reading a stage of its first tile into a buffer
// nobody reads again), so every stage issues exactly LPS loads and the wait
// before the barrier is a constant of the stage's phase: the NB - 2 stages
// issued after stage g + 1 may stay in flight, and with scale groups (GS)
// also the group loads issued since (a group is loaded at the start of the
// stage whose loads, issued at its end, are the group's first stage).  A
// tile's first stage (after the previous tile's stores) waits for everything
// instead.  PH is the stage's position in its scale group (GS).
template <class C, int NB, int PH>
__device__ __forceinline__ void mx_stage_p(v16f (&acc)[4][4], MxState<C> &st, uint8_t *smem, int64_t gs,
                                           bool first, const MxLane<C> &ln, StageIssue<C> &issue) {
    constexpr int NS = C::CH / 2;
    const int bi = (int)(gs % NB);
    uint8_t *buf = smem + bi * C::STAGE;
    const uint8_t *nbuf = smem + (bi + 1 == NB ? 0 : bi + 1) * C::STAGE;
    // scale bytes of stage gs + 1: its group's buffer, at the stage's column
    const uint8_t *nsc;
    if constexpr (C::kGS)
        nsc = smem + C::SC_RING + (int)(((gs + 1) / C::GSTAGES) & 1) * C::GROUP + ((PH + 1) % C::GSTAGES) * C::SB;
    else
        nsc = nbuf;
    issue.buf = buf;                                    // stage gs + NB goes where stage gs was
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        st.sa[i] = st.na[i];
        st.sb[i] = st.nb[i];
    }
    mx_substep<C, 0, NS>(acc, st, buf, nbuf, nsc, ln, issue);
    if constexpr (NS == 4) {
        mx_substep<C, 1, NS>(acc, st, buf, nbuf, nsc, ln, issue);
        mx_substep<C, 2, NS>(acc, st, buf, nbuf, nsc, ln, issue);
    }
    constexpr int kInFlight = (NB - 2) * C::LPS + C::GLPW * groups_after<NB, C::GSTAGES, PH>();
    if (first) wait_vmcnt<0>();
    else wait_vmcnt<kInFlight>();
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    mx_substep<C, NS - 1, NS>(acc, st, buf, nbuf, nsc, ln, issue);
}

// Scale group loads (GS): wave w takes rows 64w .. 64w+63 of A and of B, 16
// bytes (GSTAGES stages) per row, into group buffer `gbuf`; edge tiles clamp rows.
// The addresses are those of the stage loads that start the group (their
// scale pointers and row limits).
template <class C>
__device__ __forceinline__ void load_scale_group(uint8_t *gbuf, int wave, int lane, const StageIssue<C> &at) {
    const int row = 64 * wave + lane;
    const int ra = row < at.rows_a ? row : at.rows_a - 1, rb = row < at.rows_b ? row : at.rows_b - 1;
    const int64_t spr = at.spr;
    const uint8_t *a_sc = at.as_, *b_sc = at.bs_;
    g2l16(a_sc, (uint32_t)(ra * (uint32_t)spr), gbuf + wave * 1024);
    g2l16(b_sc, (uint32_t)(rb * (uint32_t)spr), gbuf + TM * C::GROW + wave * 1024);
}

template <class C, int NB>
__device__ __forceinline__ void mx_persistent(uint8_t *smem, int64_t M, int64_t N, int64_t K,
                                              const uint8_t *a_codes, const uint8_t *a_scales,
                                              const uint8_t *b_codes, const uint8_t *b_scales, void *y,
                                              int y_bf16, int64_t ldy, int wave, int lane) {
    constexpr int KS = 2 * C::ROW, NS = C::CH / 2;
    constexpr int U = C::kGS ? C::GSTAGES : 1;          // stages per unrolled loop turn
    static_assert(NS % 2 == 0 && NB >= 2, "even substeps per stage");
    static_assert((NB - 1) * C::LPS + 2 * C::GLPW <= 63, "vmcnt range");
    static_assert(!C::kGS || NB == C::GSTAGES, "a group starts at the stage whose loads go out in its first stage");
    const int h = lane >> 5, wm = wave >> 1, wn = wave & 1;
    const int64_t tm_n = (M + TM - 1) / TM, tn_n = (N + TN - 1) / TN, T = tm_n * tn_n;
    const int64_t G = gridDim.x, w = blockIdx.x;
    const int nst = (int)(K / KS);                      // a multiple of U
    const int64_t cpr = K / 2, spr = K / C::B;
    const TileGeo g0 = tile_geo(w, M, N);

    // The load stream's position: the stage s within tile v, with the row
    // bases of that tile's operands (of the workgroup's first tile once past
    // the end: those loads land in a buffer nobody reads, and any stage of
    // that tile is in range).  The bases change only with the tile, so a
    // stage adds just its K offset.
    struct Pos {
        int64_t v;
        int s, rows_a, rows_b;
        const uint8_t *ac, *bc, *as_, *bs_;
    };
    auto pos_at = [&](int64_t v) {
        const TileGeo g = v < T ? tile_geo(v, M, N) : g0;
        return Pos{v, 0, g.rows_a, g.rows_b, a_codes + g.m0 * cpr, b_codes + g.n0 * cpr,
                   a_scales + g.m0 * spr, b_scales + g.n0 * spr};
    };
    auto advance = [&](Pos &p) {
        if (++p.s == nst) p = pos_at(p.v + G);
    };
    auto issue_at = [&](const Pos &p, uint8_t *buf) {
        const int64_t k0 = (int64_t)p.s * KS;
        return StageIssue<C>{buf, true, wave, lane, p.rows_a, p.rows_b, cpr, spr,
                             p.ac + k0 / 2, p.bc + k0 / 2, p.as_ + k0 / C::B, p.bs_ + k0 / C::B};
    };
    // scale group q (stream stages GSTAGES*q ..) into group buffer q & 1 (GS),
    // from the loads of its first stage
    auto group_at = [&](const StageIssue<C> &at, int64_t q) {
        load_scale_group<C>(smem + C::SC_RING + (int)(q & 1) * C::GROUP, wave, lane, at);
    };

    // prologue: scale group 0 (GS), stages 0 .. NB-1 into buffers 0 .. NB-1,
    // then wait for stage 0
    Pos ld = pos_at(w);
    if constexpr (C::kGS) group_at(issue_at(ld, smem), 0);
#pragma unroll
    for (int p = 0; p < NB; ++p) {
        issue_at(ld, smem + p * C::STAGE).template region<0, 1>();
        advance(ld);
    }
    wait_vmcnt<(NB - 1) * C::LPS>();
    asm volatile("s_barrier" ::: "memory");

    const MxLane<C> ln(wm * 128 + (lane & 31), wn * 128 + (lane & 31), h);
    MxState<C> st;
    const uint8_t *sc0 = C::kGS ? smem + C::SC_RING : smem;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        st.a[0][i] = lds16(smem + ln.codeA[0] + 32 * C::ROW * i);
        st.b[0][i] = lds16(smem + ln.codeB[0] + 32 * C::ROW * i);
        st.na[i] = mx_scale_read<C>(sc0 + ln.scA + MxLane<C>::SCSTEP * i);
        st.nb[i] = mx_scale_read<C>(sc0 + ln.scB + MxLane<C>::SCSTEP * i);
    }

    int64_t gs = 0;                                     // stream position (buffer gs % NB)
    for (int64_t v = w; v < T; v += G) {
        v16f acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = v16f{};
        for (int s = 0; s < nst; s += U) {
            static_for<0, U>([&](auto P) {
                constexpr int ph = decltype(P)::value;
                StageIssue<C> issue = issue_at(ld, smem);   // stage gs + NB
                // the group after this one starts at stage gs + NB (NB == GSTAGES):
                // loaded ahead of the code loads of that stage
                if constexpr (C::kGS && ph == 0) group_at(issue, gs / U + 1);
                mx_stage_p<C, NB, ph>(acc, st, smem, gs, s == 0 && ph == 0, ln, issue);
                advance(ld);
                ++gs;
            });
        }
        store_tile(acc, tile_geo(v, M, N), M, N, wm, wn, lane, 1.0f, y, y_bf16, ldy);
    }
    // no load may still be writing this workgroup's LDS when it exits
    wait_vmcnt<0>();
}

template <int FMT, int KS, int NBUF, bool GS>
__global__ __launch_bounds__(kThreads, 1) void gemm_tile256_kernel(
    int64_t M, int64_t N, int64_t K, const uint8_t *__restrict__ a_codes,
    const uint8_t *__restrict__ a_scales, const float *__restrict__ ga,
    const uint8_t *__restrict__ b_codes, const uint8_t *__restrict__ b_scales,
    const float *__restrict__ gb, void *__restrict__ y, int y_bf16, int64_t ldy) {
    using C = Cfg<FMT, KS, NBUF, GS>;
    extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    if constexpr (FMT == kNV)
        nv_persistent<C>(smem, M, N, K, a_codes, a_scales, uniform_load(ga) * uniform_load(gb), b_codes,
                         b_scales, y, y_bf16, ldy, wave, lane);
    else
        mx_persistent<C, NBUF>(smem, M, N, K, a_codes, a_scales, b_codes, b_scales, y, y_bf16, ldy, wave, lane);
}

// Compute units of the current device (cached per device).
int compute_units() {
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return -1;
    if (dev < 64 && cache[dev] > 0) return cache[dev];
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
    if (dev < 64) cache[dev] = n;
    return n;
}

template <int FMT, int KS, int NBUF, bool GS>
hipError_t launch_cfg(int64_t M, int64_t N, int64_t K, const uint8_t *a_codes, const uint8_t *a_scales,
                      const float *ga, const uint8_t *b_codes, const uint8_t *b_scales,
                      const float *gb, void *y, bool y_bf16, int64_t ldy, hipStream_t stream) {
    int64_t grid = ((M + TM - 1) / TM) * ((N + TN - 1) / TN);
    // persistent: one workgroup per CU (a multiple of 8 keeps each one on its XCD)
    const int cus = compute_units();
    if (cus <= 0) return hipErrorInvalidDevice;
    if (grid > cus) grid = cus;
    const size_t lds = Cfg<FMT, KS, NBUF, GS>::TOTAL;
    hipError_t e = hipFuncSetAttribute((const void *)gemm_tile256_kernel<FMT, KS, NBUF, GS>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((gemm_tile256_kernel<FMT, KS, NBUF, GS>), dim3((unsigned)grid), dim3(kThreads), lds,
                       stream, M, N, K, a_codes, a_scales, ga, b_codes, b_scales, gb, y, (int)y_bf16,
                       ldy);
    return hipGetLastError();
}

}  // namespace

bool gemm_tile256_supported(Fmt fmt, int64_t M, int64_t N, int64_t K, int64_t ldy) {
    const int ks = fmt == kMX ? REQAT_MX_KS : REQAT_NV_KS;
    // lane offsets are 32-bit: 256 rows * K/2 bytes and 4 * ldy * 4 bytes stay below 2^31
    return K > 0 && K % ks == 0 && M > 0 && N > 0 && K <= (int64_t(1) << 24) &&
           ldy <= (int64_t(1) << 26);
}

hipError_t launch_gemm_tile256(Fmt fmt, int64_t M, int64_t N, int64_t K, const uint8_t *a_codes,
                               const uint8_t *a_scales, const float *ga, const uint8_t *b_codes,
                               const uint8_t *b_scales, const float *gb, void *y, bool y_bf16,
                               int64_t ldy, hipStream_t stream) {
    if (fmt == kMX) {
        // scale groups need whole groups (GSTAGES stages) per tile and 16-byte aligned group loads
        constexpr int kGroupK = Cfg<kMX, REQAT_MX_GS_KS, REQAT_MX_GS_NBUF, true>::GSTAGES * REQAT_MX_GS_KS;
        const bool gs = K % kGroupK == 0 && (reinterpret_cast<uintptr_t>(a_scales) & 15u) == 0 &&
                        (reinterpret_cast<uintptr_t>(b_scales) & 15u) == 0;
        if (gs)
            return launch_cfg<kMX, REQAT_MX_GS_KS, REQAT_MX_GS_NBUF, true>(M, N, K, a_codes, a_scales, ga, b_codes,
                                                                           b_scales, gb, y, y_bf16, ldy, stream);
        return launch_cfg<kMX, REQAT_MX_KS, REQAT_MX_NBUF, false>(M, N, K, a_codes, a_scales, ga, b_codes,
                                                                  b_scales, gb, y, y_bf16, ldy, stream);
    }
    return launch_cfg<kNV, REQAT_NV_KS, REQAT_NV_NBUF, false>(M, N, K, a_codes, a_scales, ga, b_codes,
                                                              b_scales, gb, y, y_bf16, ldy, stream);
}

}  // namespace reqat
