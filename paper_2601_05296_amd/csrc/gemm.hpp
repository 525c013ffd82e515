// gemm.hpp -- grouped bf16 MFMA GEMM core for the expert FFN (gfx950).
//
// One workgroup computes a BM x BN output tile with WM x WN waves; every wave
// owns a (BM/WM) x (BN/WN) sub-tile made of 32x32 fragments computed with
// v_mfma_f32_32x32x16_bf16 (float32 accumulation). K advances in slices of
// BK = 32.
//
// Data movement: operand tiles go straight from global memory into LDS with
// gfx950's global_load_lds_dwordx4 (no register staging). One instruction
// moves 64 lanes x 16 bytes into 1 KB of contiguous LDS, lane l writing bytes
// 16l..16l+15; each lane therefore fetches whichever global 16-byte chunk the
// swizzled LDS layout wants at that position (this is also how rows are
// gathered through the dispatch index maps). LDS holds a ring of NST slices:
// while the MFMAs consume slice kt, the loads for slices kt+1 .. kt+NST-1 are
// in flight. The hardware counts outstanding loads per wave (vmcnt); a wave
// waits until the loads of slice kt+1 have landed and a workgroup barrier
// publishes them to the other waves. The waits are explicit because a
// compiler-generated __syncthreads() would drain every outstanding load.
//
// A kernel may hand the main loop a pre-pass that rewrites each slice's left
// operand in LDS before it is multiplied (the h-on-load GEMMs form h =
// SiLU(A) * B there). It runs one slice ahead: while slice kt is multiplied,
// slice kt+1 (landed) is transformed, its element pairs spread between the
// MFMAs of slice kt, and slice kt+2 is in flight.
//
// MFMA 32x32x16 operand layout (wave64), verified on gfx950: for D = P * Q,
// lane L supplies P[L%32][8*(L/32) + 0..7] and Q[8*(L/32) + 0..7][L%32] and
// receives D[8*(j/4) + 4*(L/32) + j%4][L%32] in accumulator register j. The
// kernels pass P = right-operand tile (rows = output columns n) and
// Q = left-operand tile (rows = output rows m), so lane L ends up holding
// output row m = L%32 at columns n = 8*(j/4) + 4*(L/32) + (j%4): four runs of
// four consecutive columns.
//
// Two LDS tile layouts, chosen per operand by its layout in memory:
//  * KC ("K contiguous"): [R rows][32 k] bf16 (64-byte rows), for operands
//    whose K is the contiguous dimension. The 16-byte chunk index c of row r
//    is stored at c ^ ((r >> 2) & 3): a ds_read_b128 of 32 rows then has no
//    bank conflict (measured with SQ_LDS_BANK_CONFLICT on gfx950; with
//    c ^ ((r >> 1) & 3), rows r and r + 8 collide).
//  * MC ("rows contiguous"): [32 k][R] bf16, for operands whose K is the
//    outer dimension (weights [K][N], and every operand of the weight-gradient
//    GEMMs, whose K is the token dimension). The 32-byte chunk index inside a
//    k row is XOR-ed with (k & 3). Fragments are read with gfx950's
//    transposing LDS load ds_read_b64_tr_b16: within each 16-lane group, lane
//    l receives element l%4 of the 4-element pieces supplied by lanes
//    4q + l/4 (q = 0..3), so when lane 4q + c points at columns 4c..4c+3 of k
//    row q, lane l receives column l of k rows 0..3.
#pragma once

#include <type_traits>

#include "common.hpp"

namespace moe {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int GBK = 32;  // K slice
constexpr int NST = 3;   // LDS ring depth (slices)

__device__ __forceinline__ f32x16 mfma32x32x16(const bf16x8& p, const bf16x8& q, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(p, q, c, 0, 0, 0);
}

// Wait until at most N vector-memory operations of this wave are outstanding.
// Inline assembly with a memory clobber, so that the compiler moves no memory
// access across it.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier without the implicit drain of outstanding loads that
// __syncthreads() adds; also a compiler memory barrier.
__device__ __forceinline__ void barrier_only() { asm volatile("s_barrier" ::: "memory"); }

// Barrier after this wave's LDS accesses have completed.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// 16-byte global -> LDS copy by one lane: lane l writes LDS bytes
// lds_off + 16*l .. +15 (lds_off must be wave-uniform; it goes to M0). Issued
// from inline assembly so that the compiler does not track these copies: it
// would otherwise drain all of them (vmcnt(0)) before every transposing LDS
// read, which it cannot prove independent of the copies in flight. The main
// loop waits for them explicitly (wait_vmcnt), so no compiler-visible vector
// memory access may be issued inside it.
__device__ __forceinline__ void dma16(const void* g, uint32_t lds_off) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 ::"v"(g), "s"(lds_off) : "memory", "m0");
}

// 4-byte global -> LDS copy by one lane: lane l writes LDS bytes
// lds_off + 4*l .. +3 (same rules as dma16; the source needs only 4-byte
// alignment).
__device__ __forceinline__ void dma4(const void* g, uint32_t lds_off) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
                 ::"v"(g), "s"(lds_off) : "memory", "m0");
}

// LDS byte offset of a pointer into the workgroup's shared memory.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)p;
}

// Wave index as a value the compiler knows to be uniform (kept in an SGPR).
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// XA extra left-operand-shaped tiles per stage follow the left operand's tile
// (raw inputs that a pre-pass folds into it, e.g. B of h = SiLU(A) * B); the
// right-operand tiles start after them, at AREG.
template <int BM_, int BN_, int WM_, int WN_, int NB_, int XA_ = 0>
struct GemmCfg {
    static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, NB = NB_, XA = XA_;
    static constexpr int NW = WM * WN;
    static constexpr int THREADS = NW * WAVE;
    static constexpr int WTM = BM / WM, WTN = BN / WN;   // wave tile
    static constexpr int FM = WTM / 32, FN = WTN / 32;   // 32x32 fragments per wave
    static constexpr int A_BYTES = BM * GBK * 2;
    static constexpr int B_BYTES = BN * GBK * 2;
    static constexpr int AREG = (1 + XA) * A_BYTES;
    static constexpr int STAGE = AREG + NB * B_BYTES;
    static constexpr int LDS = NST * STAGE;
    static_assert(FM >= 1 && FN >= 1, "wave tile too small");
    static_assert(LDS <= 160 * 1024, "LDS budget");
    static_assert(A_BYTES % (1024 * NW) == 0 && B_BYTES % (1024 * NW) == 0,
                  "every wave issues the same number of 1 KB copies");
};

// ---- LDS layouts -------------------------------------------------------------------
__device__ __forceinline__ int kc_swz(int r, int c) { return c ^ ((r >> 2) & 3); }

// KC tile of R rows, copy q (1 KB = 16 rows): lane l -> row 16q + l/4, physical
// chunk l%4, i.e. logical chunk kc_swz(row, l%4).
struct KCDma {
    __device__ static int row(int q, int lane) { return q * 16 + (lane >> 2); }
    __device__ static int kcol(int q, int lane) { return kc_swz(row(q, lane), lane & 3) * 8; }
};

// MC tile of R columns, copy q (1 KB = 1024/(2R) k rows): lane l -> k row
// q*KPK + l/(R/8), physical 16-byte chunk p = l%(R/8), logical column
// ((p/2) ^ (k&3))*16 + (p&1)*8.
template <int R>
struct MCDma {
    static constexpr int CPR = R / 8, KPK = 1024 / (2 * R);
    static_assert(KPK >= 1 && R >= 64, "MC tile width");
    __device__ static int krow(int q, int lane) { return q * KPK + lane / CPR; }
    __device__ static int col(int q, int lane) {
        const int k = krow(q, lane);
        const int p = lane % CPR;
        return (((p >> 1) ^ (k & 3)) << 4) + ((p & 1) << 3);
    }
};

// ---- fragment reads (32 rows x 16 k of MFMA step kk in the 32-wide slice) -----
__device__ __forceinline__ bf16x8 frag_kc(const char* tile, int rbase, int kk, int lane) {
    const int r = rbase + (lane & 31);
    const int c = kk * 2 + (lane >> 5);
    return *reinterpret_cast<const bf16x8*>(tile + r * 64 + (kc_swz(r, c) << 4));
}

template <int R>
__device__ __forceinline__ bf16x8 frag_mc(const char* tile, int rbase, int kk, int lane) {
    const int g = lane >> 4;          // 16-lane group: column half (g&1), k octet (g>>1)
    const int p = lane & 15;
    const int k = kk * 16 + (g >> 1) * 8 + (p >> 2);
    const int cc = (rbase >> 4) + (g & 1);
    const int cb = (p & 3) * 8;
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    const char* a0 = tile + k * (R * 2) + (((cc ^ (k & 3)) << 5) | cb);
    const char* a1 = tile + (k + 4) * (R * 2) + (((cc ^ ((k + 4) & 3)) << 5) | cb);
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(a0));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(a1));
    typedef short i16x8 __attribute__((ext_vector_type(8)));
    const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

template <bool MC, int R>
__device__ __forceinline__ bf16x8 frag(const char* tile, int rbase, int kk, int lane) {
    if constexpr (MC) return frag_mc<R>(tile, rbase, kk, lane);
    else return frag_kc(tile, rbase, kk, lane);
}

template <class C>
using Acc = f32x16[C::NB][C::FM][C::FN];

// Zero k rows [from, GBK) of an MC tile of R columns (all threads take part).
template <class C, int R>
__device__ __forceinline__ void zero_mc_rows(char* tile, int from) {
    const int nbytes = (GBK - from) * R * 2;
    char* base = tile + from * R * 2;
    for (int o = threadIdx.x * 16; o < nbytes; o += C::THREADS * 16) st16(base + o, zero16());
}

// ---- main loop -------------------------------------------------------------------
// LA: left-operand loader (rows = output rows m), LB0/LB1: right-operand
// loaders (rows = output columns n, same layout). A loader has a static bool
// MC, a static int NQ (1 KB copies per wave per slice) and issue(kt, tile),
// which is called once per slice in increasing kt. If zero_from < GBK, k rows
// zero_from.. of the left operand's last slice are cleared after they land
// (the left operand is then MC; used for the weight gradients' token tails).
// On return acc[b][i][j] holds sum_k A[m][k] B_b[k][n] for the fragment at
// rows wm*WTM + 32i, columns wn*WTN + 32j.
// arows / bcols: rows of the left operand tile and columns of the right one
// that hold real outputs. A wave whose fragments lie wholly beyond them skips
// their LDS reads and MFMAs (its loads still land: the copies are shared).
// PRE: an optional pass over the stage of slice kt (pre(stage, kt)) run by the
// whole workgroup once the slice is visible and before any fragment is read,
// followed by a barrier: it turns the raw tiles of the left operand (the XA
// extra ones included) into the operand the MFMAs consume.
struct NoPre {
    static constexpr bool active = false;
    static constexpr int NPAIR = 0;
    struct St {};
    __device__ void operator()(char*, int) const {}
    __device__ void pair(St&, int) const {}
};
template <class C, class LA, class LB0, class LB1, class PRE = NoPre>
__device__ __forceinline__ void gemm_mainloop(LA& la, LB0& lb0, LB1& lb1, int nk, int zero_from,
                                              char* lds, Acc<C>& acc, int arows = C::BM,
                                              int bcols = C::BN, PRE pre = PRE{}) {
#pragma unroll
    for (int b = 0; b < C::NB; ++b)
#pragma unroll
        for (int i = 0; i < C::FM; ++i)
#pragma unroll
            for (int j = 0; j < C::FN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[b][i][j][r] = 0.f;
    if (nk <= 0) return;
    const int lane = threadIdx.x & 63;
    const int wv = wave_id();
    const int wm = wv / C::WN, wn = wv % C::WN;
    constexpr int PER = LA::NQ + LB0::NQ + (C::NB == 2 ? LB1::NQ : 0);  // copies per slice

    const uint32_t lds_base = lds_offset(lds);
    auto issue = [&](int kt) {
        const uint32_t t = lds_base + (kt % NST) * C::STAGE;
        la.issue(kt, t);
        lb0.issue(kt, t + C::AREG);
        if constexpr (C::NB == 2) lb1.issue(kt, t + C::AREG + C::B_BYTES);
    };
    auto fix_tail = [&](int kt) {  // called once slice kt is visible to all waves
        if (kt == nk - 1 && zero_from < GBK) {
#pragma unroll
            for (int x = 0; x <= C::XA; ++x)
                zero_mc_rows<C, C::BM>(lds + (kt % NST) * C::STAGE + x * C::A_BYTES, zero_from);
            __syncthreads();
        }
    };

    // prologue: slices 0 .. NST-2
#pragma unroll
    for (int s = 0; s < NST - 1; ++s)
        if (s < nk) issue(s);
    if (nk >= NST - 1) wait_vmcnt<PER * (NST - 2)>();
    else wait_vmcnt<0>();
    barrier_only();
    fix_tail(0);

    // fragments of this wave that hold real outputs (wave-uniform)
    const int nfm = min(C::FM, max(0, (arows - wm * C::WTM + 31) >> 5));
    const int nfn = min(C::FN, max(0, (bcols - wn * C::WTN + 31) >> 5));
    // the MFMAs of slice kt (fragments read from its LDS stage)
    auto mma = [&](int kt, auto partial) {
        constexpr bool PART = decltype(partial)::value;
        const char* cur = lds + (kt % NST) * C::STAGE;
#pragma unroll
        for (int kk = 0; kk < GBK / 16; ++kk) {
            bf16x8 fa[C::FM];
#pragma unroll
            for (int i = 0; i < C::FM; ++i)
                if (!PART || (i < nfm && nfn > 0))
                    fa[i] = frag<LA::MC, C::BM>(cur, wm * C::WTM + i * 32, kk, lane);
#pragma unroll
            for (int b = 0; b < C::NB; ++b) {
                const char* bt = cur + C::AREG + b * C::B_BYTES;
                bf16x8 fb[C::FN];
#pragma unroll
                for (int j = 0; j < C::FN; ++j)
                    if (!PART || (j < nfn && nfm > 0))
                        fb[j] = frag<LB0::MC, C::BN>(bt, wn * C::WTN + j * 32, kk, lane);
#pragma unroll
                for (int i = 0; i < C::FM; ++i)
#pragma unroll
                    for (int j = 0; j < C::FN; ++j)
                        if (!PART || (i < nfm && j < nfn))
                            acc[b][i][j] = mfma32x32x16(fb[j], fa[i], acc[b][i][j]);
            }
        }
    };
    // The MFMAs of slice kt with the pre-pass of slice kt+1 spread between
    // them: after each MFMA the thread forms its share of element pairs, fenced
    // so that the compiler keeps the order. The wave then issues vector work
    // while the matrix core runs its MFMAs. All fragment reads come first.
    auto mma_pre = [&](int kt, auto partial, auto& st) {
        constexpr bool PART = decltype(partial)::value;
        constexpr int KK = GBK / 16;
        constexpr int NM = KK * C::NB * C::FM * C::FN;   // MFMAs per slice and wave
        const char* cur = lds + (kt % NST) * C::STAGE;
        bf16x8 fa[KK][C::FM], fb[KK][C::NB][C::FN];
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
            for (int i = 0; i < C::FM; ++i)
                if (!PART || (i < nfm && nfn > 0))
                    fa[kk][i] = frag<LA::MC, C::BM>(cur, wm * C::WTM + i * 32, kk, lane);
#pragma unroll
            for (int b = 0; b < C::NB; ++b)
#pragma unroll
                for (int j = 0; j < C::FN; ++j)
                    if (!PART || (j < nfn && nfm > 0))
                        fb[kk][b][j] = frag<LB0::MC, C::BN>(cur + C::AREG + b * C::B_BYTES,
                                                            wn * C::WTN + j * 32, kk, lane);
        }
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
#pragma unroll
            for (int b = 0; b < C::NB; ++b)
#pragma unroll
                for (int i = 0; i < C::FM; ++i)
#pragma unroll
                    for (int j = 0; j < C::FN; ++j) {
                        if (!PART || (i < nfm && j < nfn))
                            acc[b][i][j] = mfma32x32x16(fb[kk][b][j], fa[kk][i], acc[b][i][j]);
                        const int m = ((kk * C::NB + b) * C::FM + i) * C::FN + j;
                        const int p0 = m * PRE::NPAIR / NM, p1 = (m + 1) * PRE::NPAIR / NM;
                        if (p1 > p0) {
                            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                            for (int q = p0; q < p1; ++q) pre.pair(st, q);
                            __builtin_amdgcn_sched_barrier(0);
                        }
                    }
    };
    if constexpr (!PRE::active) {
        auto loop = [&](auto partial) {
            for (int kt = 0; kt < nk; ++kt) {
                if (kt + NST - 1 < nk) issue(kt + NST - 1);
                mma(kt, partial);
                if (kt + 1 < nk) {
                    // slice kt+1 has landed once only the copies of later slices remain
                    if (kt + NST - 1 < nk) wait_vmcnt<PER * (NST - 2)>();
                    else wait_vmcnt<0>();
                    barrier_only();
                    fix_tail(kt + 1);
                }
            }
        };
        if (nfm == C::FM && nfn == C::FN) loop(std::false_type{});
        else loop(std::true_type{});
    } else {
        // The pre-pass runs one slice ahead of the MFMAs: while slice kt is
        // multiplied, slice kt+1 (landed) is transformed in its own stage, and
        // slice kt+2 is in flight.
        static_assert(NST == 3, "stages: multiplied, transformed, in flight");
        pre(lds, 0);
        lds_barrier();
        auto loop = [&](auto partial) {
            for (int kt = 0; kt < nk; ++kt) {
                if (kt + 1 < nk) {
                    wait_vmcnt<0>();   // slice kt+1, the last one issued, has landed
                    barrier_only();
                    fix_tail(kt + 1);
                }
                if (kt + NST - 1 < nk) issue(kt + NST - 1);   // into the stage slice kt-1 left
                // (after the last slice this transforms a spent stage, which
                // nothing reads again: one MFMA block in the loop, not two)
                char* nxt = lds + ((kt + 1) % NST) * C::STAGE;
                typename PRE::St st;
                pre.load(nxt, kt + 1, st);
                mma_pre(kt, partial, st);
                pre.store(nxt, st);
                lds_barrier();
            }
        };
        if (nfm == C::FM && nfn == C::FN) loop(std::false_type{});
        else loop(std::true_type{});
    }
    // every wave is done reading LDS before an epilogue reuses it
    __syncthreads();
}

// Placeholder loader for single-B GEMMs.
struct NoLoader {
    static constexpr bool MC = false;
    static constexpr int NQ = 0;
    __device__ void issue(int, uint32_t) {}
};

// ---- 16-byte epilogue layout ----------------------------------------------------------
// In a 32x32 accumulator fragment lane L holds row L%32 at four runs of four
// columns, 8q + 4*(L/32) + 0..3 (q = 0..3). gfx950's v_permlane32_swap trades
// values between lanes L and L+32 so that, for p = 0, 1, lane L holds the
// eight consecutive columns 16p + 8*(L/32) + 0..7 instead: epilogues then load
// and store 16 bytes of bf16 per lane, whole 32-byte sectors per row.
__device__ __forceinline__ void frag_cols8(const f32x16& a, float (&v)[2][8]) {
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const auto s = __builtin_amdgcn_permlane32_swap(
                __float_as_uint(a[8 * p + r]), __float_as_uint(a[8 * p + 4 + r]), false, false);
            v[p][r] = __uint_as_float(s[0]);
            v[p][4 + r] = __uint_as_float(s[1]);
        }
}

// ---- output coordinates of a lane ------------------------------------------------
template <class C>
struct WaveCoord {
    int lane, wm, wn;
    __device__ WaveCoord() {
        lane = threadIdx.x & 63;
        const int wv = threadIdx.x >> 6;
        wm = wv / C::WN;
        wn = wv % C::WN;
    }
    // tile-local output row of fragment row-block i
    __device__ int row(int i) const { return wm * C::WTM + i * 32 + (lane & 31); }
    // tile-local first column of run q (0..3) of fragment column-block j
    __device__ int col(int j, int q) const { return wn * C::WTN + j * 32 + q * 8 + (lane >> 5) * 4; }
    // tile-local first column of eight-column group p (0, 1) after frag_cols8
    __device__ int col8(int j, int p) const { return wn * C::WTN + j * 32 + p * 16 + (lane >> 5) * 8; }
};

// ---- f32 tile output through LDS -------------------------------------------------------
// The accumulators go through LDS, IPR fragment row-blocks of every wave per
// round, and leave as whole rows of the tile: a wave's store instruction covers
// 1 KB of consecutive output bytes (or two rows of 512 B), so every 128-byte
// line is written by a single instruction. LDS rows are padded by 16 bytes,
// which keeps both the fragment writes and the row reads free of bank conflicts.
// Call after gemm_mainloop (whose final barrier frees the LDS ring). Between
// rounds only the LDS accesses are ordered: the global stores of a round stay
// in flight while the next round is staged.

template <class C, int IPR>
struct RowStage {
    static constexpr int ROWS = C::WM * 32 * IPR;
    static constexpr int PITCH = C::BN * 4 + 16;
    static constexpr int V4_PER_ROW = C::BN / 4;
    static constexpr int PASSES = ROWS * V4_PER_ROW / C::THREADS;
    static constexpr int ROUNDS = C::NB * C::FM / IPR;
    static_assert(ROWS * PITCH <= C::LDS, "staging fits the LDS ring");
    static_assert(C::FM % IPR == 0 && (ROWS * V4_PER_ROW) % C::THREADS == 0, "even split");
    // store(b, tile_row, tile_col, f32x4) is called for every 4 consecutive outputs
    template <class F>
    __device__ static void run(const Acc<C>& acc, char* lds, F&& store) {
        const WaveCoord<C> wc;
#pragma unroll
        for (int rd = 0; rd < ROUNDS; ++rd) {
            const int b = rd / (C::FM / IPR), i0 = (rd % (C::FM / IPR)) * IPR;
            if (rd > 0) lds_barrier();
#pragma unroll
            for (int ii = 0; ii < IPR; ++ii)
#pragma unroll
                for (int j = 0; j < C::FN; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int cr = wc.wm * 32 * IPR + ii * 32 + (wc.lane & 31);
                        const f32x16& v = acc[b][i0 + ii][j];
                        *reinterpret_cast<f32x4*>(lds + cr * PITCH + wc.col(j, q) * 4) =
                            f32x4{v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
                    }
            lds_barrier();
            f32x4 v[PASSES];
#pragma unroll
            for (int p = 0; p < PASSES; ++p) {
                const int t = threadIdx.x + p * C::THREADS;
                v[p] = *reinterpret_cast<const f32x4*>(lds + (t / V4_PER_ROW) * PITCH +
                                                       (t % V4_PER_ROW) * 16);
            }
#pragma unroll
            for (int p = 0; p < PASSES; ++p) {
                const int t = threadIdx.x + p * C::THREADS;
                const int cr = t / V4_PER_ROW, c4 = t % V4_PER_ROW;
                const int row = (cr / (32 * IPR)) * C::WTM + (i0 + (cr / 32) % IPR) * 32 + (cr & 31);
                store(b, row, c4 * 4, v[p]);
            }
        }
    }
};

// ---- weight-gradient tile order ---------------------------------------------------------
// The weight-gradient GEMMs have P = MT*NT output tiles per expert, each looping
// over the expert's tokens. Workgroup ids are dealt round-robin to the 8 XCDs
// (each with its own L2). Every XCD takes, for every expert, one band of
// ceil(P/8) consecutive tiles, so that every XCD gets the same share of every
// expert whatever the experts' token counts. Inside an expert the tiles come in
// groups of WG_GM row tiles with the column tile slower: the ~32 workgroups
// an XCD runs at once then cover a WG_GM x 8 block of tiles, which read
// WG_GM + 8 operand panels per K slice from L2 instead of the 1 + 32 of a
// row-major band (an expert's last, narrower group holds its remaining rows).
// Returns false for the padding tiles of the last band.
constexpr int WG_GM = 4;
__device__ __forceinline__ bool wgrad_tile(int bid, int MT, int NT, int& e, int& mt, int& nt) {
    const int P = MT * NT;
    const int G = (P + 7) >> 3;
    const int x = bid & 7, j = bid >> 3;
    e = j / G;
    const int lt = x * G + j % G;
    if (lt >= P) return false;
    const int grp = lt / (WG_GM * NT);
    const int m_base = grp * WG_GM;
    const int gm = min(WG_GM, MT - m_base);
    const int in = lt - grp * WG_GM * NT;
    mt = m_base + in % gm;
    nt = in / gm;
    return true;
}
inline int wgrad_grid(int E, int MT, int NT) { return E * 8 * ((MT * NT + 7) / 8); }

// ---- grouped tile lookup ------------------------------------------------------------
// Tiles of expert e: ceil(M_e / BM) * NT, laid out expert after expert. With
// GM = 0 the M tile index runs fastest (neighbouring tiles share a weight
// panel). With GM > 0 the tiles come in groups of GM M tiles, N slower
// inside a group: the workgroups that run at the same time on one XCD then
// cover a GM x (32 / GM) block of tiles, which share both their row panels
// and their weight panels in that XCD's L2 (an expert's last, narrower group
// holds its remaining M tiles).
// Every thread of the block must call this. Returns false past the last tile.
struct SlotTile {
    int e;       // expert
    int m0;      // first row inside the expert's slot segment
    int mrows;   // valid rows in this tile (<= BM)
    int n0;      // first output column
    int off;     // offsets[e]
};

template <int THREADS>
__device__ bool find_slot_tile(const int32_t* __restrict__ offsets, int E, int BM, int NT,
                               int bid, int BN, SlotTile& t, int GM = 0) {
    static_assert(THREADS >= 256, "one thread per expert");
    __shared__ int s_scan[THREADS];
    __shared__ int s_res[2];
    const int tid = threadIdx.x;
    int tiles = 0;
    if (tid < E) {
        const int cnt = offsets[tid + 1] - offsets[tid];
        tiles = ((cnt + BM - 1) / BM) * NT;
    }
    s_scan[tid] = tiles;
    if (tid == 0) { s_res[0] = -1; s_res[1] = 0; }
    __syncthreads();
    for (int o = 1; o < THREADS; o <<= 1) {
        const int v = tid >= o ? s_scan[tid - o] : 0;
        __syncthreads();
        s_scan[tid] += v;
        __syncthreads();
    }
    if (tid < E) {
        const int end = s_scan[tid];
        const int start = end - tiles;
        if (bid >= start && bid < end) { s_res[0] = tid; s_res[1] = bid - start; }
    }
    __syncthreads();
    const int e = s_res[0];
    if (e < 0) return false;
    const int local = s_res[1];
    const int cnt = offsets[e + 1] - offsets[e];
    const int nmt = (cnt + BM - 1) / BM;
    const int gm = GM > 0 ? GM : nmt;         // M tiles per group
    const int full = nmt / gm * gm;           // M tiles in whole groups
    int mt, nt;
    if (local < full * NT) {
        const int g = local / (gm * NT), w = local % (gm * NT);
        mt = g * gm + w % gm;
        nt = w / gm;
    } else {
        const int rem = nmt - full, l2 = local - full * NT;
        mt = full + l2 % rem;
        nt = l2 / rem;
    }
    t.e = e;
    t.off = offsets[e];
    t.m0 = mt * BM;
    t.mrows = min(BM, cnt - t.m0);
    t.n0 = nt * BN;
    return true;
}

}  // namespace moe
