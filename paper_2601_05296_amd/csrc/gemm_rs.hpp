// gemm_rs.hpp -- grouped bf16 MFMA GEMM core with register-staged operands
// (gfx950).
//
// One workgroup computes a BM x BN output tile with WM x WN waves; every wave
// owns a (BM/WM) x (BN/WN) sub-tile of 32x32 fragments computed with
// v_mfma_f32_32x32x16_bf16 (float32 accumulation). K advances in slices of
// KS = 64 elements (128 bytes of every K-contiguous row: each row of a slice
// is one whole cache line).
//
// Data movement. Every thread owns a fixed set of 16-byte chunks of each
// operand tile. A chunk is loaded from global memory into registers one slice
// ahead of the LDS write that commits it, and the LDS holds two slice buffers:
// while the MFMAs of slice kt read buffer kt&1, the chunks of slice kt+1 are
// written into the other buffer and the loads of slice kt+2 are issued into
// the registers those writes have just freed. A loader may transform a chunk
// between its load and its LDS write (h = SiLU(A) * B is formed there).
//
// Schedule. The main loop is unrolled over the four 16-deep MFMA steps of a
// slice. The fragments of step kk+1 are read from LDS while the MFMAs of step
// kk run, and the LDS writes and global loads of the chunks are spread between
// the MFMAs too: every group of one MFMA and its share of these operations is
// fenced with sched_barrier, so the compiler keeps this order and the vector
// memory, LDS and matrix units work at the same time. A single workgroup
// barrier per slice, in the middle of the last step, publishes the next
// slice; the first fragments of that slice are read after it, between the
// remaining MFMAs.
//
// MFMA 32x32x16 operand layout (wave64), verified on gfx950: for D = P * Q,
// lane L supplies P[L%32][8*(L/32) + 0..7] and Q[8*(L/32) + 0..7][L%32] and
// receives D[8*(j/4) + 4*(L/32) + j%4][L%32] in accumulator register j. The
// kernels pass P = right-operand tile (rows = output columns n) and
// Q = left-operand tile (rows = output rows m), so lane L ends up holding
// output row m = L%32 at columns n = 8*(j/4) + 4*(L/32) + (j%4).
//
// LDS tile layouts, chosen per operand by its layout in memory:
//  * KC ("K contiguous"): [R rows][64 k] bf16, 128-byte rows. The 16-byte
//    chunk c of row r sits at c ^ ((r >> 1) & 7): a ds_read_b128 of 16
//    consecutive rows at one chunk then touches 16 distinct 16-byte bank
//    groups of the 64 banks, and a chunk write of two whole rows does too.
//  * MC ("rows contiguous"): [64 k][R] bf16, for operands whose K is the
//    outer dimension. The 32-byte chunk index inside a k row is XOR-ed with
//    2 * (k & 3). A fragment read's 32 lanes of one pass take k rows k0..k0+3
//    at two neighbouring chunks (one even, one odd), so these eight
//    (row, chunk) pairs land on eight distinct 32-byte bank groups of the
//    256 bytes a k row spans in the banks (with (k & 3) alone, the odd and
//    the even chunk fell on the same four groups: a two-way bank conflict).
//    Fragments are read with gfx950's transposing LDS load
//    ds_read_b64_tr_b16: within each 16-lane group, lane l receives element
//    l%4 of the 4-element pieces supplied by lanes 4q + l/4 (q = 0..3), so
//    when lane 4q + c points at columns 4c..4c+3 of k row q, lane l receives
//    column l of k rows 0..3.
#pragma once

#include <type_traits>
#include <utility>

#include "common.hpp"

namespace moe {
namespace rs {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int KS = 64;          // K slice
constexpr int KSTEPS = KS / 16; // MFMA steps per slice

__device__ __forceinline__ f32x16 mfma32x32x16(const bf16x8& p, const bf16x8& q, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(p, q, c, 0, 0, 0);
}

// compile-time loop: f(integral_constant<int, 0>) ... f(integral_constant<int, N-1>)
template <class F, int... I>
__device__ __forceinline__ void sfor_impl(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void sfor(F&& f) {
    sfor_impl(f, std::make_integer_sequence<int, N>{});
}

template <int BM_, int BN_, int WM_, int WN_, int NB_>
struct Cfg {
    static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, NB = NB_;
    static constexpr int NW = WM * WN;
    static constexpr int THREADS = NW * WAVE;
    static constexpr int WTM = BM / WM, WTN = BN / WN;   // wave tile
    static constexpr int FM = WTM / 32, FN = WTN / 32;   // 32x32 fragments per wave
    static constexpr int A_BYTES = BM * KS * 2;
    static constexpr int B_BYTES = BN * KS * 2;
    static constexpr int STAGE = A_BYTES + NB * B_BYTES;
    static constexpr int LDS = 2 * STAGE;                // two slice buffers
    static_assert(FM >= 1 && FN >= 1, "wave tile too small");
    static_assert(LDS <= 160 * 1024, "LDS budget");
};

// ---- LDS layouts -------------------------------------------------------------------
__device__ __forceinline__ int kc_off(int r, int c) { return r * 128 + ((c ^ ((r >> 1) & 7)) << 4); }
template <int R>
__device__ __forceinline__ int mc_off(int k, int p) {   // p: logical 16-byte chunk of k row
    static_assert(R >= 128, "the MC swizzle permutes 32-byte chunks 0..7 of a k row");
    return k * (R * 2) + ((((p >> 1) ^ ((k & 3) << 1)) << 5) | ((p & 1) << 4));
}

// ---- fragment reads (32 rows x 16 k of MFMA step kk of the slice) ------------------
__device__ __forceinline__ bf16x8 frag_kc(const char* tile, int rbase, int kk, int lane) {
    const int r = rbase + (lane & 31);
    const int c = kk * 2 + (lane >> 5);
    return *reinterpret_cast<const bf16x8*>(tile + kc_off(r, c));
}
template <int R>
__device__ __forceinline__ bf16x8 frag_mc(const char* tile, int rbase, int kk, int lane) {
    const int g = lane >> 4;          // 16-lane group: column half (g&1), k octet (g>>1)
    const int p = lane & 15;
    const int k = kk * 16 + (g >> 1) * 8 + (p >> 2);
    const int cc = (rbase >> 4) + (g & 1);
    const int cb = (p & 3) * 8;
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    const char* a0 = tile + k * (R * 2) + (((cc ^ ((k & 3) << 1)) << 5) | cb);
    const char* a1 = tile + (k + 4) * (R * 2) + (((cc ^ (((k + 4) & 3) << 1)) << 5) | cb);
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

__device__ __forceinline__ u32x4 ldg16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void sts16(char* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }

// ---- chunk geometry ------------------------------------------------------------------
// KC tile of R rows: chunk q of the tile (q = i * THREADS + tid) is row q / 8,
// logical chunk q % 8 (k = 8 * (q % 8) .. + 7).
// MC tile of R columns: chunk q is k row q / (R / 8), columns 8 * (q % (R / 8)).
template <class C, int R>
struct KCGeom {
    static constexpr int NCH = R * KS * 2 / 16 / C::THREADS;   // chunks per thread
    static_assert(R * KS * 2 / 16 % C::THREADS == 0, "whole chunks per thread");
    __device__ static int row(int i) { return (i * C::THREADS + (int)threadIdx.x) >> 3; }
    __device__ static int chunk(int i) { return (i * C::THREADS + (int)threadIdx.x) & 7; }
    __device__ static int lds(int i) { return kc_off(row(i), chunk(i)); }
};
template <class C, int R>
struct MCGeom {
    static constexpr int CPR = R / 8;
    static constexpr int NCH = R * KS * 2 / 16 / C::THREADS;
    static_assert(R * KS * 2 / 16 % C::THREADS == 0, "whole chunks per thread");
    static_assert(C::THREADS % CPR == 0, "a thread's chunks share one column");
    __device__ static int krow(int i) { return (i * C::THREADS + (int)threadIdx.x) / CPR; }
    __device__ static int col(int i) { return 8 * ((i * C::THREADS + (int)threadIdx.x) % CPR); }
    __device__ static int lds(int i) {
        const int q = i * C::THREADS + (int)threadIdx.x;
        return mc_off<R>(q / CPR, q % CPR);
    }
};

// ---- main loop ---------------------------------------------------------------------
// LA: left-operand loader (rows = output rows m), LB0 / LB1: right-operand
// loaders (rows = output columns n, same layout). A loader has static bool MC
// (its LDS layout), static int NCH (chunks per thread per slice),
// load<i>(kt) (issue the global load(s) of chunk i of slice kt into its
// registers), static int NSUB and sub<i, p>() for p < NSUB (the pieces of a
// transform of chunk i in registers, run in order after its data has arrived;
// NSUB = 0 for a plain copy) and store<i, TAIL>(tile) (write chunk i at its place in
// the LDS tile). On return acc[b][i][j] holds sum_k A[m][k] B_b[k][n] for the
// fragment at rows wm*WTM + 32i, columns wn*WTN + 32j.
// Every wave computes all its fragments, also those that lie beyond the
// tile's real rows or columns (on clamped operand rows; the epilogues do not
// store them). Skipping them would need a second copy of the scheduled loop
// (or a branch per MFMA), and either costs the register allocation of the
// loop some 30 VGPRs, which it does not have.
// The LDS must be free on entry: callers that used it before (the tile
// lookup) put a barrier between.
struct NoLoader {
    static constexpr bool MC = false;
    static constexpr int NCH = 0;
    static constexpr int NSUB = 0;
    template <int i> __device__ void load(int) {}
    template <int i, int p> __device__ void sub() {}
    template <int i, bool TAIL> __device__ void store(char*) {}
};

// ---- side operations of one slice -------------------------------------------------------
// The chunk work of a slice, in issue order: for every chunk, its transform
// pieces, its LDS write (slice kt+1) and its load (slice kt+2). The chunks of
// the loaders are interleaved in proportion to their numbers, and every
// operation is placed after one of the slice's NPOS MFMAs before the barrier,
// by its cumulative weight: a transform piece (h of one element: some 6
// vector instructions and 2 transcendentals) weighs W_PIECE, a memory
// instruction 1, so that the vector work is spread evenly between the MFMAs.
constexpr int W_PIECE = 4;
template <int MAXN>
struct SliceOps {
    int n = 0;
    int kind[MAXN] = {};    // 0 transform piece, 1 LDS write, 2 load
    int chunk[MAXN] = {};
    int piece[MAXN] = {};
    int pos[MAXN] = {};     // MFMA of the slice after which the operation issues
};
template <int NA, int N0, int N1, int SA, int S0, int S1, int MODE, int NPOS>
constexpr auto slice_ops() {
    constexpr int NCH = NA + N0 + N1;
    constexpr int SMAX = SA > S0 ? (SA > S1 ? SA : S1) : (S0 > S1 ? S0 : S1);
    SliceOps<NCH * (SMAX + 2) + 1> L;
    if (MODE == 2) return L;
    const int cnt[3] = {NA, N0, N1};
    const int nsub[3] = {SA, S0, S1};
    const int base[3] = {0, NA, NA + N0};
    int used[3] = {0, 0, 0};
    int total = 0;
    for (int q = 0; q < NCH; ++q) {
        // the loader whose next chunk is furthest behind its share
        int l = -1;
        for (int c = 0; c < 3; ++c) {
            if (used[c] >= cnt[c]) continue;
            if (l < 0 || (2 * used[c] + 1) * cnt[l] < (2 * used[l] + 1) * cnt[c]) l = c;
        }
        const int g = base[l] + used[l]++;
        for (int p = 0; p < nsub[l]; ++p) {
            L.kind[L.n] = 0; L.chunk[L.n] = g; L.piece[L.n] = p; L.pos[L.n] = total; ++L.n;
            total += W_PIECE;
        }
        L.kind[L.n] = 1; L.chunk[L.n] = g; L.pos[L.n] = total; ++L.n;
        total += 1;
        if (MODE == 0) {
            L.kind[L.n] = 2; L.chunk[L.n] = g; L.pos[L.n] = total; ++L.n;
            total += 1;
        }
    }
    for (int o = 0; o < L.n; ++o) L.pos[o] = L.pos[o] * NPOS / (total > 0 ? total : 1);
    return L;
}
// the schedule of a slice of the main loop (MODE as in mainloop)
template <class C, class LA, class LB0, class LB1, int MODE>
struct SliceSchedule {
    static constexpr int NM = C::NB * C::FM * C::FN;
    static constexpr int NPOS = (KSTEPS - 1) * NM + NM / 2;   // MFMAs before the barrier
    static constexpr auto ops =
        slice_ops<LA::NCH, LB0::NCH, C::NB == 2 ? LB1::NCH : 0, LA::NSUB, LB0::NSUB,
                  C::NB == 2 ? LB1::NSUB : 0, MODE, NPOS>();
};
// first operation placed at MFMA p or later
template <class L>
constexpr int first_op_at(const L& ops, int p) {
    int o = 0;
    while (o < ops.n && ops.pos[o] < p) ++o;
    return o;
}

template <class C, class LA, class LB0, class LB1>
__device__ __forceinline__ void mainloop(LA& la, LB0& lb0, LB1& lb1, int nk, char* lds,
                                         Acc<C>& acc) {
    sfor<C::NB>([&](auto b) {
        sfor<C::FM>([&](auto i) {
            sfor<C::FN>([&](auto j) {
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[b][i][j][r] = 0.f;
            });
        });
    });
    if (nk <= 0) return;
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int wm = wv / C::WN, wn = wv % C::WN;
    constexpr int NA = LA::NCH, N0 = LB0::NCH, N1 = C::NB == 2 ? LB1::NCH : 0;
    constexpr int NCH = NA + N0 + N1;              // chunks per thread per slice
    constexpr int NR = C::FM + C::NB * C::FN;      // fragment reads per MFMA step
    constexpr int NM = C::NB * C::FM * C::FN;      // MFMAs per step and wave

    // chunk g of the slice: which loader, which of its chunks
    auto load_chunk = [&](auto g_c, int kt) __attribute__((always_inline)) {
        constexpr int g = decltype(g_c)::value;
        if constexpr (g < NA) la.template load<g>(kt);
        else if constexpr (g < NA + N0) lb0.template load<g - NA>(kt);
        else lb1.template load<g - NA - N0>(kt);
    };
    // TAIL: the chunk belongs to the last slice, whose K rows may run past the
    // operand's extent (loaders that zero such rows do so only then)
    auto store_chunk = [&](auto g_c, char* stage, auto tail_c) __attribute__((always_inline)) {
        constexpr int g = decltype(g_c)::value;
        constexpr bool TAIL = decltype(tail_c)::value;
        if constexpr (g < NA) la.template store<g, TAIL>(stage);
        else if constexpr (g < NA + N0) lb0.template store<g - NA, TAIL>(stage + C::A_BYTES);
        else lb1.template store<g - NA - N0, TAIL>(stage + C::A_BYTES + C::B_BYTES);
    };
    auto sub_chunk = [&](auto g_c, auto p_c) __attribute__((always_inline)) {
        constexpr int g = decltype(g_c)::value, p = decltype(p_c)::value;
        if constexpr (g < NA) la.template sub<g, p>();
        else if constexpr (g < NA + N0) lb0.template sub<g - NA, p>();
        else lb1.template sub<g - NA - N0, p>();
    };
    auto nsub_of = [](auto g_c) {
        constexpr int g = decltype(g_c)::value;
        return std::integral_constant<int, g < NA ? LA::NSUB : g < NA + N0 ? LB0::NSUB : LB1::NSUB>{};
    };
    // the chunk's transform and LDS write, all at once (prologue)
    auto commit_chunk = [&](auto g_c, char* stage) __attribute__((always_inline)) {
        sfor<decltype(nsub_of(g_c))::value>([&](auto p) { sub_chunk(g_c, p); });
        store_chunk(g_c, stage, std::true_type{});   // slice 0 may be the last
    };

    bf16x8 fr[2][NR];
    auto read_frag = [&](auto slot_c, auto r_c, const char* stage, int kk) __attribute__((always_inline)) {
        constexpr int slot = decltype(slot_c)::value, r = decltype(r_c)::value;
        if constexpr (r < C::FM) {
            fr[slot][r] = frag<LA::MC, C::BM>(stage, wm * C::WTM + r * 32, kk, lane);
        } else {
            constexpr int b = (r - C::FM) / C::FN, j = (r - C::FM) % C::FN;
            fr[slot][r] = frag<LB0::MC, C::BN>(stage + C::A_BYTES + b * C::B_BYTES,
                                               wn * C::WTN + j * 32, kk, lane);
        }
    };


    // prologue: slice 0 into buffer 0, slice 1 into registers, fragments of step 0
    sfor<NCH>([&](auto g) { load_chunk(g, 0); });
    sfor<NCH>([&](auto g) { commit_chunk(g, lds); });
    if (nk > 1) sfor<NCH>([&](auto g) { load_chunk(g, 1); });
    __syncthreads();
    sfor<NR>([&](auto r) { read_frag(std::integral_constant<int, 0>{}, r, lds, 0); });

    // one slice. MODE 0: write slice kt+1, load slice kt+2; 1: write only; 2: last.
    // Fragment order: the MFMAs of a step run in NRUN runs of RUN MFMAs that
    // share one fragment of the larger set (the left fragments when FM >= NBF,
    // the right ones otherwise): MFMA m pairs run m / RUN with member m % RUN.
    // The next step's fragments of the smaller set are read right after the
    // first MFMAs of the step (they live next to the current ones: two sets);
    // the next step's fragment of run q is read right after the run's last
    // MFMA (the two never live at the same time, so they can share registers).
    constexpr int NBF = C::NB * C::FN;
    constexpr bool ROW_RUNS = C::FM >= NBF;          // runs share a left fragment
    constexpr int NRUN = ROW_RUNS ? C::FM : NBF;     // runs per step
    constexpr int RUN = ROW_RUNS ? NBF : C::FM;      // MFMAs per run
    static_assert(NRUN % 2 == 0, "barrier between runs");
    auto slice = [&](int kt, auto mode_c, auto idle_c) __attribute__((always_inline)) {
        constexpr int MODE = decltype(mode_c)::value;
        constexpr bool IDLE = decltype(idle_c)::value;
        const char* cur = lds + (kt & 1) * C::STAGE;
        char* nxt = lds + ((kt + 1) & 1) * C::STAGE;
        sfor<KSTEPS>([&](auto kk_c) __attribute__((always_inline)) {
            constexpr int kk = decltype(kk_c)::value;
            constexpr int cs = kk & 1, ns = (kk + 1) & 1;
            constexpr bool last_kk = kk == KSTEPS - 1;
            constexpr bool split = last_kk && MODE <= 1;    // barrier inside this step
            constexpr int nm_pre = split ? NM / 2 : NM;      // MFMAs before the barrier
            constexpr bool reads_here = !IDLE && !last_kk;
            constexpr bool reads_next_slice = !IDLE && split;
            sfor<NM>([&](auto m_c) __attribute__((always_inline)) {
                constexpr int m = decltype(m_c)::value;
                constexpr int q = m / RUN, u = m % RUN;      // run, member
                constexpr int i = ROW_RUNS ? q : u;
                constexpr int bj = ROW_RUNS ? u : q;
                constexpr int b = bj / C::FN, j = bj % C::FN;
                // fragment slots: left i -> i, right bj -> FM + bj
                constexpr int run_slot = ROW_RUNS ? q : C::FM + q;
                constexpr int NSMALL = RUN;                  // fragments of the smaller set
                if constexpr (split && m == nm_pre) {
                    // the chunks of slice kt+1 are in LDS once every wave's
                    // writes have completed
                    __builtin_amdgcn_sched_barrier(0);
                    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
                    __builtin_amdgcn_sched_barrier(0);
                }
                if constexpr (!IDLE)
                    acc[b][i][j] = mfma32x32x16(fr[cs][C::FM + bj], fr[cs][i], acc[b][i][j]);
                __builtin_amdgcn_sched_barrier(0);
                auto rd = [&](auto r_c, const char* stage, int kstep) __attribute__((always_inline)) {
                    read_frag(std::integral_constant<int, ns>{}, r_c, stage, kstep);
                };
                // slot of member-set fragment x (the smaller set)
                auto small_slot = [](auto x_c) {
                    constexpr int x = decltype(x_c)::value;
                    return std::integral_constant<int, ROW_RUNS ? C::FM + x : x>{};
                };
                if constexpr (reads_here) {
                    if constexpr (m < NSMALL) rd(small_slot(std::integral_constant<int, m>{}), cur, kk + 1);
                    if constexpr (u == RUN - 1) rd(std::integral_constant<int, run_slot>{}, cur, kk + 1);
                }
                if constexpr (reads_next_slice && m >= nm_pre) {
                    if constexpr (m == nm_pre) {
                        // the smaller set, and the run fragments of runs finished before the barrier
                        sfor<NSMALL>([&](auto x) { rd(small_slot(x), nxt, 0); });
                        sfor<nm_pre / RUN>([&](auto x) {
                            rd(std::integral_constant<int, ROW_RUNS ? decltype(x)::value : C::FM + decltype(x)::value>{}, nxt, 0);
                        });
                    }
                    if constexpr (u == RUN - 1 && q >= nm_pre / RUN)
                        rd(std::integral_constant<int, run_slot>{}, nxt, 0);
                }
                if constexpr (m < nm_pre) {
                    // the chunk operations placed after this MFMA
                    constexpr int p = kk * NM + m;
                    using SCH = SliceSchedule<C, LA, LB0, LB1, MODE>;
                    constexpr int o0 = first_op_at(SCH::ops, p), o1 = first_op_at(SCH::ops, p + 1);
                    sfor<o1 - o0>([&](auto oi_c) __attribute__((always_inline)) {
                        constexpr int o = o0 + decltype(oi_c)::value;
                        constexpr int g = SCH::ops.chunk[o];
                        if constexpr (SCH::ops.kind[o] == 0)
                            sub_chunk(std::integral_constant<int, g>{},
                                      std::integral_constant<int, SCH::ops.piece[o]>{});
                        else if constexpr (SCH::ops.kind[o] == 1)
                            store_chunk(std::integral_constant<int, g>{}, nxt,
                                        std::integral_constant<bool, MODE == 1>{});
                        else
                            load_chunk(std::integral_constant<int, g>{}, kt + 2);
                    });
                }
                __builtin_amdgcn_sched_barrier(0);
            });
        });
    };
    auto run = [&](auto idle_c) __attribute__((always_inline)) {
        int kt = 0;
        for (; kt + 2 < nk; ++kt) slice(kt, std::integral_constant<int, 0>{}, idle_c);
        if (kt + 1 < nk) {
            slice(kt, std::integral_constant<int, 1>{}, idle_c);
            ++kt;
        }
        slice(kt, std::integral_constant<int, 2>{}, idle_c);
    };
    run(std::false_type{});
    // every wave is done reading LDS before an epilogue reuses it
    __syncthreads();
}

// ---- operand loaders -------------------------------------------------------------------
// Rows or columns at or beyond an operand's extent are clamped to valid memory;
// the epilogues never store the outputs that depend on them. A loader keeps one
// base pointer and at most a 32-bit row number per chunk; chunk addresses are
// formed when the load is issued (the main loop has vector-ALU time to spare,
// and registers are what limits its schedule).

// element offset of row r in a matrix of row stride ld
__device__ __forceinline__ int64_t roff(int64_t r, int ld) { return r * (int64_t)ld; }

// KC rows gathered through an index list: tile row r -> base[idx[r]] (rows at
// or beyond `rows` read row idx[0]).
template <class C, int R>
struct GatherKC {
    static constexpr bool MC = false;
    using G = KCGeom<C, R>;
    static constexpr int NCH = G::NCH;
    static constexpr int NSUB = 0;
    template <int i, int p> __device__ void sub() {}
    const bf16_t* p;       // base + this thread's chunk column
    int ld;
    int row[NCH];          // gathered row of each chunk
    u32x4 v[NCH];
    __device__ void init(const bf16_t* base, int ld_, const int32_t* idx, int rows) {
        ld = ld_;
        p = base + G::chunk(0) * 8;   // the same column for every chunk of the thread
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            int r = G::row(i);
            r = r < rows ? r : 0;
            row[i] = idx[r];
        }
    }
    template <int i> __device__ void load(int kt) { v[i] = ldg16(p + roff(row[i], ld) + kt * KS); }
    template <int i, bool TAIL> __device__ void store(char* tile) { sts16(tile + G::lds(i), v[i]); }
};

// KC rows row0 + r (r < rows, else row0) of a dense row-major matrix, K split
// over two sources: k < ksplit from src0, k >= ksplit from src1 (same ld;
// ksplit a multiple of the slice).
template <class C, int R>
struct DenseKC2 {
    static constexpr bool MC = false;
    using G = KCGeom<C, R>;
    static constexpr int NCH = G::NCH;
    static constexpr int NSUB = 0;
    template <int i, int p> __device__ void sub() {}
    const bf16_t* p0;      // src0 + row0 * ld + this thread's chunk column
    int64_t d01;           // src1 - src0 - ksplit, in elements
    int ld, rows, kst;     // kst: slices served by src0
    u32x4 v[NCH];
    __device__ void init(const bf16_t* src0, const bf16_t* src1, int ld_, int64_t row0, int rows_,
                         int ksplit) {
        ld = ld_;
        rows = rows_;
        kst = ksplit / KS;
        d01 = (src1 - src0) - (int64_t)ksplit;
        p0 = src0 + roff(row0, ld) + G::chunk(0) * 8;
    }
    template <int i> __device__ void load(int kt) {
        int r = G::row(i);
        r = r < rows ? r : 0;
        v[i] = ldg16(p0 + roff(r, ld) + kt * KS + (kt < kst ? 0 : d01));
    }
    template <int i, bool TAIL> __device__ void store(char* tile) { sts16(tile + G::lds(i), v[i]); }
};

// MC tile of a dense row-major [K][ncols] matrix, columns col0.. (clamped)
template <class C, int R>
struct DenseMC {
    static constexpr bool MC = true;
    using G = MCGeom<C, R>;
    static constexpr int NCH = G::NCH;
    static constexpr int NSUB = 0;
    template <int i, int p> __device__ void sub() {}
    const bf16_t* p;       // W + this thread's first k row and column
    int ld;
    u32x4 v[NCH];
    __device__ void init(const bf16_t* W, int ld_, int col0, int ncols) {
        ld = ld_;
        int c = col0 + G::col(0);   // the same column for every chunk of the thread
        c = c < ncols ? c : ncols - 8;
        p = W + roff(G::krow(0), ld) + c;
    }
    template <int i> __device__ void load(int kt) {
        v[i] = ldg16(p + roff(kt * KS + (G::krow(i) - G::krow(0)), ld));
    }
    template <int i, bool TAIL> __device__ void store(char* tile) { sts16(tile + G::lds(i), v[i]); }
};

// MC tile of a [K][ncols] matrix whose K rows come from two row ranges of one
// matrix: k < ksplit -> row k, k >= ksplit -> row k - ksplit; rows at or
// beyond nrows are clamped (the other operand is zero there).
template <class C, int R>
struct SplitRowsMC {
    static constexpr bool MC = true;
    using G = MCGeom<C, R>;
    static constexpr int NCH = G::NCH;
    static constexpr int NSUB = 0;
    template <int i, int p> __device__ void sub() {}
    const bf16_t* base;
    int ld, ksplit, nrows;
    u32x4 v[NCH];
    __device__ void init(const bf16_t* W, int ld_, int col0, int ncols, int ksplit_, int nrows_) {
        ld = ld_;
        ksplit = ksplit_;
        nrows = nrows_;
        int c = col0 + G::col(0);
        c = c < ncols ? c : ncols - 8;
        base = W + c;
    }
    template <int i> __device__ void load(int kt) {
        int k = kt * KS + G::krow(i);
        k = k < ksplit ? k : k - ksplit;
        k = k < nrows ? k : nrows - 1;
        v[i] = ldg16(base + roff(k, ld));
    }
    template <int i, bool TAIL> __device__ void store(char* tile) { sts16(tile + G::lds(i), v[i]); }
};

// ---- loaders whose K is the slot dimension of one expert (weight gradients) ----
// K row kr (0 <= kr < cnt) is slot off + kr. Rows at or past cnt are read
// from row cnt - 1 and stored as zeros, so that the last slice's extra rows
// add nothing.

// MC rows gathered through eti: K row kr -> base[eti[off + kr]] (x or dY). The
// row index of a chunk is loaded one slice ahead of the row itself.
// When a whole wave covers one K row (R a multiple of 512 columns), the index
// is the same for the whole wave. All NCH indices of a wave's slice then come
// in by one vector load, lane j holding chunk j's, issued with the first chunk
// of the slice before (so that the wait for it is a counted one), and each
// chunk takes its index with a lane read. With scalar loads instead (one per
// chunk) the compiler cannot count LDS reads while one is outstanding, and the
// LDS waits of the loop became waits for everything.
template <class C, int R>
struct GatherMC {
    static constexpr bool MC = true;
    using G = MCGeom<C, R>;
    static constexpr int NCH = G::NCH;
    static constexpr int NSUB = 0;
    template <int i, int p> __device__ void sub() {}
    static constexpr bool UNIFORM = G::CPR % WAVE == 0;
    static_assert(!UNIFORM || NCH <= WAVE, "one lane per chunk index");
    const bf16_t* base;
    const int32_t* idx;   // eti + off
    int ld, cnt;
    // row of the chunk's next slice; UNIFORM: [0] this slice's rows, [1] the
    // next slice's (lane j: chunk j)
    int nidx[UNIFORM ? 2 : NCH];
    uint32_t zmask;       // chunks of the loaded slice that lie past cnt
    u32x4 v[NCH];
    __device__ static int krow(int i) {
        if constexpr (UNIFORM)   // wave w covers k rows i * (THREADS / CPR) + w * WAVE / CPR
            return i * (C::THREADS / G::CPR) +
                   __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6) * WAVE / G::CPR;
        else return G::krow(i);
    }
    __device__ int kr(int i, int kt) const {
        const int k = kt * KS + krow(i);
        return k < cnt ? k : cnt - 1;
    }
    // UNIFORM: the indices of all of this wave's chunks at slice kt, lane j
    // loading chunk j's (lanes past NCH repeat the last)
    __device__ int lane_rows(int kt) const {
        const int j = min((int)(threadIdx.x & (WAVE - 1)), NCH - 1);
        const int k = kt * KS + j * (C::THREADS / G::CPR) + ((int)threadIdx.x >> 6) * WAVE / G::CPR;
        return idx[k < cnt ? k : cnt - 1];
    }
    // cnt_ >= 1
    __device__ void init(const bf16_t* b, int ld_, int col0, int ncols, const int32_t* ix,
                         int cnt_) {
        ld = ld_;
        idx = ix;
        cnt = cnt_;
        zmask = 0;
        int c = col0 + G::col(0);
        c = c < ncols ? c : ncols - 8;
        base = b + c;
        if constexpr (UNIFORM) nidx[1] = lane_rows(0);
        else {
#pragma unroll
            for (int i = 0; i < NCH; ++i) nidx[i] = idx[kr(i, 0)];
        }
    }
    // chunks are loaded in the order i = 0 .. NCH-1 within a slice
    template <int i> __device__ void load(int kt) {
        const bool past = kt * KS + krow(i) >= cnt;
        zmask = past ? (zmask | (1u << i)) : (zmask & ~(1u << i));
        if constexpr (UNIFORM) {
            if constexpr (i == 0) {
                // a real move (identity DPP), never merged with the load: at the
                // loop head no index register may still wait for its load, or
                // the compiler waits there for every load in flight
                nidx[0] = __builtin_amdgcn_update_dpp(0, nidx[1], 0xE4, 0xF, 0xF, false);
                nidx[1] = lane_rows(kt + 1);
            }
            v[i] = ldg16(base + roff(__builtin_amdgcn_readlane(nidx[0], i), ld));
        } else {
            v[i] = ldg16(base + roff(nidx[i], ld));
            nidx[i] = idx[kr(i, kt + 1)];
        }
    }
    template <int i, bool TAIL> __device__ void store(char* tile) {
        const u32x4 z = {0u, 0u, 0u, 0u};
        if constexpr (TAIL) sts16(tile + G::lds(i), (zmask >> i) & 1 ? z : v[i]);
        else sts16(tile + G::lds(i), v[i]);
    }
};

// MC rows of a slot-ordered [S][ld] matrix (g*h, dA, dB, or a token-ordered
// matrix with off = first token): K row kr -> src[off + kr].
template <class C, int R>
struct SlotMC {
    static constexpr bool MC = true;
    using G = MCGeom<C, R>;
    static constexpr int NCH = G::NCH;
    static constexpr int NSUB = 0;
    template <int i, int p> __device__ void sub() {}
    const bf16_t* base;
    int ld, cnt;
    uint32_t zmask;
    u32x4 v[NCH];
    __device__ void init(const bf16_t* src, int ld_, int64_t off, int col0, int ncols, int cnt_) {
        ld = ld_;
        cnt = cnt_;
        zmask = 0;
        int c = col0 + G::col(0);
        c = c < ncols ? c : ncols - 8;
        base = src + roff(off, ld) + c;
    }
    template <int i> __device__ void load(int kt) {
        int k = kt * KS + G::krow(i);
        const bool past = k >= cnt;
        zmask = past ? (zmask | (1u << i)) : (zmask & ~(1u << i));
        k = past ? cnt - 1 : k;
        v[i] = ldg16(base + roff(k, ld));
    }
    template <int i, bool TAIL> __device__ void store(char* tile) {
        const u32x4 z = {0u, 0u, 0u, 0u};
        if constexpr (TAIL) sts16(tile + G::lds(i), (zmask >> i) & 1 ? z : v[i]);
        else sts16(tile + G::lds(i), v[i]);
    }
};

// slices of a K extent of cnt rows
__device__ __forceinline__ int slices(int cnt) { return (cnt + KS - 1) / KS; }

}  // namespace rs
}  // namespace moe
