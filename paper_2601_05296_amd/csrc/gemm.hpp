// gemm.hpp -- pieces shared by the grouped GEMM kernels, the router and the
// router backward (gfx950): MFMA and LDS helpers, direct-to-LDS copies (used
// by the router's ring), the 16-byte epilogue layout of a 32x32 accumulator
// fragment, a wave's output coordinates, float32 tile output through LDS, and
// the tile orders of the weight-gradient and the row-wise grouped GEMMs. The
// GEMM main loop and its operand loaders are in gemm_rs.hpp.
//
// MFMA 32x32x16 operand layout (wave64), verified on gfx950: for D = P * Q,
// lane L supplies P[L%32][8*(L/32) + 0..7] and Q[8*(L/32) + 0..7][L%32] and
// receives D[8*(j/4) + 4*(L/32) + j%4][L%32] in accumulator register j. The
// kernels pass P = right-operand tile (rows = output columns n) and
// Q = left-operand tile (rows = output rows m), so lane L ends up holding
// output row m = L%32 at columns n = 8*(j/4) + 4*(L/32) + (j%4): four runs of
// four consecutive columns.
#pragma once

#include <type_traits>

#include "common.hpp"

namespace moe {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void_t;


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

// accumulators of a tile configuration C: [right operand][fragment row][fragment column]
template <class C>
using Acc = f32x16[C::NB][C::FM][C::FN];

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
// Call after rs::mainloop (whose final barrier frees the LDS). Between
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
// over the expert's tokens, so a tile's length is its expert's token count.
// Workgroup ids are dealt round-robin to the 8 XCDs (each with its own L2).
// Every XCD takes, for every expert, one band of ceil(P/8) consecutive tiles,
// so that every XCD gets the same share of every expert whatever the experts'
// token counts. The experts are taken longest first: rank[r] holds the expert
// of rank r by token count (descending, ties to the lower index), its first
// slot and its count (expert_ranks). Under a skewed routing the longest tiles
// then start first and the many short ones fill in around them, instead of a
// late start of the longest tiles setting the kernel's end. Inside an expert
// the tiles are grouped WG_GM row tiles at a time with the column tile slower:
// the ~32 workgroups an XCD runs at once then cover a WG_GM x 8 block of
// tiles, which read WG_GM + 8 operand panels per K slice from L2 instead of
// the 1 + 32 of a row-major band (an expert's last, narrower group holds its
// remaining rows). Returns false for the padding tiles of the last band.
constexpr int WG_GM = 4;
struct ExpertRank {
    int32_t e, off, cnt, pad;
};
__device__ __forceinline__ bool wgrad_tile(const ExpertRank* __restrict__ rank, int bid, int MT,
                                           int NT, ExpertRank& er, int& mt, int& nt) {
    const int P = MT * NT;
    const int G = (P + 7) >> 3;
    const int x = bid & 7, j = bid >> 3;
    const int lt = x * G + j % G;
    if (lt >= P) return false;
    er = rank[j / G];
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
// holds its remaining M tiles). Every thread of the block must call this;
// `sh` is 8 ints of LDS, free on entry and again on return. Returns false past
// the last tile.
struct SlotTile {
    int e;       // expert
    int m0;      // first row inside the expert's slot segment
    int mrows;   // valid rows in this tile (<= BM)
    int n0;      // first output column
    int off;     // offsets[e]
};

template <int THREADS>
__device__ bool find_slot_tile(int* sh, const int32_t* __restrict__ offsets, int E, int BM, int NT,
                               int bid, int BN, SlotTile& t, int GM = 0) {
    static_assert(THREADS >= 256, "one thread per expert");
    const int tid = threadIdx.x, lane = tid & (WAVE - 1), wv = tid / WAVE;
    int tiles = 0, cnt = 0, off = 0;
    if (tid < E) {
        off = offsets[tid];
        cnt = offsets[tid + 1] - off;
        tiles = ((cnt + BM - 1) / BM) * NT;
    }
    // expert e's tiles are [start, end): a wave-level scan, plus the totals of
    // the waves before (E <= 256: four waves)
    const int inc = wave_incl_scan(tiles);
    if (wv < 4 && lane == WAVE - 1) sh[wv] = inc;
    if (tid == 0) sh[4] = -1;
    __syncthreads();
    if (tid < E) {
        int end = inc;
        for (int w = 0; w < wv; ++w) end += sh[w];
        const int start = end - tiles;
        if (bid >= start && bid < end) { sh[4] = tid; sh[5] = bid - start; sh[6] = off; sh[7] = cnt; }
    }
    __syncthreads();
    const int e = sh[4], local = sh[5];
    off = sh[6];
    cnt = sh[7];
    __syncthreads();
    if (e < 0) return false;
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
    t.off = off;
    t.m0 = mt * BM;
    t.mrows = min(BM, cnt - t.m0);
    t.n0 = nt * BN;
    return true;
}

}  // namespace moe
