// gemm.hpp -- grouped bf16 MFMA GEMM core for the expert FFN (gfx950).
//
// One workgroup computes a BM x BN output tile with WM x WN waves; every wave
// owns a (BM/WM) x (BN/WN) sub-tile made of 16x16 MFMA fragments. K advances
// in slices of 64. Operand tiles are staged in LDS, double-buffered: global
// loads of slice kt+1 are issued before the MFMAs of slice kt, written to the
// other LDS buffer after them, and a single barrier per slice separates the
// two.
//
// Two LDS tile layouts, chosen per operand by its global layout:
//  * KC ("K contiguous"): [R rows][64 k] bf16, used when K is the contiguous
//    dimension in memory (activations with K = d, weights read transposed).
//    The 16-byte chunk index inside a 128-byte row is XOR-ed with (row & 7).
//    Fragments are single ds_read_b128 loads.
//  * MC ("rows contiguous"): [64 k][R] bf16, used when K is the outer
//    dimension (weights [K][N], and every operand of the weight-gradient
//    GEMMs, whose K is the token dimension). The 32-byte chunk index inside a
//    row is XOR-ed with (k & 3). Fragments are read with gfx950's transposing
//    LDS load ds_read_b64_tr_b16: within each 16-lane group, lane l receives
//    element l%4 of the 4-element pieces supplied by lanes 4q + l/4, q = 0..3,
//    so 16 lanes that each point at 4 consecutive columns of 4 consecutive k
//    rows receive, per lane, one column's 4 k values.
//
// The operand loaders (fetch: global -> registers, stage: registers -> LDS,
// possibly computing on the way) are supplied per GEMM stage.
#pragma once

#include "common.hpp"

namespace moe {

constexpr int GBK = 64;  // K slice

template <int BM_, int BN_, int WM_, int WN_, int NB_>
struct GemmCfg {
    static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, NB = NB_;
    static constexpr int THREADS = WM * WN * WAVE;
    static constexpr int WTM = BM / WM, WTN = BN / WN;
    static constexpr int FM = WTM / 16, FN = WTN / 16;
    static constexpr int A_BYTES = BM * GBK * 2;
    static constexpr int B_BYTES = BN * GBK * 2;
    static constexpr int STAGE = A_BYTES + NB * B_BYTES;
    static constexpr int LDS = 2 * STAGE;
    static_assert(FM >= 1 && FN >= 1, "wave tile too small");
};

// ---- per-thread chunk maps ---------------------------------------------------
// KC tile of R rows: chunk c = tid + i*THREADS -> row c/8, 16-byte chunk c%8.
template <int R, int THREADS>
struct KCMap {
    static constexpr int NCH = R * 8 / THREADS;
    static_assert(NCH >= 1 && R * 8 % THREADS == 0, "KC tile / thread count mismatch");
    __device__ static int row(int tid, int i) { return (tid >> 3) + i * (THREADS / 8); }
    __device__ static int kcol(int tid) { return (tid & 7) * 8; }  // element offset in slice
    __device__ static int off(int tid, int i) {
        const int r = row(tid, i);
        return r * 128 + (((tid & 7) ^ (r & 7)) << 4);
    }
};

// MC tile of R columns: chunk c = tid + i*THREADS -> k row c/(R/8), column chunk c%(R/8).
template <int R, int THREADS>
struct MCMap {
    static constexpr int CPR = R / 8;
    static constexpr int NCH = GBK * CPR / THREADS;
    static_assert(NCH >= 1 && GBK * CPR % THREADS == 0, "MC tile / thread count mismatch");
    static_assert(R >= 64, "MC tile needs at least 64 columns for the swizzle");
    __device__ static int krow(int tid, int i) { return tid / CPR + i * (THREADS / CPR); }
    __device__ static int col(int tid) { return (tid % CPR) * 8; }
    __device__ static int off(int tid, int i) {
        const int k = krow(tid, i);
        const int c = tid % CPR;
        return k * (R * 2) + ((((c >> 1) ^ (k & 3)) << 5) | ((c & 1) << 4));
    }
};

// ---- fragment reads ------------------------------------------------------------
// 8 consecutive k (k-octet L/16 of MFMA step kk) of tile row rbase + L%16.
__device__ __forceinline__ bf16x8 frag_kc(const char* tile, int rbase, int kk, int lane) {
    const int r = rbase + (lane & 15);
    const int c = kk * 4 + (lane >> 4);
    return *reinterpret_cast<const bf16x8*>(tile + r * 128 + ((c ^ (r & 7)) << 4));
}

template <int R>
__device__ __forceinline__ bf16x8 frag_mc(const char* tile, int rbase, int kk, int lane) {
    const int p = lane & 15;
    const int k = kk * 32 + (lane >> 4) * 8 + (p >> 2);
    const int cc = rbase >> 4;
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

// ---- main loop -------------------------------------------------------------------
// LA: left-operand loader (rows = output rows m), LB0/LB1: right-operand
// loaders (rows = output columns n). Each loader has a static bool MC, and
// members fetch(int kt) and stage(char* tile). acc[b][fm][fn] receives
// sum_k A[m][k] B_b[k][n] for m = wm*WTM + fm*16 + L%16,
// n = wn*WTN + fn*16 + 4*(L/16) + r.
template <class C, class LA, class LB0, class LB1>
__device__ __forceinline__ void gemm_mainloop(LA& la, LB0& lb0, LB1& lb1, int nk, char* lds,
                                              f32x4 (&acc)[C::NB][C::FM][C::FN]) {
#pragma unroll
    for (int b = 0; b < C::NB; ++b)
#pragma unroll
        for (int i = 0; i < C::FM; ++i)
#pragma unroll
            for (int j = 0; j < C::FN; ++j) acc[b][i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (nk <= 0) return;
    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int wm = wv / C::WN, wn = wv % C::WN;

    la.fetch(0);
    lb0.fetch(0);
    if constexpr (C::NB == 2) lb1.fetch(0);
    la.stage(lds);
    lb0.stage(lds + C::A_BYTES);
    if constexpr (C::NB == 2) lb1.stage(lds + C::A_BYTES + C::B_BYTES);
    __syncthreads();

    for (int kt = 0; kt < nk; ++kt) {
        char* cur = lds + (kt & 1) * C::STAGE;
        char* nxt = lds + ((kt + 1) & 1) * C::STAGE;
        const bool more = kt + 1 < nk;
        if (more) {
            la.fetch(kt + 1);
            lb0.fetch(kt + 1);
            if constexpr (C::NB == 2) lb1.fetch(kt + 1);
        }
#pragma unroll
        for (int kk = 0; kk < GBK / 32; ++kk) {
            bf16x8 fa[C::FM];
#pragma unroll
            for (int i = 0; i < C::FM; ++i)
                fa[i] = frag<LA::MC, C::BM>(cur, wm * C::WTM + i * 16, kk, lane);
#pragma unroll
            for (int b = 0; b < C::NB; ++b) {
                const char* bt = cur + C::A_BYTES + b * C::B_BYTES;
                bf16x8 fb[C::FN];
#pragma unroll
                for (int j = 0; j < C::FN; ++j)
                    fb[j] = frag<LB0::MC, C::BN>(bt, wn * C::WTN + j * 16, kk, lane);
#pragma unroll
                for (int i = 0; i < C::FM; ++i)
#pragma unroll
                    for (int j = 0; j < C::FN; ++j)
                        acc[b][i][j] = mfma16x16x32(fb[j], fa[i], acc[b][i][j]);
            }
        }
        if (more) {
            la.stage(nxt);
            lb0.stage(nxt + C::A_BYTES);
            if constexpr (C::NB == 2) lb1.stage(nxt + C::A_BYTES + C::B_BYTES);
        }
        __syncthreads();
    }
}

// Placeholder loader for single-B GEMMs.
struct NoLoader {
    static constexpr bool MC = false;
    __device__ void fetch(int) {}
    __device__ void stage(char*) {}
};

// ---- grouped tile lookup ------------------------------------------------------------
// Tiles of expert e: ceil(M_e / BM) * NT, laid out expert after expert, with
// the M tile index running fastest (neighbouring tiles share a weight panel).
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
                               int bid, int BN, SlotTile& t) {
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
    const int mtiles = tiles;  // unused by other threads
    (void)mtiles;
    const int cnt = offsets[e + 1] - offsets[e];
    const int nmt = (cnt + BM - 1) / BM;
    const int mt = local % nmt;
    const int nt = local / nmt;
    t.e = e;
    t.off = offsets[e];
    t.m0 = mt * BM;
    t.mrows = min(BM, cnt - t.m0);
    t.n0 = nt * BN;
    return true;
}

}  // namespace moe
