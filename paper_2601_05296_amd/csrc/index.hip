// index.hip -- dispatch index maps without global atomics.
//
// Builds the data structures of the MoEBlaze paper, Section 4.1
// (expert_token_indices, expert_token_offsets, token_index_map, plus the
// per-expert lengths and the inverse slot map), following the three-step,
// atomic-free construction of Section 4.2, re-shaped for gfx950:
//
//   1. tile_hist:   each workgroup counts the expert choices of one tile of
//                   tokens with LDS counters and writes them expert-major to
//                   cnt[e][tile] (the expert lengths, split by tile). No dense
//                   [T, E] map is materialised: the per-tile counts carry the
//                   same information.
//   2. tile_scan:   one workgroup takes the exclusive prefix sum of cnt in
//                   expert-major order (wave-level scans over batches of
//                   16K entries). Entry (e, tile) then holds offsets[e] + (tokens
//                   of e in earlier tiles), i.e. the first slot of that
//                   tile's run inside expert e's segment.
//   3. tile_rank:   each workgroup revisits its tile in chunks of 64 tokens per
//                   wave. A lane sets its bit in an LDS 64-bit mask per chosen
//                   expert; the token's rank among the expert's tokens is the
//                   popcount of the lower lanes' bits plus the counts of
//                   earlier waves and chunks. Slots are therefore assigned in
//                   ascending token order inside every expert, as in the
//                   paper's worked example, and the result is deterministic.
//
// A choice whose id lies outside [0, E) or repeats an earlier id of its row
// (top-k never produces either) is rejected by both passes alike: it gets no
// slot and its token_index_map entry is -1. Every slot below offsets[E] is
// then written exactly once, whatever the ids hold.
#include <mutex>

#include "common.hpp"
#include "launch.hpp"
#include "probe.hpp"

// Scratch of the no-allocation index build (moe_build_index_noalloc): the
// per-tile expert counts of at most 256 experts x 1024 tiles. The workspace of
// moe_build_index never needs more for any T (the tile count is capped at
// 1024). Each GPU holds its own copy, at its own address, for the life of the
// process; calls that overlap on one GPU share it and race.
static __device__ __align__(256) int32_t scratch[256 * 1024];

namespace moe {
namespace {

constexpr int IDX_THREADS = 256;
constexpr int MAX_TILES = 1024;

// tokens per tile: a multiple of 256 keeping the number of tiles <= MAX_TILES
// does choice j of a row take a slot: its id is in [0, E) and differs from the
// ids of the row's earlier choices
__device__ inline bool choice_ok(const int32_t* row, int j, int E) {
    const int e = row[j];
    if ((unsigned)e >= (unsigned)E) return false;
    for (int i = 0; i < j; ++i)
        if (row[i] == e) return false;
    return true;
}

inline int64_t tile_tokens(int64_t T) {
    int64_t tb = (T + MAX_TILES - 1) / MAX_TILES;
    tb = ((tb + IDX_THREADS - 1) / IDX_THREADS) * IDX_THREADS;
    return tb < IDX_THREADS ? IDX_THREADS : tb;
}

__global__ void __launch_bounds__(IDX_THREADS)
tile_hist(const int32_t* __restrict__ ids, int64_t T, int E, int k, int64_t tb, int ntiles,
          int32_t* __restrict__ cnt) {
    __shared__ int32_t c[256];
    const int tid = threadIdx.x;
    const int b = blockIdx.x;
    for (int e = tid; e < E; e += IDX_THREADS) c[e] = 0;
    __syncthreads();
    const int64_t t_lo = (int64_t)b * tb;
    int64_t t_hi = t_lo + tb;
    if (t_hi > T) t_hi = T;
    for (int64_t t = t_lo + tid; t < t_hi; t += IDX_THREADS) {
        const int32_t* row = ids + t * k;
        for (int j = 0; j < k; ++j)
            if (choice_ok(row, j, E)) atomicAdd(&c[row[j]], 1);
    }
    __syncthreads();
    for (int e = tid; e < E; e += IDX_THREADS) cnt[(int64_t)e * ntiles + b] = c[e];
}

constexpr int SCAN_THREADS = 1024;

// One workgroup scans cnt (expert-major) in batches of SCAN_RB rounds of 1024
// consecutive entries. All loads of a batch are issued together; each wave
// scans its 64 entries of every round (wave-level scans), the batch's
// SCAN_RB x 16 wave totals, which lie in entry order, are scanned by the
// first four waves, and a carry runs from batch to batch.
constexpr int SCAN_RB = 16;

__global__ void __launch_bounds__(SCAN_THREADS)
tile_scan(int32_t* __restrict__ cnt, int E, int ntiles, int32_t* __restrict__ counts,
          int32_t* __restrict__ offsets) {
    constexpr int NW = SCAN_THREADS / WAVE;
    constexpr int NT = SCAN_RB * NW;            // wave totals per batch (256)
    static_assert(NT <= SCAN_THREADS && NT % WAVE == 0, "one thread per wave total");
    __shared__ int32_t wt[NT];                  // wave totals, then their exclusive prefix
    __shared__ int32_t wt_ex[NT];
    __shared__ int32_t part[NT / WAVE];         // totals of the four scanning waves
    const int tid = threadIdx.x;
    const int lane = tid & (WAVE - 1);
    const int wv = tid / WAVE;
    const int n = E * ntiles;
    int carry = 0;
    for (int b0 = 0; b0 < n; b0 += SCAN_RB * SCAN_THREADS) {
        int v[SCAN_RB], inc[SCAN_RB];
#pragma unroll
        for (int r = 0; r < SCAN_RB; ++r) {
            const int i = b0 + r * SCAN_THREADS + tid;
            v[r] = i < n ? cnt[i] : 0;
        }
        // rounds past the end hold zeros (the test is uniform over the workgroup)
#pragma unroll
        for (int r = 0; r < SCAN_RB; ++r) {
            inc[r] = b0 + r * SCAN_THREADS < n ? wave_incl_scan(v[r]) : 0;
            if (lane == WAVE - 1) wt[r * NW + wv] = inc[r];
        }
        __syncthreads();
        int x = 0, xi = 0;
        if (tid < NT) {                         // whole waves 0..3
            x = wt[tid];
            xi = wave_incl_scan(x);
            if (lane == WAVE - 1) part[wv] = xi;
        }
        __syncthreads();
        int total = 0, before = 0;
#pragma unroll
        for (int w = 0; w < NT / WAVE; ++w) {
            total += part[w];
            before += w < wv ? part[w] : 0;
        }
        if (tid < NT) wt_ex[tid] = before + xi - x;
        __syncthreads();
#pragma unroll
        for (int r = 0; r < SCAN_RB; ++r) {
            const int i = b0 + r * SCAN_THREADS + tid;
            if (i < n) cnt[i] = carry + wt_ex[r * NW + wv] + inc[r] - v[r];
        }
        carry += total;
        __syncthreads();                        // wt, wt_ex and part are reused
    }
    // carry is now the number of choices that take a slot
    for (int e = tid; e <= E; e += SCAN_THREADS) offsets[e] = e < E ? cnt[e * ntiles] : carry;
    for (int e = tid; e < E; e += SCAN_THREADS)
        counts[e] = (e + 1 < E ? cnt[(e + 1) * ntiles] : carry) - cnt[e * ntiles];
}

__global__ void __launch_bounds__(IDX_THREADS)
tile_rank(const int32_t* __restrict__ ids, int64_t T, int E, int k, int64_t tb, int ntiles,
          const int32_t* __restrict__ base, int32_t* __restrict__ eti,
          int32_t* __restrict__ tim, int32_t* __restrict__ slot_src) {
    __shared__ int32_t run[256];
    __shared__ unsigned long long mask[IDX_THREADS / WAVE][256];
    __shared__ int32_t chunk_ids[IDX_THREADS * 16];
    __shared__ int32_t chunk_tim[IDX_THREADS * 16];
    const int tid = threadIdx.x;
    const int lane = tid & (WAVE - 1);
    const int wv = tid / WAVE;
    const int b = blockIdx.x;
    for (int e = tid; e < E; e += IDX_THREADS) run[e] = base[(int64_t)e * ntiles + b];
    const int64_t t_lo = (int64_t)b * tb;
    int64_t t_hi = t_lo + tb;
    if (t_hi > T) t_hi = T;
    const unsigned long long below = (1ull << lane) - 1ull;
    for (int64_t c0 = t_lo; c0 < t_hi; c0 += IDX_THREADS) {
        const int nt = (int)min((int64_t)IDX_THREADS, t_hi - c0);
        for (int e = tid; e < E; e += IDX_THREADS)
#pragma unroll
            for (int w = 0; w < IDX_THREADS / WAVE; ++w) mask[w][e] = 0ull;
        for (int i = tid; i < nt * k; i += IDX_THREADS) chunk_ids[i] = ids[c0 * k + i];
        __syncthreads();
        const bool valid = tid < nt;
        unsigned ok = 0;   // bit j: choice j of this lane's token takes a slot
        if (valid)
            for (int j = 0; j < k; ++j)
                if (choice_ok(chunk_ids + tid * k, j, E)) {
                    ok |= 1u << j;
                    atomicOr(&mask[wv][chunk_ids[tid * k + j]], 1ull << lane);
                }
        __syncthreads();
        if (valid) {
            const int64_t t = c0 + tid;
            for (int j = 0; j < k; ++j) {
                if (!((ok >> j) & 1u)) {
                    chunk_tim[tid * k + j] = -1;
                    continue;
                }
                const int e = chunk_ids[tid * k + j];
                int r = run[e] + __popcll(mask[wv][e] & below);
                for (int w = 0; w < wv; ++w) r += __popcll(mask[w][e]);
                eti[r] = (int32_t)t;
                slot_src[r] = (int32_t)(t * k + j);
                chunk_tim[tid * k + j] = r;
            }
        }
        __syncthreads();
        for (int e = tid; e < E; e += IDX_THREADS) {
            int add = 0;
#pragma unroll
            for (int w = 0; w < IDX_THREADS / WAVE; ++w) add += __popcll(mask[w][e]);
            run[e] += add;
        }
        for (int i = tid; i < nt * k; i += IDX_THREADS) tim[c0 * k + i] = chunk_tim[i];
        __syncthreads();
    }
}

}  // namespace

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept. In host code the array's name
// is only a stand-in for the symbol: kernels must be given this address.
namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES];
}  // namespace

hipError_t noalloc_scratch(void** ptr, size_t* bytes) {
    int dev = -1;
    if (hipError_t e = hipGetDevice(&dev); e != hipSuccess) return e;
    if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)); e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    *bytes = sizeof(scratch);
    return hipSuccess;
}

size_t build_index_workspace(int64_t T, int E, int k) {
    (void)k;
    const int64_t tb = tile_tokens(T);
    const int64_t ntiles = (T + tb - 1) / tb;
    return (size_t)(E * ntiles * (int64_t)sizeof(int32_t));
}

hipError_t build_index(const int32_t* ids, int64_t T, int E, int k, int32_t* counts,
                       int32_t* offsets, int32_t* eti, int32_t* tim, int32_t* slot_src,
                       void* ws, hipStream_t st) {
    const int64_t tb = tile_tokens(T);
    const int ntiles = (int)((T + tb - 1) / tb);
    int32_t* cnt = static_cast<int32_t*>(ws);
    hipLaunchKernelGGL(tile_hist, dim3(ntiles), dim3(IDX_THREADS), 0, st, ids, T, E, k, tb,
                       ntiles, cnt);
    probe::mark("tile_hist", st);
    hipLaunchKernelGGL(tile_scan, dim3(1), dim3(SCAN_THREADS), 0, st, cnt, E, ntiles, counts,
                       offsets);
    probe::mark("tile_scan", st);
    hipLaunchKernelGGL(tile_rank, dim3(ntiles), dim3(IDX_THREADS), 0, st, ids, T, E, k, tb,
                       ntiles, cnt, eti, tim, slot_src);
    probe::mark("tile_rank", st);
    return hipGetLastError();
}

}  // namespace moe
