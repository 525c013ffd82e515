// combine.hip -- gate-weighted aggregation through token_index_map.
//
// MoEBlaze paper, Section 2.3 (y = sum_i g_i(x) E_i(x), only the k chosen
// experts contributing) carried out as in Section 3.1: each token finds its k
// expert outputs through the per-token slot list and reduces them directly
// into y, with no routed-token buffer. With unit weights the same kernel is the
// token gradient accumulation of Section 3.2, step 3.
//
// HBM-bound gather-reduce: one workgroup per token (several for narrow column
// strips), 16-byte vector loads along d, all k source rows of a chunk in
// flight before the float32 accumulation, which adds the k terms in order
// j = 0..k-1. A token_index_map entry of -1 (a choice the index build
// rejected) adds nothing.
#include "common.hpp"
#include "launch.hpp"
#include "probe.hpp"

namespace moe {
namespace {

constexpr int CMB_THREADS = 256;

// A workgroup handles TPB tokens (TPB = 256 / LPT) with LPT lanes per token;
// lane c owns 16-byte column chunks c, c + LPT, ... of its token's ncols
// columns. Source rows are src_ld elements apart and output rows out_ld, so
// the kernel also combines one column strip of a wider matrix. The token's k
// slot rows and weights are read once; all k source chunks of a lane are
// loaded before the float32 sum, which runs in order j = 0..k-1. KMAX >= k
// sizes the per-lane arrays: the smallest bound that fits keeps the register
// count, and with it the number of loads in flight per CU, where it belongs
// (KMAX = 16 would hold 135 VGPRs and three waves per SIMD for any k).
template <bool F32, int NC, int KMAX>
__global__ void __launch_bounds__(CMB_THREADS)
combine_kernel(const void* __restrict__ src_, int64_t src_ld, const float* __restrict__ w,
               const int32_t* __restrict__ tim, int64_t T, int ncols, int k, int accumulate,
               void* __restrict__ out_, int64_t out_ld, int lpt_log2) {
    const int lpt = 1 << lpt_log2;
    const int64_t t = (int64_t)blockIdx.x * (CMB_THREADS >> lpt_log2) + (threadIdx.x >> lpt_log2);
    const int lane = threadIdx.x & (lpt - 1);
    if (t >= T) return;
    constexpr int EPV = F32 ? 4 : 8;  // elements per 16-byte vector
    const int nchunk = ncols / EPV;
    int64_t row[KMAX];
    float g[KMAX];
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
        if (j < k) {
            const int32_t slot = tim[t * k + j];
            row[j] = slot < 0 ? -1 : (int64_t)slot * src_ld;
            g[j] = w ? w[t * k + j] : 1.0f;
        }
    }
    const char* src = static_cast<const char*>(src_);
    char* out = static_cast<char*>(out_);
    const int esz = F32 ? 4 : 2;
    for (int c0 = 0; c0 < nchunk; c0 += NC * lpt) {
        uint4 v[NC][KMAX];
#pragma unroll
        for (int u = 0; u < NC; ++u) {
            const int c = c0 + u * lpt + lane;
#pragma unroll
            for (int j = 0; j < KMAX; ++j)
                if (j < k && c < nchunk && row[j] >= 0)
                {
                    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
                    const u32x4 x = __builtin_nontemporal_load(
                        reinterpret_cast<const u32x4*>(src + (row[j] + (int64_t)c * EPV) * esz));
                    v[u][j] = make_uint4(x[0], x[1], x[2], x[3]);
                }
        }
#pragma unroll
        for (int u = 0; u < NC; ++u) {
            const int c = c0 + u * lpt + lane;
            if (c >= nchunk) continue;
            float acc[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
#pragma unroll
            for (int j = 0; j < KMAX; ++j) {
                if (j < k && row[j] >= 0) {
                    if (F32) {
                        acc[0] += g[j] * __uint_as_float(v[u][j].x);
                        acc[1] += g[j] * __uint_as_float(v[u][j].y);
                        acc[2] += g[j] * __uint_as_float(v[u][j].z);
                        acc[3] += g[j] * __uint_as_float(v[u][j].w);
                    } else {
                        float f[8];
                        unpack8(v[u][j], f);
#pragma unroll
                        for (int i = 0; i < 8; ++i) acc[i] += g[j] * f[i];
                    }
                }
            }
            char* dst = out + (t * out_ld + (int64_t)c * EPV) * esz;
            if (accumulate) {
                const uint4 o = ld16(dst);
                if (F32) {
                    acc[0] += __uint_as_float(o.x); acc[1] += __uint_as_float(o.y);
                    acc[2] += __uint_as_float(o.z); acc[3] += __uint_as_float(o.w);
                } else {
                    float f[8];
                    unpack8(o, f);
#pragma unroll
                    for (int i = 0; i < 8; ++i) acc[i] += f[i];
                }
            }
            if (F32)
                st16(dst, make_uint4(__float_as_uint(acc[0]), __float_as_uint(acc[1]),
                                     __float_as_uint(acc[2]), __float_as_uint(acc[3])));
            else
                st16(dst, pack8(acc));
        }
    }
}

template <int KMAX>
void launch_combine(const void* src, int64_t src_ld, const float* w, const int32_t* tim,
                    int64_t T, int ncols, int k, bool f32, bool accumulate, void* out,
                    int64_t out_ld, hipStream_t st) {
    const int nchunk = ncols / (f32 ? 4 : 8);
    // lanes per token: the smallest power of two covering the row's chunks
    // (at most the whole workgroup; wider rows loop). A row whose chunk count
    // is not a power of two, or a token with more than four sources, takes at
    // most one wave per token instead, so that no lane idles and each lane
    // keeps more source loads in flight (measured faster on both).
    const bool pow2 = (nchunk & (nchunk - 1)) == 0;
    const int cap = (!pow2 || k > 4) ? WAVE : CMB_THREADS;
    int lpt_log2 = 0;
    while ((1 << lpt_log2) < nchunk && (1 << lpt_log2) < cap) ++lpt_log2;
    const int64_t tpb = CMB_THREADS >> lpt_log2;
    const dim3 grid((unsigned)((T + tpb - 1) / tpb));
    if (f32) {
        hipLaunchKernelGGL((combine_kernel<true, 2, KMAX>), grid, dim3(CMB_THREADS), 0, st, src,
                           src_ld, w, tim, T, ncols, k, (int)accumulate, out, out_ld, lpt_log2);
        probe::mark("combine_f32", st);
    } else if (nchunk <= (1 << lpt_log2) || k > 4) {
        hipLaunchKernelGGL((combine_kernel<false, 1, KMAX>), grid, dim3(CMB_THREADS), 0, st, src,
                           src_ld, w, tim, T, ncols, k, (int)accumulate, out, out_ld, lpt_log2);
        probe::mark("combine", st);
    } else {
        hipLaunchKernelGGL((combine_kernel<false, 2, KMAX>), grid, dim3(CMB_THREADS), 0, st, src,
                           src_ld, w, tim, T, ncols, k, (int)accumulate, out, out_ld, lpt_log2);
        probe::mark("combine", st);
    }
}

}  // namespace

hipError_t combine_cols(const void* src, int64_t src_ld, const float* w, const int32_t* tim,
                        int64_t T, int ncols, int k, bool f32, bool accumulate, void* out,
                        int64_t out_ld, hipStream_t st) {
    if (k <= 4)
        launch_combine<4>(src, src_ld, w, tim, T, ncols, k, f32, accumulate, out, out_ld, st);
    else if (k <= 8)
        launch_combine<8>(src, src_ld, w, tim, T, ncols, k, f32, accumulate, out, out_ld, st);
    else
        launch_combine<16>(src, src_ld, w, tim, T, ncols, k, f32, accumulate, out, out_ld, st);
    return hipGetLastError();
}

hipError_t combine(const void* src, const float* w, const int32_t* tim, int64_t T, int d,
                   int k, bool f32, bool accumulate, void* out, hipStream_t st) {
    return combine_cols(src, d, w, tim, T, d, k, f32, accumulate, out, d, st);
}

}  // namespace moe
