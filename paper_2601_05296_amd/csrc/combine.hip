// combine.hip -- gate-weighted aggregation through token_index_map.
//
// MoEBlaze paper, Section 2.3 (y = sum_i g_i(x) E_i(x), only the k chosen
// experts contributing) carried out as in Section 3.1: each token finds its k
// expert outputs through the per-token slot list and reduces them directly
// into y, with no routed-token buffer. With unit weights the same kernel is the
// token gradient accumulation of Section 3.2, step 3.
//
// HBM-bound gather-reduce: one wave per token, 16-byte vector loads along d,
// all k source rows of a chunk in flight before the float32 accumulation,
// which adds the k terms in order j = 0..k-1.
#include "common.hpp"
#include "launch.hpp"
#include "probe.hpp"

namespace moe {
namespace {

constexpr int CMB_THREADS = 256;
constexpr int CMB_TOK = CMB_THREADS / WAVE;  // tokens per workgroup
constexpr int KMAX = 16;

template <bool F32>
__global__ void __launch_bounds__(CMB_THREADS)
combine_kernel(const void* __restrict__ src_, const float* __restrict__ w,
               const int32_t* __restrict__ tim, int64_t T, int d, int k, int accumulate,
               void* __restrict__ out_) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int64_t t = (int64_t)blockIdx.x * CMB_TOK + (threadIdx.x / WAVE);
    if (t >= T) return;
    constexpr int EPV = F32 ? 4 : 8;  // elements per 16-byte vector
    const int nchunk = d / EPV;
    int64_t row[KMAX];
    float g[KMAX];
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
        if (j < k) {
            row[j] = (int64_t)tim[t * k + j] * d;
            g[j] = w ? w[t * k + j] : 1.0f;
        }
    }
    const char* src = static_cast<const char*>(src_);
    char* out = static_cast<char*>(out_);
    const int esz = F32 ? 4 : 2;
    for (int c = lane; c < nchunk; c += WAVE) {
        uint4 v[KMAX];
#pragma unroll
        for (int j = 0; j < KMAX; ++j)
            if (j < k) v[j] = ld16(src + (row[j] + (int64_t)c * EPV) * esz);
        float acc[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
#pragma unroll
        for (int j = 0; j < KMAX; ++j) {
            if (j < k) {
                if (F32) {
                    acc[0] += g[j] * __uint_as_float(v[j].x);
                    acc[1] += g[j] * __uint_as_float(v[j].y);
                    acc[2] += g[j] * __uint_as_float(v[j].z);
                    acc[3] += g[j] * __uint_as_float(v[j].w);
                } else {
                    float f[8];
                    unpack8(v[j], f);
#pragma unroll
                    for (int i = 0; i < 8; ++i) acc[i] += g[j] * f[i];
                }
            }
        }
        char* dst = out + (t * d + (int64_t)c * EPV) * esz;
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

}  // namespace

hipError_t combine(const void* src, const float* w, const int32_t* tim, int64_t T, int d,
                   int k, bool f32, bool accumulate, void* out, hipStream_t st) {
    const dim3 grid((unsigned)((T + CMB_TOK - 1) / CMB_TOK));
    if (f32) {
        hipLaunchKernelGGL(combine_kernel<true>, grid, dim3(CMB_THREADS), 0, st, src, w, tim,
                           T, d, k, (int)accumulate, out);
        probe::mark("combine_f32", st);
    } else {
        hipLaunchKernelGGL(combine_kernel<false>, grid, dim3(CMB_THREADS), 0, st, src, w, tim,
                           T, d, k, (int)accumulate, out);
        probe::mark("combine", st);
    }
    return hipGetLastError();
}

}  // namespace moe
