// combine.hip -- gate-weighted aggregation through token_index_map.
//
// MoEBlaze paper, Section 2.3 (y = sum_i g_i(x) E_i(x), only the k chosen
// experts contributing) carried out as in Section 3.1: each token finds its k
// expert outputs through the per-token slot list and reduces them directly
// into y, with no routed-token buffer. With unit weights the same kernel is the
// token gradient accumulation of Section 3.2, step 3.
//
// HBM-bound gather-reduce: one workgroup per token, 16-byte vector loads
// along d, all k source rows of a chunk in flight before the float32
// accumulation, which adds the k terms in order j = 0..k-1.
#include "common.hpp"
#include "launch.hpp"
#include "probe.hpp"

namespace moe {
namespace {

constexpr int CMB_THREADS = 256;
constexpr int KMAX = 16;

// One workgroup per token; thread c owns 16-byte column chunks c and c + 256
// (d <= 4096 bf16 / 2048 float32 per pass; wider rows loop). The token's k
// slot rows and weights are wave-uniform (scalar loads); all k source chunks
// of a thread are loaded before the float32 sum, which runs in order j = 0..k-1.
template <bool F32, int NC>
__global__ void __launch_bounds__(CMB_THREADS)
combine_kernel(const void* __restrict__ src_, const float* __restrict__ w,
               const int32_t* __restrict__ tim, int64_t T, int d, int k, int accumulate,
               void* __restrict__ out_) {
    const int64_t t = blockIdx.x;
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
    for (int c0 = 0; c0 < nchunk; c0 += NC * CMB_THREADS) {
        uint4 v[NC][KMAX];
#pragma unroll
        for (int u = 0; u < NC; ++u) {
            const int c = c0 + u * CMB_THREADS + threadIdx.x;
#pragma unroll
            for (int j = 0; j < KMAX; ++j)
                if (j < k && c < nchunk)
                {
                    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
                    const u32x4 x = __builtin_nontemporal_load(
                        reinterpret_cast<const u32x4*>(src + (row[j] + (int64_t)c * EPV) * esz));
                    v[u][j] = make_uint4(x[0], x[1], x[2], x[3]);
                }
        }
#pragma unroll
        for (int u = 0; u < NC; ++u) {
            const int c = c0 + u * CMB_THREADS + threadIdx.x;
            if (c >= nchunk) continue;
            float acc[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] = 0.0f;
#pragma unroll
            for (int j = 0; j < KMAX; ++j) {
                if (j < k) {
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
}

}  // namespace

hipError_t combine(const void* src, const float* w, const int32_t* tim, int64_t T, int d,
                   int k, bool f32, bool accumulate, void* out, hipStream_t st) {
    const dim3 grid((unsigned)T);
    const int nchunk = d / (f32 ? 4 : 8);
    if (f32) {
        hipLaunchKernelGGL((combine_kernel<true, 2>), grid, dim3(CMB_THREADS), 0, st, src, w, tim,
                           T, d, k, (int)accumulate, out);
        probe::mark("combine_f32", st);
    } else if (nchunk <= CMB_THREADS) {
        hipLaunchKernelGGL((combine_kernel<false, 1>), grid, dim3(CMB_THREADS), 0, st, src, w,
                           tim, T, d, k, (int)accumulate, out);
        probe::mark("combine", st);
    } else {
        hipLaunchKernelGGL((combine_kernel<false, 2>), grid, dim3(CMB_THREADS), 0, st, src, w,
                           tim, T, d, k, (int)accumulate, out);
        probe::mark("combine", st);
    }
    return hipGetLastError();
}

}  // namespace moe
