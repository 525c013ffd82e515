// route.hip -- top-k softmax gating, forward (MoEBlaze paper, Section 2.1:
// topk_experts = TopK(softmax(W_g x)), gate weights of Section 2.3).
//
// bf16 path: the router product logits[T,E] = x W_g^T is a skinny GEMM
// (E <= 256 columns) whose cost is reading x once from HBM, so it runs on the
// matrix cores: each wave owns 16 tokens and all E experts, x fragments are
// loaded straight from global memory (every x element is read exactly once)
// and W_g is staged through LDS in 64-wide K slices shared by the 4 waves of a
// workgroup, double-buffered: the next slice's W_g and x are in flight while
// the current one is multiplied. Softmax and the top-k selection run on the accumulators in
// registers: the 4 lanes holding one token's logits find the k largest by k
// rounds of (local best, two cross-lane exchanges), ties going to the lower
// expert id.
//
// f32 path (debug mode): one thread per token, float32 FMA.
#include "common.hpp"
#include "launch.hpp"
#include "probe.hpp"

namespace moe {
namespace {

constexpr int RT_THREADS = 256;
constexpr int RT_TOK = 64;   // tokens per workgroup (16 per wave)
constexpr int RT_BK = 64;    // K slice staged in LDS

// LDS offset (bytes) of 16-byte chunk `c` (0..7) of row `r` in a row-major
// [rows][64] bf16 tile; the chunk index is XOR-swizzled with the row so that
// the 16 rows read by one fragment load hit distinct banks.
__device__ __forceinline__ int kc64_off(int r, int c) { return r * 128 + ((c ^ (r & 7)) << 4); }

template <int NE>  // number of 16-expert fragments, E <= 16*NE
__global__ void __launch_bounds__(RT_THREADS)
route_bf16(const bf16_t* __restrict__ x, const bf16_t* __restrict__ wg,
           const float* __restrict__ bias, int64_t T, int d, int E, int k, int renorm,
           int32_t* __restrict__ ids, float* __restrict__ gates, float* __restrict__ logits) {
    extern __shared__ __align__(16) char lds[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = tid >> 6;
    const int grp = lane >> 4;    // which 4-column group of each 16-expert fragment
    const int col = lane & 15;    // token within the wave's 16
    const int64_t t0 = (int64_t)blockIdx.x * RT_TOK + wv * 16;
    int64_t trow = t0 + col;
    if (trow >= T) trow = T - 1;  // clamp: valid memory, result discarded
    const bf16_t* xrow = x + trow * d;

    f32x4 acc[NE];
#pragma unroll
    for (int i = 0; i < NE; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int Ep = NE * 16;
    const int nchunks = Ep * 8;  // 16-byte chunks of one W_g slice
    constexpr int WPT = (NE * 16 * 8 + RT_THREADS - 1) / RT_THREADS;  // chunks per thread
    // software pipeline: the W_g slice and the x fragments of slice s+1 are
    // loaded into registers while slice s is multiplied; W_g alternates
    // between two LDS buffers
    uint4 wreg[WPT], xreg[2];
    auto load_w = [&](int k0) {
#pragma unroll
        for (int i = 0; i < WPT; ++i) {
            const int c = tid + i * RT_THREADS;
            const int r = c >> 3, cc = c & 7;
            wreg[i] = (c < nchunks && r < E) ? ld16(wg + (int64_t)r * d + k0 + cc * 8) : zero16();
        }
    };
    auto store_w = [&](char* buf) {
#pragma unroll
        for (int i = 0; i < WPT; ++i) {
            const int c = tid + i * RT_THREADS;
            if (c < nchunks) st16(buf + kc64_off(c >> 3, c & 7), wreg[i]);
        }
    };
    auto load_x = [&](int k0) {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) xreg[kk] = ld16(xrow + k0 + kk * 32 + grp * 8);
    };
    char* const buf1 = lds + Ep * 128;
    load_w(0);
    load_x(0);
    store_w(lds);
    __syncthreads();
    for (int k0 = 0, s = 0; k0 < d; k0 += RT_BK, ++s) {
        const char* cur = (s & 1) ? buf1 : lds;
        const uint4 xc0 = xreg[0], xc1 = xreg[1];
        const bool more = k0 + RT_BK < d;
        if (more) {
            load_w(k0 + RT_BK);
            load_x(k0 + RT_BK);
        }
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const bf16x8 q = __builtin_bit_cast(bf16x8, kk ? xc1 : xc0);
#pragma unroll
            for (int fe = 0; fe < NE; ++fe) {
                const bf16x8 p = *reinterpret_cast<const bf16x8*>(
                    cur + kc64_off(fe * 16 + col, kk * 4 + grp));
                acc[fe] = mfma16x16x32(p, q, acc[fe]);
            }
        }
        if (more) store_w((s & 1) ? lds : buf1);
        __syncthreads();
    }
    // lane holds logits of token t0+col, experts fe*16 + 4*grp + r
    const int64_t t = t0 + col;
    const bool tvalid = t < T;
    float v[NE * 4];
#pragma unroll
    for (int fe = 0; fe < NE; ++fe)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int e = fe * 16 + grp * 4 + r;
            float l = acc[fe][r];
            if (e < E) {
                if (bias) l += bias[e];
                if (logits && tvalid) logits[t * E + e] = l;
            }
            v[fe * 4 + r] = l;
        }
    // softmax statistics over all E experts
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < NE * 4; ++i) {
        const int e = (i >> 2) * 16 + grp * 4 + (i & 3);
        if (e < E) mx = fmaxf(mx, v[i]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float z = 0.f;
#pragma unroll
    for (int i = 0; i < NE * 4; ++i) {
        const int e = (i >> 2) * 16 + grp * 4 + (i & 3);
        if (e < E) z += __expf(v[i] - mx);
    }
    z += __shfl_xor(z, 16, 64);
    z += __shfl_xor(z, 32, 64);
    // top-k: k rounds of argmax over the untaken experts
    unsigned long long taken = 0ull;
    float selv[16];
    int sele[16];
    float ssum = 0.f;
    for (int j = 0; j < k; ++j) {
        float bv = -INFINITY;
        int be = 0x7fffffff;
#pragma unroll
        for (int i = 0; i < NE * 4; ++i) {
            const int e = (i >> 2) * 16 + grp * 4 + (i & 3);
            const bool ok = e < E && !((taken >> i) & 1ull);
            if (ok && (v[i] > bv || (v[i] == bv && e < be))) { bv = v[i]; be = e; }
        }
#pragma unroll
        for (int o = 16; o <= 32; o <<= 1) {
            const float ov = __shfl_xor(bv, o, 64);
            const int oe = __shfl_xor(be, o, 64);
            if (ov > bv || (ov == bv && oe < be)) { bv = ov; be = oe; }
        }
        // the owner lane of expert be marks it taken
        if (((be & 15) >> 2) == grp) taken |= 1ull << ((be >> 4) * 4 + (be & 3));
        selv[j] = bv;
        sele[j] = be;
        ssum += __expf(bv - mx);
    }
    if (grp == 0 && tvalid) {
        for (int j = 0; j < k; ++j) {
            const float pe = __expf(selv[j] - mx);
            ids[t * k + j] = sele[j];
            gates[t * k + j] = renorm ? pe / ssum : pe / z;
        }
    }
}

__global__ void route_f32(const float* __restrict__ x, const float* __restrict__ wg,
                          const float* __restrict__ bias, int64_t T, int d, int E, int k,
                          int renorm, int32_t* __restrict__ ids, float* __restrict__ gates,
                          float* __restrict__ logits) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= T) return;
    float l[256];
    float mx = -INFINITY;
    for (int e = 0; e < E; ++e) {
        float a = 0.f;
        for (int i = 0; i < d; ++i) a = fmaf(x[t * d + i], wg[(int64_t)e * d + i], a);
        if (bias) a += bias[e];
        l[e] = a;
        if (logits) logits[t * E + e] = a;
        mx = fmaxf(mx, a);
    }
    float z = 0.f;
    for (int e = 0; e < E; ++e) z += __expf(l[e] - mx);
    unsigned long long taken[4] = {0ull, 0ull, 0ull, 0ull};
    float pe[16];
    float ssum = 0.f;
    for (int j = 0; j < k; ++j) {
        int be = -1;
        float bv = 0.f;
        for (int e = 0; e < E; ++e) {
            if ((taken[e >> 6] >> (e & 63)) & 1ull) continue;
            if (be < 0 || l[e] > bv) { be = e; bv = l[e]; }
        }
        taken[be >> 6] |= 1ull << (be & 63);
        ids[t * k + j] = be;
        pe[j] = __expf(bv - mx);
        ssum += pe[j];
    }
    for (int j = 0; j < k; ++j) gates[t * k + j] = renorm ? pe[j] / ssum : pe[j] / z;
}

template <int NE>
hipError_t launch_route_bf16(const void* x, const void* wg, const float* bias, int64_t T,
                             int d, int E, int k, bool renorm, int32_t* ids, float* gates,
                             float* logits, hipStream_t st) {
    const dim3 grid((unsigned)((T + RT_TOK - 1) / RT_TOK));
    const size_t lds = (size_t)2 * NE * 16 * 128;   // two W_g slices
    hipLaunchKernelGGL(route_bf16<NE>, grid, dim3(RT_THREADS), lds, st,
                       static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(wg), bias, T,
                       d, E, k, (int)renorm, ids, gates, logits);
    probe::mark("route_bf16", st);
    return hipGetLastError();
}

}  // namespace

hipError_t route(const void* x, const void* wg, const float* bias, int64_t T, int d, int E,
                 int k, bool f32, bool renorm, int32_t* ids, float* gates, float* logits,
                 hipStream_t st) {
    if (f32) {
        const dim3 grid((unsigned)((T + 127) / 128));
        hipLaunchKernelGGL(route_f32, grid, dim3(128), 0, st, static_cast<const float*>(x),
                           static_cast<const float*>(wg), bias, T, d, E, k, (int)renorm, ids,
                           gates, logits);
        probe::mark("route_f32", st);
        return hipGetLastError();
    }
    if (E <= 16) return launch_route_bf16<1>(x, wg, bias, T, d, E, k, renorm, ids, gates, logits, st);
    if (E <= 32) return launch_route_bf16<2>(x, wg, bias, T, d, E, k, renorm, ids, gates, logits, st);
    if (E <= 64) return launch_route_bf16<4>(x, wg, bias, T, d, E, k, renorm, ids, gates, logits, st);
    if (E <= 128) return launch_route_bf16<8>(x, wg, bias, T, d, E, k, renorm, ids, gates, logits, st);
    return launch_route_bf16<16>(x, wg, bias, T, d, E, k, renorm, ids, gates, logits, st);
}

}  // namespace moe
