// route_bwd.hip -- router backward. The MoEBlaze paper states the gating
// forward (Section 2.1) but not its gradient; this is the closed form of the
// softmax Jacobian restricted to the top-k gates:
//   no renorm: g_j = p[id_j]            dl = p * (dp - sum_j g_j dg_j)
//   renorm:    g_j = p[id_j]/sum p[id]  dl[id_j] = g_j (dg_j - sum_j' g_j' dg_j')
// followed by dW_g = dl^T x and dx += dl W_g.
//
// Kernels: (1) one wave per token computes dl [T,E] into the workspace;
// (2) dx: each workgroup keeps the dl rows of 32 tokens in LDS and streams
// W_g column blocks (W_g is read once per 32 tokens); (3) dW_g: split over
// token chunks, each workgroup accumulating 32 experts x 256 columns, then
// (4) a fixed-order sum of the chunk partials. Float32 FMA throughout.
#include "common.hpp"
#include "launch.hpp"
#include "probe.hpp"

namespace moe {
namespace {

constexpr int RB_TOK = 32;     // tokens per workgroup in the dx kernel
constexpr int RB_CHUNK = 1024; // tokens per split in the dW_g kernel
constexpr int RB_EB = 32;      // experts per workgroup in the dW_g kernel

__global__ void __launch_bounds__(256)
rb_dlogits(const float* __restrict__ dg, const float* __restrict__ logits,
           const int32_t* __restrict__ ids, const float* __restrict__ gates, int64_t T, int E,
           int k, int renorm, float* __restrict__ dl) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;
    float gdg = 0.f;
    for (int j = 0; j < k; ++j) gdg += gates[t * k + j] * dg[t * k + j];
    float* out = dl + t * E;
    if (renorm) {
        for (int e = lane; e < E; e += 64) {
            float v = 0.f;
            for (int j = 0; j < k; ++j)
                if (ids[t * k + j] == e) v = gates[t * k + j] * (dg[t * k + j] - gdg);
            out[e] = v;
        }
        return;
    }
    const float* lt = logits + t * E;
    float mx = -INFINITY;
    for (int e = lane; e < E; e += 64) mx = fmaxf(mx, lt[e]);
    mx = wave_max(mx);
    float z = 0.f;
    for (int e = lane; e < E; e += 64) z += __expf(lt[e] - mx);
    z = wave_sum(z);
    for (int e = lane; e < E; e += 64) {
        float dp = 0.f;
        for (int j = 0; j < k; ++j)
            if (ids[t * k + j] == e) dp = dg[t * k + j];
        out[e] = (__expf(lt[e] - mx) / z) * (dp - gdg);
    }
}

template <bool F32>
__global__ void __launch_bounds__(256)
rb_dx(const float* __restrict__ dl, const void* __restrict__ wg_, int64_t T, int d, int E,
      int accumulate, void* __restrict__ dx_) {
    __shared__ float s_dl[RB_TOK][256];
    const int tid = threadIdx.x;
    const int64_t t0 = (int64_t)blockIdx.x * RB_TOK;
    const int nt = (int)min((int64_t)RB_TOK, T - t0);
    for (int i = tid; i < RB_TOK * E; i += 256) {
        const int tt = i / E, e = i % E;
        s_dl[tt][e] = tt < nt ? dl[(t0 + tt) * E + e] : 0.f;
    }
    __syncthreads();
    for (int c = tid; c < d; c += 256) {
        float acc[RB_TOK];
#pragma unroll
        for (int tt = 0; tt < RB_TOK; ++tt) acc[tt] = 0.f;
        for (int e = 0; e < E; ++e) {
            float w;
            if (F32) w = static_cast<const float*>(wg_)[(int64_t)e * d + c];
            else w = bf2f(static_cast<const bf16_t*>(wg_)[(int64_t)e * d + c]);
#pragma unroll
            for (int tt = 0; tt < RB_TOK; ++tt) acc[tt] = fmaf(s_dl[tt][e], w, acc[tt]);
        }
        for (int tt = 0; tt < nt; ++tt) {
            const int64_t o = (t0 + tt) * d + c;
            if (F32) {
                float* p = static_cast<float*>(dx_) + o;
                *p = accumulate ? *p + acc[tt] : acc[tt];
            } else {
                bf16_t* p = static_cast<bf16_t*>(dx_) + o;
                const float v = accumulate ? bf2f(*p) + acc[tt] : acc[tt];
                *p = (bf16_t)f2bf(v);
            }
        }
    }
}

template <bool F32>
__global__ void __launch_bounds__(256)
rb_dwg_partial(const float* __restrict__ dl, const void* __restrict__ x_, int64_t T, int d,
               int E, float* __restrict__ part) {
    __shared__ float s_dl[64][RB_EB];
    const int tid = threadIdx.x;
    const int c = blockIdx.x * 256 + tid;
    const int e0 = blockIdx.y * RB_EB;
    const int split = blockIdx.z;
    const int64_t tlo = (int64_t)split * RB_CHUNK;
    const int64_t thi = min(T, tlo + RB_CHUNK);
    float acc[RB_EB];
#pragma unroll
    for (int i = 0; i < RB_EB; ++i) acc[i] = 0.f;
    for (int64_t tb = tlo; tb < thi; tb += 64) {
        __syncthreads();
        for (int i = tid; i < 64 * RB_EB; i += 256) {
            const int tt = i / RB_EB, ee = i % RB_EB;
            const int64_t t = tb + tt;
            s_dl[tt][ee] = (t < thi && e0 + ee < E) ? dl[t * E + e0 + ee] : 0.f;
        }
        __syncthreads();
        const int ntt = (int)min((int64_t)64, thi - tb);
        if (c < d) {
            for (int tt = 0; tt < ntt; ++tt) {
                const int64_t o = (tb + tt) * d + c;
                const float xv = F32 ? static_cast<const float*>(x_)[o]
                                     : bf2f(static_cast<const bf16_t*>(x_)[o]);
#pragma unroll
                for (int ee = 0; ee < RB_EB; ++ee) acc[ee] = fmaf(s_dl[tt][ee], xv, acc[ee]);
            }
        }
    }
    if (c < d)
        for (int ee = 0; ee < RB_EB && e0 + ee < E; ++ee)
            part[((int64_t)split * E + e0 + ee) * d + c] = acc[ee];
}

__global__ void rb_dwg_reduce(const float* __restrict__ part, int nsplit, int E, int d,
                              float* __restrict__ dwg) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t n = (int64_t)E * d;
    if (i >= n) return;
    float acc = 0.f;
    for (int s = 0; s < nsplit; ++s) acc += part[s * n + i];
    dwg[i] = acc;
}

inline int nsplits(int64_t T) { return (int)((T + RB_CHUNK - 1) / RB_CHUNK); }

}  // namespace

size_t route_bwd_workspace(int64_t T, int d, int E, int k, bool f32) {
    (void)k; (void)f32;
    const size_t dl = (size_t)T * E * sizeof(float);
    const size_t part = (size_t)nsplits(T) * E * d * sizeof(float);
    return ((dl + 255) / 256) * 256 + part;
}

hipError_t route_bwd(const float* dgates, const float* logits, const int32_t* ids,
                     const float* gates, const void* x, const void* wg, int64_t T, int d,
                     int E, int k, bool f32, bool renorm, bool accumulate, float* dwg,
                     void* dx, void* ws, hipStream_t st) {
    float* dl = static_cast<float*>(ws);
    const size_t dl_bytes = (((size_t)T * E * sizeof(float) + 255) / 256) * 256;
    float* part = reinterpret_cast<float*>(static_cast<char*>(ws) + dl_bytes);
    hipLaunchKernelGGL(rb_dlogits, dim3((unsigned)((T + 3) / 4)), dim3(256), 0, st, dgates,
                       logits, ids, gates, T, E, k, (int)renorm, dl);
    probe::mark("rb_dlogits", st);
    const dim3 gdx((unsigned)((T + RB_TOK - 1) / RB_TOK));
    const int ns = nsplits(T);
    const dim3 gdw((unsigned)((d + 255) / 256), (unsigned)((E + RB_EB - 1) / RB_EB), (unsigned)ns);
    if (f32) {
        hipLaunchKernelGGL(rb_dx<true>, gdx, dim3(256), 0, st, dl, wg, T, d, E, (int)accumulate, dx);
        probe::mark("rb_dx", st);
        hipLaunchKernelGGL(rb_dwg_partial<true>, gdw, dim3(256), 0, st, dl, x, T, d, E, part);
        probe::mark("rb_dwg_partial", st);
    } else {
        hipLaunchKernelGGL(rb_dx<false>, gdx, dim3(256), 0, st, dl, wg, T, d, E, (int)accumulate, dx);
        probe::mark("rb_dx", st);
        hipLaunchKernelGGL(rb_dwg_partial<false>, gdw, dim3(256), 0, st, dl, x, T, d, E, part);
        probe::mark("rb_dwg_partial", st);
    }
    hipLaunchKernelGGL(rb_dwg_reduce, dim3((unsigned)(((int64_t)E * d + 255) / 256)), dim3(256), 0,
                       st, part, ns, E, d, dwg);
    probe::mark("rb_dwg_reduce", st);
    return hipGetLastError();
}

}  // namespace moe
