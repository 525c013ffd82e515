// route_bwd.hip -- router backward. The MoEBlaze paper states the gating
// forward (Section 2.1) but not its gradient; this is the closed form of the
// softmax Jacobian restricted to the top-k gates:
//   no renorm: g_j = p[id_j]            dl = p * (dp - sum_j g_j dg_j)
//   renorm:    g_j = p[id_j]/sum p[id]  dl[id_j] = g_j (dg_j - sum_j' g_j' dg_j')
// followed by dW_g = dl^T x and dx += dl W_g.
//
// bf16 path: one wave per token computes dl and stores it as two bf16 terms
// dl = hi + lo (hi = bf16(dl), lo = bf16(dl - hi); relative error about
// 2^-16), laid out [T][2Ep] with Ep = E rounded up to 32 (zero padding). Both
// products then run on the matrix cores with the grouped GEMM core:
//   dx  += [hi|lo] [W_g; W_g]       (K = 2Ep)
//   dW_g = hi^T x + lo^T x          (K = tokens, split into chunks; the
//                                    chunk partials and the two halves are
//                                    summed in a fixed order)
// f32 debug path: dl in float32, dx from LDS-staged dl rows, dW_g from
// token-chunk partials, float32 FMA throughout.
#include "common.hpp"
#include "gemm.hpp"
#include "gemm_rs.hpp"
#include "launch.hpp"
#include "probe.hpp"

namespace moe {
namespace {

constexpr int RB_TOK = 32;        // tokens per workgroup in the dx kernel
constexpr int RB_CHUNK = 1024;    // least tokens per split in the dW_g kernels
constexpr int RB_MAXSPLIT = 128;  // most splits: the partials stay O(E d), not O(T)
constexpr int RB_EB = 32;         // experts per workgroup in the dW_g kernel

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
               int E, int64_t chunk, float* __restrict__ part) {
    __shared__ float s_dl[64][RB_EB];
    const int tid = threadIdx.x;
    const int c = blockIdx.x * 256 + tid;
    const int e0 = blockIdx.y * RB_EB;
    const int split = blockIdx.z;
    const int64_t tlo = (int64_t)split * chunk;
    const int64_t thi = min(T, tlo + chunk);
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

using CR = rs::Cfg<256, 256, 2, 4, 1>;
constexpr int RB_MCH = 512;  // least tokens per split of the MFMA dW_g kernel

inline int epad(int E) { return (E + 31) / 32 * 32; }

// dl of token t as bf16 hi/lo pairs: hl[t][e] = hi, hl[t][Ep + e] = lo.
// One wave per token. The token's k (id, gate, gate gradient) triples are read
// once by lanes 0..k-1 and spread through LDS: every expert column then finds
// its own entry there instead of scanning the k ids in global memory. The
// gate sum runs in order j = 0..k-1.
__global__ void __launch_bounds__(256)
rb_dlogits_hilo(const float* __restrict__ dg, const float* __restrict__ logits,
                const int32_t* __restrict__ ids, const float* __restrict__ gates, int64_t T,
                int E, int Ep, int k, int renorm, bf16_t* __restrict__ hl) {
    __shared__ float s_dp[4][256], s_gs[4][256];   // per wave, by expert (Ep <= 256)
    __shared__ float s_g[4][16], s_dg[4][16];       // per wave, by slot j (k <= 16)
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t t = (int64_t)blockIdx.x * 4 + w;
    const bool valid = t < T;
    for (int e = lane; e < Ep; e += 64) { s_dp[w][e] = 0.f; s_gs[w][e] = 0.f; }
    __syncthreads();
    if (valid && lane < k) {
        const int e = ids[t * k + lane];
        const float gj = gates[t * k + lane], dj = dg[t * k + lane];
        s_g[w][lane] = gj;
        s_dg[w][lane] = dj;
        if ((unsigned)e < (unsigned)E) {   // ids outside [0, E) address no logit
            s_dp[w][e] = dj;
            s_gs[w][e] = gj;
        }
    }
    __syncthreads();
    if (!valid) return;
    float gdg = 0.f;
    for (int j = 0; j < k; ++j) gdg += s_g[w][j] * s_dg[w][j];
    const float* lt = logits + t * E;
    float mx = -INFINITY, z = 0.f;
    if (!renorm) {
        for (int e = lane; e < E; e += 64) mx = fmaxf(mx, lt[e]);
        mx = wave_max(mx);
        for (int e = lane; e < E; e += 64) z += __expf(lt[e] - mx);
        z = wave_sum(z);
    }
    bf16_t* out = hl + t * 2 * Ep;
    for (int e = lane; e < Ep; e += 64) {
        float v = 0.f;
        if (e < E) {
            // unselected experts: dp = 0 and (renorm) gate 0
            const float dp = s_dp[w][e];
            if (renorm) v = s_gs[w][e] * (dp - gdg);
            else v = (__expf(lt[e] - mx) / z) * (dp - gdg);
        }
        const uint32_t hi = f2bf(v);
        const uint32_t lo = f2bf(v - bf2f(hi));
        out[e] = (bf16_t)hi;
        out[Ep + e] = (bf16_t)lo;
    }
}

// dx[t] (+)= sum_k hl[t][k] * W_g[k mod Ep]   (tile: 256 tokens x 256 columns)
__global__ void __launch_bounds__(CR::THREADS)
rb_dx_mfma(const bf16_t* __restrict__ hl, const bf16_t* __restrict__ wg, int64_t T, int d,
           int E, int Ep, int accumulate, bf16_t* __restrict__ dx) {
    extern __shared__ __align__(16) char lds[];
    using C = CR;
    const int64_t m0 = (int64_t)blockIdx.x * C::BM;
    const int n0 = blockIdx.y * C::BN;
    const int rows = (int)min((int64_t)C::BM, T - m0);
    rs::DenseKC2<C, C::BM> la;
    la.init(hl, hl, 2 * Ep, m0, rows, 2 * Ep);
    rs::SplitRowsMC<C, C::BN> lb;
    lb.init(wg, d, n0, d, Ep, E);
    rs::NoLoader nl;
    rs::Acc<C> acc;
    rs::mainloop<C>(la, lb, nl, 2 * Ep / rs::KS, lds, acc);
    WaveCoord<C> wc;
    // The lane's dx values are all loaded before the first store: loads placed
    // after a store to the same rows would each wait for the previous one.
    // (rows >= 1 and d >= 8 hold for every launched tile.)
    uint4 old[C::FM][C::FN][2];
    if (accumulate) {
#pragma unroll
        for (int i = 0; i < C::FM; ++i)
#pragma unroll
            for (int j = 0; j < C::FN; ++j)
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    // clamped into the tile's valid rows and columns, so that
                    // the loads need no branch (values off the tile are unused)
                    const int m = min(wc.row(i), rows - 1), n = min(n0 + wc.col8(j, p), d - 8);
                    old[i][j][p] = ld16(dx + (m0 + m) * d + n);
                }
    }
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        const int m = wc.row(i);
        if (m >= rows) continue;
        bf16_t* row = dx + (m0 + m) * d;
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            float v[2][8];
            frag_cols8(acc[0][i][j], v);
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                const int n = n0 + wc.col8(j, p);
                if (n >= d) continue;
                if (accumulate) {
                    float o[8];
                    unpack8(old[i][j][p], o);
#pragma unroll
                    for (int r = 0; r < 8; ++r) v[p][r] += o[r];
                }
                st16(row + n, pack8(v[p]));
            }
        }
    }
}

// part[split][m][n] = sum over the split's tokens of hl[t][m] * x[t][n], m < 2Ep
__global__ void __launch_bounds__(CR::THREADS)
rb_dwg_mfma(const bf16_t* __restrict__ hl, const bf16_t* __restrict__ x, int64_t T, int d,
            int Ep, int64_t chunk, float* __restrict__ part) {
    extern __shared__ __align__(16) char lds[];
    using C = CR;
    const int n0 = blockIdx.x * C::BN;
    const int m0 = blockIdx.y * C::BM;
    const int split = blockIdx.z;
    const int64_t t0 = (int64_t)split * chunk;
    const int cnt = (int)min(chunk, T - t0);
    const int M = 2 * Ep;
    rs::SlotMC<C, C::BM> la;
    la.init(hl, M, t0, m0, M, cnt);
    rs::SlotMC<C, C::BN> lb;
    lb.init(x, d, t0, n0, d, cnt);
    rs::NoLoader nl;
    rs::Acc<C> acc;
    rs::mainloop<C>(la, lb, nl, rs::slices(cnt), lds, acc);
    WaveCoord<C> wc;
    float* out = part + (int64_t)split * M * d;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        const int m = m0 + wc.row(i);
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int n = n0 + wc.col(j, q);
                if (n >= d) continue;
                const f32x16& v = acc[0][i][j];
                *reinterpret_cast<f32x4*>(out + (int64_t)m * d + n) =
                    f32x4{v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
            }
    }
}

// dw_gate[e][i] = sum_split (part[split][e][i] + part[split][Ep + e][i])
__global__ void rb_dwg_reduce_hilo(const float* __restrict__ part, int nsplit, int E, int Ep,
                                   int d, float* __restrict__ dwg) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)E * d) return;
    const int64_t per = (int64_t)2 * Ep * d;
    const int64_t lo_off = (int64_t)Ep * d;
    float acc = 0.f;
    // unrolled so that the loads of several splits are in flight at once; the
    // sum still runs in split order
#pragma unroll 8
    for (int s = 0; s < nsplit; ++s) acc += part[s * per + i] + part[s * per + lo_off + i];
    dwg[i] = acc;
}

// tokens per split: at least `least`, and at most RB_MAXSPLIT splits
inline int64_t split_tokens(int64_t T, int64_t least) {
    int64_t c = (T + RB_MAXSPLIT - 1) / RB_MAXSPLIT;
    c = (c + 63) / 64 * 64;
    return c > least ? c : least;
}
inline int nsplits(int64_t T) { const int64_t c = split_tokens(T, RB_CHUNK); return (int)((T + c - 1) / c); }
inline int msplits(int64_t T) { const int64_t c = split_tokens(T, RB_MCH); return (int)((T + c - 1) / c); }
inline size_t al256(size_t b) { return (b + 255) / 256 * 256; }

hipError_t set_rb_lds_limits() {
    static hipError_t status = [] {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(rb_dx_mfma),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, CR::LDS);
        if (e == hipSuccess)
            e = hipFuncSetAttribute(reinterpret_cast<const void*>(rb_dwg_mfma),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, CR::LDS);
        return e;
    }();
    return status;
}

}  // namespace

size_t route_bwd_workspace(int64_t T, int d, int E, int k, bool f32) {
    (void)k;
    if (f32) {
        const size_t dl = (size_t)T * E * sizeof(float);
        const size_t part = (size_t)nsplits(T) * E * d * sizeof(float);
        return al256(dl) + part;
    }
    const int Ep = epad(E);
    return al256((size_t)T * 2 * Ep * sizeof(bf16_t)) + (size_t)msplits(T) * 2 * Ep * d * sizeof(float);
}

hipError_t route_bwd(const float* dgates, const float* logits, const int32_t* ids,
                     const float* gates, const void* x, const void* wg, int64_t T, int d,
                     int E, int k, bool f32, bool renorm, bool accumulate, float* dwg,
                     void* dx, void* ws, hipStream_t st) {
    if (f32) {
        float* dl = static_cast<float*>(ws);
        float* part = reinterpret_cast<float*>(static_cast<char*>(ws) + al256((size_t)T * E * sizeof(float)));
        hipLaunchKernelGGL(rb_dlogits, dim3((unsigned)((T + 3) / 4)), dim3(256), 0, st, dgates,
                           logits, ids, gates, T, E, k, (int)renorm, dl);
        probe::mark("rb_dlogits", st);
        hipLaunchKernelGGL(rb_dx<true>, dim3((unsigned)((T + RB_TOK - 1) / RB_TOK)), dim3(256), 0,
                           st, dl, wg, T, d, E, (int)accumulate, dx);
        probe::mark("rb_dx", st);
        const int ns = nsplits(T);
        hipLaunchKernelGGL(rb_dwg_partial<true>,
                           dim3((unsigned)((d + 255) / 256), (unsigned)((E + RB_EB - 1) / RB_EB), (unsigned)ns),
                           dim3(256), 0, st, dl, x, T, d, E, split_tokens(T, RB_CHUNK), part);
        probe::mark("rb_dwg_partial", st);
        hipLaunchKernelGGL(rb_dwg_reduce, dim3((unsigned)(((int64_t)E * d + 255) / 256)), dim3(256), 0,
                           st, part, ns, E, d, dwg);
        probe::mark("rb_dwg_reduce", st);
        return hipGetLastError();
    }
    if (hipError_t e = set_rb_lds_limits(); e != hipSuccess) return e;
    const int Ep = epad(E);
    bf16_t* hl = static_cast<bf16_t*>(ws);
    float* part = reinterpret_cast<float*>(static_cast<char*>(ws) +
                                           al256((size_t)T * 2 * Ep * sizeof(bf16_t)));
    hipLaunchKernelGGL(rb_dlogits_hilo, dim3((unsigned)((T + 3) / 4)), dim3(256), 0, st, dgates,
                       logits, ids, gates, T, E, Ep, k, (int)renorm, hl);
    probe::mark("rb_dlogits", st);
    hipLaunchKernelGGL(rb_dx_mfma, dim3((unsigned)((T + CR::BM - 1) / CR::BM), (unsigned)((d + CR::BN - 1) / CR::BN)),
                       dim3(CR::THREADS), CR::LDS, st, (const bf16_t*)hl, (const bf16_t*)wg, T, d, E,
                       Ep, (int)accumulate, (bf16_t*)dx);
    probe::mark("rb_dx", st);
    const int ms = msplits(T);
    hipLaunchKernelGGL(rb_dwg_mfma, dim3((unsigned)((d + CR::BN - 1) / CR::BN), (unsigned)((2 * Ep + CR::BM - 1) / CR::BM), (unsigned)ms),
                       dim3(CR::THREADS), CR::LDS, st, (const bf16_t*)hl, (const bf16_t*)x, T, d, Ep,
                       split_tokens(T, RB_MCH), part);
    probe::mark("rb_dwg_partial", st);
    hipLaunchKernelGGL(rb_dwg_reduce_hilo, dim3((unsigned)(((int64_t)E * d + 255) / 256)), dim3(256), 0,
                       st, part, ms, E, Ep, d, dwg);
    probe::mark("rb_dwg_reduce", st);
    return hipGetLastError();
}

}  // namespace moe
