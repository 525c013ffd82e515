// route.hip -- top-k softmax gating, forward (MoEBlaze paper, Section 2.1:
// topk_experts = TopK(softmax(W_g x)), gate weights of Section 2.3).
//
// bf16 path: the router product logits[T,E] = x W_g^T is a skinny GEMM
// (E <= 256 columns) whose cost is reading x once from HBM, so it runs on the
// matrix cores: each wave owns 16 tokens and all E experts (or, for small
// grids, one of two K halves of them). The x rows of a workgroup (every x
// element is read exactly once) and W_g come through an LDS ring of 64-wide K
// slices filled by direct-to-LDS copies, two or three slices ahead of the one
// being multiplied. Softmax and the top-k selection run on the accumulators
// in registers: the 4 lanes holding one token's logits find the k largest by
// k rounds of (local best, two cross-lane exchanges), ties going to the lower
// expert id.
//
// f32 path (debug mode): one thread per token, float32 FMA.
#include "common.hpp"
#include "gemm.hpp"
#include "launch.hpp"
#include "probe.hpp"

namespace moe {
namespace {

constexpr int RT_BK = 64;    // K slice staged in LDS

// Workgroup shapes. A workgroup routes TB tokens (16 per wave) over all
// experts; its waves form TB/16 token groups times KG K groups, group g taking
// the g-th contiguous share of the K slices. Every workgroup streams all of
// W_g, so larger TB reads fewer W_g bytes per x byte; KG = 2 doubles the waves
// (and with them the copies in flight, which follow the number of waves, not
// the ring depth) for a grid too small to give each CU two workgroups.
//   (64, 1): 4 waves, the default;
//   (64, 2): 8 waves, T < 32768 (fewer than 512 workgroups of 64 tokens);
//   (128, 1): 8 waves, E > 64 and T >= 65536 (W_g is then as large as 128 x rows).
template <int NE, int TB, int KG>
struct RtShape {
    static constexpr int EP = NE * 16;                 // expert rows staged (E padded)
    static constexpr int TG = TB / 16;                 // token groups
    static constexpr int NWAVE = TG * KG;
    static constexpr int THREADS = NWAVE * WAVE;
    static constexpr int RG = (TB + EP) * 128;         // one K group's share of a stage
    static constexpr int STAGE = KG * RG;
    static constexpr int NCOPY = STAGE / 1024;         // 1 KB copies per stage
    static constexpr int PER = NCOPY / NWAVE;          // ... per wave
    // ring depth: four stages, three when four would not fit
    static constexpr int NST = 4 * STAGE <= 160 * 1024 ? 4 : 3;
    static constexpr int LDS = NST * STAGE;
    static_assert(NCOPY % NWAVE == 0, "copies split evenly over the waves");
    static_assert(LDS <= 160 * 1024, "LDS budget");
    static_assert(TG * NE * 4 * WAVE * 4 <= LDS, "K-group reduction fits the ring");
};

// LDS offset (bytes) of 16-byte chunk `c` (0..7) of row `r` in a row-major
// [rows][64] bf16 tile; the chunk index is XOR-swizzled with the row so that
// the 16 rows read by one fragment load hit distinct banks.
__device__ __forceinline__ int kc64_off(int r, int c) { return r * 128 + ((c ^ (r & 7)) << 4); }

// NE: number of 16-expert fragments, E <= 16*NE. nk / KG slices per K group
// (the launch takes KG = 2 only for an even slice count).
template <int NE, int TB, int KG>
__global__ void __launch_bounds__((RtShape<NE, TB, KG>::THREADS))
route_bf16(const bf16_t* __restrict__ x, const bf16_t* __restrict__ wg,
           const float* __restrict__ bias, int64_t T, int d, int E, int k, int renorm,
           int32_t* __restrict__ ids, float* __restrict__ gates, float* __restrict__ logits) {
    using SH = RtShape<NE, TB, KG>;
    extern __shared__ __align__(16) char lds[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = tid >> 6;
    const int tg = wv % SH::TG;   // token group: tokens 16*tg .. of the workgroup
    const int kg = wv / SH::TG;   // K group
    const int grp = lane >> 4;    // which 4-column group of each 16-expert fragment
    const int col = lane & 15;    // token within the wave's 16
    const int64_t t0 = (int64_t)blockIdx.x * TB + tg * 16;

    f32x4 acc[NE];
#pragma unroll
    for (int i = 0; i < NE; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    // LDS ring of NST stages; a stage holds, for every K group, the 64-wide K
    // slice of the workgroup's TB x rows and of all EP W_g rows, 128-byte rows
    // swizzled by kc64_off. Both arrive by direct-to-LDS copies of 1 KB (8
    // rows, lane l fetching the 16-byte chunk that lands at byte 16l), so
    // every request is a whole 128-byte line and the copies of the next
    // NST-1 slices are in flight while a slice is multiplied. Rows past T or E
    // repeat the last valid row: their products are never read.
    constexpr int NST = SH::NST, PER = SH::PER, STAGE = SH::STAGE;
    constexpr int QPG = SH::RG / 1024;                // copies per K group
    const int nks = d / RT_BK / KG;                   // slices per K group
    const uint32_t lds_base = lds_offset(lds);
    const int wvu = wave_id();                        // wave index, uniform (SGPR)
    const int64_t xrow0 = (int64_t)blockIdx.x * TB;
    auto issue = [&](int s) {
        const uint32_t dst = lds_base + (s % NST) * STAGE;
#pragma unroll
        for (int c = 0; c < PER; ++c) {
            const int q = wvu + SH::NWAVE * c;        // copy index within the stage
            const int g = q / QPG;                    // its K group
            const int r = (q % QPG) * 8 + (lane >> 3);   // row (x rows first, then W_g)
            const int ch = (lane & 7) ^ (r & 7);      // logical chunk at this lane's slot
            const int k0 = (g * nks + s) * RT_BK;
            const bf16_t* src;
            if (r < TB) {
                int64_t t = xrow0 + r;
                t = t < T ? t : T - 1;
                src = x + t * d + k0 + ch * 8;
            } else {
                int e = r - TB;
                e = e < E ? e : E - 1;
                src = wg + (int64_t)e * d + k0 + ch * 8;
            }
            dma16(src, dst + q * 1024);
        }
    };
#pragma unroll
    for (int s = 0; s < NST - 1; ++s)
        if (s < nks) issue(s);
    if (nks >= NST - 1) wait_vmcnt<PER * (NST - 2)>();
    else wait_vmcnt<0>();
    barrier_only();
    for (int s = 0; s < nks; ++s) {
        if (s + NST - 1 < nks) issue(s + NST - 1);
        const char* xt = lds + (s % NST) * STAGE + kg * SH::RG;
        const char* wt = xt + TB * 128;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const bf16x8 q = *reinterpret_cast<const bf16x8*>(
                xt + kc64_off(tg * 16 + col, kk * 4 + grp));
#pragma unroll
            for (int fe = 0; fe < NE; ++fe) {
                const bf16x8 p = *reinterpret_cast<const bf16x8*>(
                    wt + kc64_off(fe * 16 + col, kk * 4 + grp));
                acc[fe] = mfma16x16x32(p, q, acc[fe]);
            }
        }
        if (s + 1 < nks) {
            // slice s+1 has landed once only the copies of later slices remain
            if (s + NST - 1 < nks) wait_vmcnt<PER * (NST - 2)>();
            else wait_vmcnt<0>();
            lds_barrier();
        }
    }
    if constexpr (KG == 2) {
        // the second K group's partial logits join the first group's through LDS
        __syncthreads();
        float* red = reinterpret_cast<float*>(lds) + tg * NE * 4 * WAVE + lane;
        if (kg == 1)
#pragma unroll
            for (int fe = 0; fe < NE; ++fe)
#pragma unroll
                for (int r = 0; r < 4; ++r) red[(fe * 4 + r) * WAVE] = acc[fe][r];
        __syncthreads();
        if (kg == 1) return;
#pragma unroll
        for (int fe = 0; fe < NE; ++fe)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[fe][r] += red[(fe * 4 + r) * WAVE];
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

template <int NE, int TB, int KG>
hipError_t launch_route_shape(const void* x, const void* wg, const float* bias, int64_t T,
                              int d, int E, int k, bool renorm, int32_t* ids, float* gates,
                              float* logits, hipStream_t st) {
    using SH = RtShape<NE, TB, KG>;
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(route_bf16<NE, TB, KG>),
        hipFuncAttributeMaxDynamicSharedMemorySize, SH::LDS);
    if (attr != hipSuccess) return attr;
    const dim3 grid((unsigned)((T + TB - 1) / TB));
    hipLaunchKernelGGL((route_bf16<NE, TB, KG>), grid, dim3(SH::THREADS), SH::LDS, st,
                       static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(wg), bias, T,
                       d, E, k, (int)renorm, ids, gates, logits);
    probe::mark("route_bf16", st);
    return hipGetLastError();
}

template <int NE>
hipError_t launch_route_bf16(const void* x, const void* wg, const float* bias, int64_t T,
                             int d, int E, int k, bool renorm, int32_t* ids, float* gates,
                             float* logits, hipStream_t st) {
    if constexpr (NE >= 8) {
        if (T >= 65536)
            return launch_route_shape<NE, 128, 1>(x, wg, bias, T, d, E, k, renorm, ids, gates,
                                                  logits, st);
    }
    if constexpr (NE <= 8) {
        if (T < 32768 && (d / RT_BK) % 2 == 0)
            return launch_route_shape<NE, 64, 2>(x, wg, bias, T, d, E, k, renorm, ids, gates,
                                                 logits, st);
    }
    return launch_route_shape<NE, 64, 1>(x, wg, bias, T, d, E, k, renorm, ids, gates, logits, st);
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
    if (E <= 32) return launch_route_bf16<2>(x, wg, bias, T, d, E, k, renorm, ids, gates, logits, st);
    if (E <= 64) return launch_route_bf16<4>(x, wg, bias, T, d, E, k, renorm, ids, gates, logits, st);
    if (E <= 128) return launch_route_bf16<8>(x, wg, bias, T, d, E, k, renorm, ids, gates, logits, st);
    return launch_route_bf16<16>(x, wg, bias, T, d, E, k, renorm, ids, gates, logits, st);
}

}  // namespace moe
