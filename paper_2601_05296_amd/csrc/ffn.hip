// ffn.hip -- SwiGLU expert FFN of the MoE layer as grouped GEMMs that read
// token rows through the dispatch index maps (MoEBlaze paper, Section 3 and
// Section 5, Algorithm 1), bf16 MFMA with float32 accumulation on gfx950.
//
// Forward (moe_ffn_fwd):
//   G1  A|B = x[eti] [W1|W3]      x rows gathered on load, both first-layer
//                                 projections from one x tile (Section 5.2);
//                                 A and B are the only saved activations.
//   G2  O = (SiLU(A) * B) W2      h = SiLU(A)*B formed on load from A, B and
//                                 never written (SiLU recomputed, Section 5.2).
// Backward (moe_ffn_bwd), in this order so A and B can be overwritten:
//   G3  dW2 = h^T (g dY[eti])     h recomputed on load and scaled by the gate,
//                                 dY rows gathered (the expert-summation
//                                 backward of Section 3.2, never materialised).
//   G4  u = dY[eti] W2^T, then in the epilogue: d_gate partials sum(u*h),
//       dA = g u B SiLU'(A), dB = g u SiLU(A), written over A and B.
//   G5  dW1 = x[eti]^T dA, dW3 = x[eti]^T dB   (one x tile, two products)
//   G6  dX_slot = [dA|dB] [W1|W3]^T             (both branches in one K loop)
// The token gradient is then a unit-weight combine (combine.hip).
//
// Row-wise GEMMs (G1, G2, G4, G6) tile each expert's slot segment; their grid
// is sized for the worst case (S/BM + E tiles per column block) and each
// workgroup finds its (expert, tile) from `offsets` on the device, so nothing
// waits for the host. The weight-gradient GEMMs (G3, G5) have a fixed tile grid
// per expert and loop over the expert's slots as K.
//
// The float32 debug mode uses plain one-output-per-thread kernels.
#include "common.hpp"
#include "gemm.hpp"
#include "launch.hpp"

namespace moe {
namespace {

using C1 = GemmCfg<128, 128, 2, 2, 2>;  // G1, G5 (two right operands)
using CS = GemmCfg<128, 128, 2, 2, 1>;  // G2, G3, G4, G6

// ============================ operand loaders ===================================

// KC rows gathered through an index list: row r -> base[idx[r]] (rows beyond
// `rows` read row 0; their results are discarded).
template <class C, int R>
struct GatherKC {
    static constexpr bool MC = false;
    using Map = KCMap<R, C::THREADS>;
    const bf16_t* p[Map::NCH];
    uint4 reg[Map::NCH];
    __device__ void init(const bf16_t* base, int ld, const int32_t* idx, int rows) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) {
            int r = Map::row(threadIdx.x, i);
            r = r < rows ? r : 0;
            p[i] = base + (int64_t)idx[r] * ld + Map::kcol(threadIdx.x);
        }
    }
    __device__ void fetch(int kt) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) reg[i] = ld16(p[i] + kt * GBK);
    }
    __device__ void stage(char* t) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) st16(t + Map::off(threadIdx.x, i), reg[i]);
    }
};

// KC rows of a dense row-major matrix, K split over two sources:
// k < ksplit from src0, k >= ksplit from src1 (same row, same ld).
template <class C, int R>
struct DenseKC2 {
    static constexpr bool MC = false;
    using Map = KCMap<R, C::THREADS>;
    const bf16_t* p0[Map::NCH];
    const bf16_t* p1[Map::NCH];
    int kst;  // K slices served by src0
    uint4 reg[Map::NCH];
    __device__ void init(const bf16_t* src0, const bf16_t* src1, int ld, int64_t row0, int rows,
                         int ksplit) {
        kst = ksplit / GBK;
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) {
            int r = Map::row(threadIdx.x, i);
            r = r < rows ? r : 0;
            const int64_t o = (row0 + r) * (int64_t)ld + Map::kcol(threadIdx.x);
            p0[i] = src0 + o;
            p1[i] = src1 + o - (int64_t)ksplit;
        }
    }
    __device__ void fetch(int kt) {
        const bool first = kt < kst;
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) reg[i] = ld16((first ? p0[i] : p1[i]) + kt * GBK);
    }
    __device__ void stage(char* t) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) st16(t + Map::off(threadIdx.x, i), reg[i]);
    }
};

// KC rows of h = SiLU(A) * B, computed from the saved A, B (rows = slots).
template <class C, int R>
struct SwigluKC {
    static constexpr bool MC = false;
    using Map = KCMap<R, C::THREADS>;
    const bf16_t* pa[Map::NCH];
    const bf16_t* pb[Map::NCH];
    uint4 ra[Map::NCH], rb[Map::NCH];
    __device__ void init(const bf16_t* A, const bf16_t* B, int ld, int64_t row0, int rows) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) {
            int r = Map::row(threadIdx.x, i);
            r = r < rows ? r : 0;
            const int64_t o = (row0 + r) * (int64_t)ld + Map::kcol(threadIdx.x);
            pa[i] = A + o;
            pb[i] = B + o;
        }
    }
    __device__ void fetch(int kt) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) {
            ra[i] = ld16(pa[i] + kt * GBK);
            rb[i] = ld16(pb[i] + kt * GBK);
        }
    }
    __device__ void stage(char* t) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) {
            float a[8], b[8], h[8];
            unpack8(ra[i], a);
            unpack8(rb[i], b);
#pragma unroll
            for (int j = 0; j < 8; ++j) h[j] = a[j] * sigmoidf_(a[j]) * b[j];
            st16(t + Map::off(threadIdx.x, i), pack8(h));
        }
    }
};

// MC tile of a dense row-major [K][N] matrix (K rows k0.., columns col0..).
template <class C, int R>
struct DenseMC {
    static constexpr bool MC = true;
    using Map = MCMap<R, C::THREADS>;
    const bf16_t* p[Map::NCH];
    int64_t step;
    uint4 reg[Map::NCH];
    __device__ void init(const bf16_t* W, int ld, int col0) {
        step = (int64_t)GBK * ld;
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i)
            p[i] = W + (int64_t)Map::krow(threadIdx.x, i) * ld + col0 + Map::col(threadIdx.x);
    }
    __device__ void fetch(int kt) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) reg[i] = ld16(p[i] + kt * step);
    }
    __device__ void stage(char* t) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) st16(t + Map::off(threadIdx.x, i), reg[i]);
    }
};

// ---- loaders whose K is the slot dimension of one expert (weight gradients) ----
// K row kr (0 <= kr < cnt) is slot off + kr. Rows at or past cnt are either
// zero (ZERO = true; used for the left operand so the tail adds nothing) or a
// copy of a valid row (right operand; multiplied by the zero rows).

// MC rows gathered through eti: row kr -> base[eti[off + kr]] (x or dY).
// Indices are fetched one slice ahead of the data.
template <class C, int R, bool ZERO>
struct GatherMC {
    static constexpr bool MC = true;
    using Map = MCMap<R, C::THREADS>;
    const bf16_t* base;
    const int32_t* idx;  // eti + off
    int ld, cnt;
    int nidx[Map::NCH];
    uint4 reg[Map::NCH];
    __device__ int load_idx(int kt, int i) const {
        int kr = kt * GBK + Map::krow(threadIdx.x, i);
        kr = kr < cnt ? kr : cnt - 1;
        return idx[kr];
    }
    __device__ void init(const bf16_t* b, int ld_, int col0, const int32_t* ix, int cnt_) {
        base = b + col0 + Map::col(threadIdx.x);
        ld = ld_;
        idx = ix;
        cnt = cnt_;
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) nidx[i] = load_idx(0, i);
    }
    __device__ void fetch(int kt) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) {
            const int kr = kt * GBK + Map::krow(threadIdx.x, i);
            uint4 v = ld16(base + (int64_t)nidx[i] * ld);
            if (ZERO && kr >= cnt) v = zero16();
            reg[i] = v;
            nidx[i] = load_idx(kt + 1, i);
        }
    }
    __device__ void stage(char* t) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) st16(t + Map::off(threadIdx.x, i), reg[i]);
    }
};

// MC rows of a slot-ordered matrix (dA or dB): row kr -> src[off + kr].
template <class C, int R>
struct SlotMC {
    static constexpr bool MC = true;
    using Map = MCMap<R, C::THREADS>;
    const bf16_t* base;
    int ld, cnt;
    uint4 reg[Map::NCH];
    __device__ void init(const bf16_t* src, int ld_, int64_t off, int col0, int cnt_) {
        base = src + off * ld_ + col0 + Map::col(threadIdx.x);
        ld = ld_;
        cnt = cnt_;
    }
    __device__ void fetch(int kt) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) {
            int kr = kt * GBK + Map::krow(threadIdx.x, i);
            kr = kr < cnt ? kr : cnt - 1;
            reg[i] = ld16(base + (int64_t)kr * ld);
        }
    }
    __device__ void stage(char* t) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) st16(t + Map::off(threadIdx.x, i), reg[i]);
    }
};

// MC rows of g * SiLU(A) * B (h scaled by the slot's gate), zero past cnt.
template <class C, int R>
struct SwigluGateMC {
    static constexpr bool MC = true;
    using Map = MCMap<R, C::THREADS>;
    const bf16_t* pa;
    const bf16_t* pb;
    const float* gates;
    const int32_t* src;  // slot_src + off
    int ld, cnt;
    float ng[Map::NCH];
    uint4 ra[Map::NCH], rb[Map::NCH];
    float rg[Map::NCH];
    __device__ float load_g(int kt, int i) const {
        int kr = kt * GBK + Map::krow(threadIdx.x, i);
        if (kr >= cnt) return 0.0f;
        return gates[src[kr]];
    }
    __device__ void init(const bf16_t* A, const bf16_t* B, const float* g, const int32_t* ss,
                         int ld_, int64_t off, int col0, int cnt_) {
        const int64_t o = off * ld_ + col0 + Map::col(threadIdx.x);
        pa = A + o;
        pb = B + o;
        gates = g;
        src = ss;
        ld = ld_;
        cnt = cnt_;
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) ng[i] = load_g(0, i);
    }
    __device__ void fetch(int kt) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) {
            int kr = kt * GBK + Map::krow(threadIdx.x, i);
            kr = kr < cnt ? kr : cnt - 1;
            ra[i] = ld16(pa + (int64_t)kr * ld);
            rb[i] = ld16(pb + (int64_t)kr * ld);
            rg[i] = ng[i];
            ng[i] = load_g(kt + 1, i);
        }
    }
    __device__ void stage(char* t) {
#pragma unroll
        for (int i = 0; i < Map::NCH; ++i) {
            float a[8], b[8], h[8];
            unpack8(ra[i], a);
            unpack8(rb[i], b);
#pragma unroll
            for (int j = 0; j < 8; ++j) h[j] = rg[i] * (a[j] * sigmoidf_(a[j]) * b[j]);
            st16(t + Map::off(threadIdx.x, i), pack8(h));
        }
    }
};

// ============================ epilogue helpers ===================================

// Store acc (one 16x16 fragment row-slice: 4 consecutive columns) as bf16.
__device__ __forceinline__ void store4_bf16(bf16_t* p, const f32x4& v) {
    uint2 w;
    w.x = pack_bf2(v[0], v[1]);
    w.y = pack_bf2(v[2], v[3]);
    *reinterpret_cast<uint2*>(p) = w;
}

template <class C>
struct WaveCoord {
    int lane, wm, wn;
    __device__ WaveCoord() {
        lane = threadIdx.x & 63;
        const int wv = threadIdx.x >> 6;
        wm = wv / C::WN;
        wn = wv % C::WN;
    }
    __device__ int row(int fm) const { return wm * C::WTM + fm * 16 + (lane & 15); }
    __device__ int col(int fn) const { return wn * C::WTN + fn * 16 + (lane >> 4) * 4; }
};

// ============================ kernels ==============================================

// G1: A = x[eti] W1[e], B = x[eti] W3[e]
__global__ void __launch_bounds__(C1::THREADS)
g1_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ w1,
          const bf16_t* __restrict__ w3, const int32_t* __restrict__ offsets,
          const int32_t* __restrict__ eti, int d, int f, int E, bf16_t* __restrict__ A,
          bf16_t* __restrict__ B) {
    extern __shared__ __align__(16) char lds[];
    using C = C1;
    SlotTile t;
    const int NT = f / C::BN;
    if (!find_slot_tile<C::THREADS>(offsets, E, C::BM, NT, xcd_remap(blockIdx.x, gridDim.x), C::BN, t))
        return;
    GatherKC<C, C::BM> la;
    la.init(x, d, eti + t.off + t.m0, t.mrows);
    DenseMC<C, C::BN> lb0, lb1;
    lb0.init(w1 + (int64_t)t.e * d * f, f, t.n0);
    lb1.init(w3 + (int64_t)t.e * d * f, f, t.n0);
    f32x4 acc[C::NB][C::FM][C::FN];
    gemm_mainloop<C>(la, lb0, lb1, d / GBK, lds, acc);
    WaveCoord<C> wc;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        const int m = wc.row(i);
        if (m >= t.mrows) continue;
        const int64_t s = (int64_t)t.off + t.m0 + m;
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            const int n = t.n0 + wc.col(j);
            store4_bf16(A + s * f + n, acc[0][i][j]);
            store4_bf16(B + s * f + n, acc[1][i][j]);
        }
    }
}

// G2: O = (SiLU(A) * B) W2[e]
__global__ void __launch_bounds__(CS::THREADS)
g2_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ B,
          const bf16_t* __restrict__ w2, const int32_t* __restrict__ offsets, int d, int f,
          int E, bf16_t* __restrict__ O) {
    extern __shared__ __align__(16) char lds[];
    using C = CS;
    SlotTile t;
    const int NT = d / C::BN;
    if (!find_slot_tile<C::THREADS>(offsets, E, C::BM, NT, xcd_remap(blockIdx.x, gridDim.x), C::BN, t))
        return;
    SwigluKC<C, C::BM> la;
    la.init(A, B, f, (int64_t)t.off + t.m0, t.mrows);
    DenseMC<C, C::BN> lb;
    lb.init(w2 + (int64_t)t.e * f * d, d, t.n0);
    NoLoader nl;
    f32x4 acc[C::NB][C::FM][C::FN];
    gemm_mainloop<C>(la, lb, nl, f / GBK, lds, acc);
    WaveCoord<C> wc;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        const int m = wc.row(i);
        if (m >= t.mrows) continue;
        const int64_t s = (int64_t)t.off + t.m0 + m;
#pragma unroll
        for (int j = 0; j < C::FN; ++j) store4_bf16(O + s * d + t.n0 + wc.col(j), acc[0][i][j]);
    }
}

// G3: dW2[e] = sum_s (g_s h_s)^T dY[eti[s]]   (M = f, N = d, K = slots of e)
__global__ void __launch_bounds__(CS::THREADS)
g3_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ B,
          const bf16_t* __restrict__ dy, const float* __restrict__ gates,
          const int32_t* __restrict__ offsets, const int32_t* __restrict__ eti,
          const int32_t* __restrict__ slot_src, int d, int f, float* __restrict__ dw2) {
    extern __shared__ __align__(16) char lds[];
    using C = CS;
    const int MT = f / C::BM, NT = d / C::BN;
    const int bid = blockIdx.x;
    const int e = bid / (MT * NT);
    const int rem = bid % (MT * NT);
    const int m0 = (rem % MT) * C::BM;
    const int n0 = (rem / MT) * C::BN;
    const int off = offsets[e];
    const int cnt = offsets[e + 1] - off;
    SwigluGateMC<C, C::BM> la;
    GatherMC<C, C::BN, false> lb;
    NoLoader nl;
    if (cnt > 0) {
        la.init(A, B, gates, slot_src + off, f, off, m0, cnt);
        lb.init(dy, d, n0, eti + off, cnt);
    }
    f32x4 acc[C::NB][C::FM][C::FN];
    gemm_mainloop<C>(la, lb, nl, (cnt + GBK - 1) / GBK, lds, acc);
    WaveCoord<C> wc;
    float* out = dw2 + (int64_t)e * f * d;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        const int m = m0 + wc.row(i);
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
            *reinterpret_cast<f32x4*>(out + (int64_t)m * d + n0 + wc.col(j)) = acc[0][i][j];
    }
}

// G4: u = dY[eti] W2[e]^T; epilogue: d_gate partials, dA/dB over A/B.
__global__ void __launch_bounds__(CS::THREADS)
g4_kernel(const bf16_t* __restrict__ dy, const bf16_t* __restrict__ w2,
          const float* __restrict__ gates, const int32_t* __restrict__ offsets,
          const int32_t* __restrict__ eti, const int32_t* __restrict__ slot_src, int d, int f,
          int E, bf16_t* __restrict__ A, bf16_t* __restrict__ B, float* __restrict__ part) {
    extern __shared__ __align__(16) char lds[];
    using C = CS;
    SlotTile t;
    const int NT = f / C::BN;
    if (!find_slot_tile<C::THREADS>(offsets, E, C::BM, NT, xcd_remap(blockIdx.x, gridDim.x), C::BN, t))
        return;
    GatherKC<C, C::BM> la;
    la.init(dy, d, eti + t.off + t.m0, t.mrows);
    DenseKC2<C, C::BN> lb;  // rows c of W2[e] ([f][d]), K = d
    const bf16_t* W2e = w2 + (int64_t)t.e * f * d;
    lb.init(W2e, W2e, d, t.n0, C::BN, d);
    NoLoader nl;
    f32x4 acc[C::NB][C::FM][C::FN];
    gemm_mainloop<C>(la, lb, nl, d / GBK, lds, acc);
    WaveCoord<C> wc;
    const int nparts = NT * C::WN;
    const int pidx = (t.n0 / C::BN) * C::WN + wc.wn;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        const int m = wc.row(i);
        const bool valid = m < t.mrows;
        const int64_t s = (int64_t)t.off + t.m0 + (valid ? m : 0);
        const float g = gates[slot_src[s]];
        float dg = 0.f;
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            const int n = t.n0 + wc.col(j);
            bf16_t* pa = A + s * f + n;
            bf16_t* pb = B + s * f + n;
            const uint2 av = *reinterpret_cast<const uint2*>(pa);
            const uint2 bv = *reinterpret_cast<const uint2*>(pb);
            const float a[4] = {bf_lo(av.x), bf_hi(av.x), bf_lo(av.y), bf_hi(av.y)};
            const float b[4] = {bf_lo(bv.x), bf_hi(bv.x), bf_lo(bv.y), bf_hi(bv.y)};
            float da[4], db[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float u = acc[0][i][j][r];
                const float sg = sigmoidf_(a[r]);
                const float sl = a[r] * sg;
                dg += u * sl * b[r];
                const float dh = g * u;
                da[r] = dh * b[r] * sg * (1.0f + a[r] * (1.0f - sg));
                db[r] = dh * sl;
            }
            if (valid) {
                *reinterpret_cast<uint2*>(pa) = make_uint2(pack_bf2(da[0], da[1]), pack_bf2(da[2], da[3]));
                *reinterpret_cast<uint2*>(pb) = make_uint2(pack_bf2(db[0], db[1]), pack_bf2(db[2], db[3]));
            }
        }
        dg += __shfl_xor(dg, 16, 64);
        dg += __shfl_xor(dg, 32, 64);
        if (valid && (wc.lane >> 4) == 0) part[s * nparts + pidx] = dg;
    }
}

// G5: dW1[e] = x[eti]^T dA, dW3[e] = x[eti]^T dB   (M = d, N = f, K = slots of e)
__global__ void __launch_bounds__(C1::THREADS)
g5_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ dA,
          const bf16_t* __restrict__ dB, const int32_t* __restrict__ offsets,
          const int32_t* __restrict__ eti, int d, int f, float* __restrict__ dw1,
          float* __restrict__ dw3) {
    extern __shared__ __align__(16) char lds[];
    using C = C1;
    const int MT = d / C::BM, NT = f / C::BN;
    const int bid = blockIdx.x;
    const int e = bid / (MT * NT);
    const int rem = bid % (MT * NT);
    const int m0 = (rem % MT) * C::BM;
    const int n0 = (rem / MT) * C::BN;
    const int off = offsets[e];
    const int cnt = offsets[e + 1] - off;
    GatherMC<C, C::BM, true> la;
    SlotMC<C, C::BN> lb0, lb1;
    if (cnt > 0) {
        la.init(x, d, m0, eti + off, cnt);
        lb0.init(dA, f, off, n0, cnt);
        lb1.init(dB, f, off, n0, cnt);
    }
    f32x4 acc[C::NB][C::FM][C::FN];
    gemm_mainloop<C>(la, lb0, lb1, (cnt + GBK - 1) / GBK, lds, acc);
    WaveCoord<C> wc;
    float* o1 = dw1 + (int64_t)e * d * f;
    float* o3 = dw3 + (int64_t)e * d * f;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        const int m = m0 + wc.row(i);
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            const int64_t o = (int64_t)m * f + n0 + wc.col(j);
            *reinterpret_cast<f32x4*>(o1 + o) = acc[0][i][j];
            *reinterpret_cast<f32x4*>(o3 + o) = acc[1][i][j];
        }
    }
}

// G6: dX_slot = dA W1[e]^T + dB W3[e]^T   (K = 2f)
__global__ void __launch_bounds__(CS::THREADS)
g6_kernel(const bf16_t* __restrict__ dA, const bf16_t* __restrict__ dB,
          const bf16_t* __restrict__ w1, const bf16_t* __restrict__ w3,
          const int32_t* __restrict__ offsets, int d, int f, int E, bf16_t* __restrict__ dX) {
    extern __shared__ __align__(16) char lds[];
    using C = CS;
    SlotTile t;
    const int NT = d / C::BN;
    if (!find_slot_tile<C::THREADS>(offsets, E, C::BM, NT, xcd_remap(blockIdx.x, gridDim.x), C::BN, t))
        return;
    DenseKC2<C, C::BM> la;
    la.init(dA, dB, f, (int64_t)t.off + t.m0, t.mrows, f);
    DenseKC2<C, C::BN> lb;  // rows i of W1[e] / W3[e] ([d][f]), K = f then f
    lb.init(w1 + (int64_t)t.e * d * f, w3 + (int64_t)t.e * d * f, f, t.n0, C::BN, f);
    NoLoader nl;
    f32x4 acc[C::NB][C::FM][C::FN];
    gemm_mainloop<C>(la, lb, nl, 2 * f / GBK, lds, acc);
    WaveCoord<C> wc;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        const int m = wc.row(i);
        if (m >= t.mrows) continue;
        const int64_t s = (int64_t)t.off + t.m0 + m;
#pragma unroll
        for (int j = 0; j < C::FN; ++j) store4_bf16(dX + s * d + t.n0 + wc.col(j), acc[0][i][j]);
    }
}

// d_gates[slot_src[s]] = sum of the G4 partials of slot s (fixed order)
__global__ void dgate_reduce(const float* __restrict__ part, int nparts,
                             const int32_t* __restrict__ slot_src, int64_t S,
                             float* __restrict__ dgates) {
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= S) return;
    float acc = 0.f;
    for (int p = 0; p < nparts; ++p) acc += part[s * nparts + p];
    dgates[slot_src[s]] = acc;
}

// ============================ float32 debug kernels ===============================

__device__ int expert_of(const int32_t* offsets, int E, int64_t s) {
    int lo = 0, hi = E - 1;  // largest e with offsets[e] <= s
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (offsets[mid] <= s) lo = mid; else hi = mid - 1;
    }
    return lo;
}
__device__ float silu32(float a) { return a / (1.0f + __expf(-a)); }

__global__ void f32_g1(const float* x, const float* w1, const float* w3, const int32_t* offsets,
                       const int32_t* eti, int64_t S, int d, int f, int E, float* A, float* B) {
    const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= S * f) return;
    const int64_t s = id / f;
    const int n = (int)(id % f);
    const int e = expert_of(offsets, E, s);
    const float* xr = x + (int64_t)eti[s] * d;
    float a = 0.f, b = 0.f;
    for (int i = 0; i < d; ++i) {
        a = fmaf(xr[i], w1[((int64_t)e * d + i) * f + n], a);
        b = fmaf(xr[i], w3[((int64_t)e * d + i) * f + n], b);
    }
    A[id] = a;
    B[id] = b;
}

__global__ void f32_g2(const float* A, const float* B, const float* w2, const int32_t* offsets,
                       int64_t S, int d, int f, int E, float* O) {
    const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= S * d) return;
    const int64_t s = id / d;
    const int n = (int)(id % d);
    const int e = expert_of(offsets, E, s);
    float o = 0.f;
    for (int c = 0; c < f; ++c)
        o = fmaf(silu32(A[s * f + c]) * B[s * f + c], w2[((int64_t)e * f + c) * d + n], o);
    O[id] = o;
}

__global__ void f32_g3(const float* A, const float* B, const float* dy, const float* gates,
                       const int32_t* offsets, const int32_t* eti, const int32_t* slot_src,
                       int d, int f, int E, float* dw2) {
    const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= (int64_t)E * f * d) return;
    const int e = (int)(id / ((int64_t)f * d));
    const int c = (int)((id / d) % f);
    const int n = (int)(id % d);
    float acc = 0.f;
    for (int s = offsets[e]; s < offsets[e + 1]; ++s)
        acc = fmaf(gates[slot_src[s]] * silu32(A[(int64_t)s * f + c]) * B[(int64_t)s * f + c],
                   dy[(int64_t)eti[s] * d + n], acc);
    dw2[id] = acc;
}

// one thread per slot: u, d_gate, dA, dB (in place)
__global__ void f32_g4(const float* dy, const float* w2, const float* gates,
                       const int32_t* offsets, const int32_t* eti, const int32_t* slot_src,
                       int64_t S, int d, int f, int E, float* A, float* B, float* dgates) {
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= S) return;
    const int e = expert_of(offsets, E, s);
    const float* dyr = dy + (int64_t)eti[s] * d;
    const float g = gates[slot_src[s]];
    float dg = 0.f;
    for (int c = 0; c < f; ++c) {
        float u = 0.f;
        const float* wr = w2 + ((int64_t)e * f + c) * d;
        for (int n = 0; n < d; ++n) u = fmaf(dyr[n], wr[n], u);
        const float a = A[s * f + c], b = B[s * f + c];
        const float sg = 1.0f / (1.0f + __expf(-a));
        dg = fmaf(u, a * sg * b, dg);
        const float dh = g * u;
        A[s * f + c] = dh * b * sg * (1.0f + a * (1.0f - sg));
        B[s * f + c] = dh * a * sg;
    }
    dgates[slot_src[s]] = dg;
}

__global__ void f32_g5(const float* x, const float* dA, const float* dB, const int32_t* offsets,
                       const int32_t* eti, int d, int f, int E, float* dw1, float* dw3) {
    const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= (int64_t)E * d * f) return;
    const int e = (int)(id / ((int64_t)d * f));
    const int i = (int)((id / f) % d);
    const int c = (int)(id % f);
    float a1 = 0.f, a3 = 0.f;
    for (int s = offsets[e]; s < offsets[e + 1]; ++s) {
        const float xv = x[(int64_t)eti[s] * d + i];
        a1 = fmaf(xv, dA[(int64_t)s * f + c], a1);
        a3 = fmaf(xv, dB[(int64_t)s * f + c], a3);
    }
    dw1[id] = a1;
    dw3[id] = a3;
}

__global__ void f32_g6(const float* dA, const float* dB, const float* w1, const float* w3,
                       const int32_t* offsets, int64_t S, int d, int f, int E, float* dX) {
    const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= S * d) return;
    const int64_t s = id / d;
    const int i = (int)(id % d);
    const int e = expert_of(offsets, E, s);
    const float* r1 = w1 + ((int64_t)e * d + i) * f;
    const float* r3 = w3 + ((int64_t)e * d + i) * f;
    float acc = 0.f;
    for (int c = 0; c < f; ++c) {
        acc = fmaf(dA[s * f + c], r1[c], acc);
        acc = fmaf(dB[s * f + c], r3[c], acc);
    }
    dX[id] = acc;
}

inline dim3 grid1d(int64_t n, int bs) { return dim3((unsigned)((n + bs - 1) / bs)); }

// Raise the dynamic LDS limit of the GEMM kernels once per process.
hipError_t set_lds_limits() {
    static hipError_t status = [] {
        hipError_t e = hipSuccess;
        auto set = [&](const void* fn, int bytes) {
            if (e == hipSuccess)
                e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
        };
        set(reinterpret_cast<const void*>(g1_kernel), C1::LDS);
        set(reinterpret_cast<const void*>(g2_kernel), CS::LDS);
        set(reinterpret_cast<const void*>(g3_kernel), CS::LDS);
        set(reinterpret_cast<const void*>(g4_kernel), CS::LDS);
        set(reinterpret_cast<const void*>(g5_kernel), C1::LDS);
        set(reinterpret_cast<const void*>(g6_kernel), CS::LDS);
        return e;
    }();
    return status;
}

// number of workgroups for a row-wise grouped GEMM (upper bound on tiles)
inline unsigned slot_grid(int64_t S, int E, int BM, int NT) {
    return (unsigned)(((S + BM - 1) / BM + E) * NT);
}

}  // namespace

hipError_t ffn_fwd(const FfnArgs& a, bool f32, hipStream_t st) {
    const int64_t S = a.T * a.k;
    if (f32) {
        hipLaunchKernelGGL(f32_g1, grid1d(S * a.f, 256), dim3(256), 0, st,
                           (const float*)a.x, (const float*)a.w1, (const float*)a.w3, a.offsets,
                           a.eti, S, a.d, a.f, a.E, (float*)a.A, (float*)a.B);
        hipLaunchKernelGGL(f32_g2, grid1d(S * a.d, 256), dim3(256), 0, st,
                           (const float*)a.A, (const float*)a.B, (const float*)a.w2, a.offsets, S,
                           a.d, a.f, a.E, (float*)a.O);
        return hipGetLastError();
    }
    if (hipError_t e = set_lds_limits(); e != hipSuccess) return e;
    hipLaunchKernelGGL(g1_kernel, dim3(slot_grid(S, a.E, C1::BM, a.f / C1::BN)), dim3(C1::THREADS),
                       C1::LDS, st, (const bf16_t*)a.x, (const bf16_t*)a.w1, (const bf16_t*)a.w3,
                       a.offsets, a.eti, a.d, a.f, a.E, (bf16_t*)a.A, (bf16_t*)a.B);
    hipLaunchKernelGGL(g2_kernel, dim3(slot_grid(S, a.E, CS::BM, a.d / CS::BN)), dim3(CS::THREADS),
                       CS::LDS, st, (const bf16_t*)a.A, (const bf16_t*)a.B, (const bf16_t*)a.w2,
                       a.offsets, a.d, a.f, a.E, (bf16_t*)a.O);
    return hipGetLastError();
}

size_t ffn_bwd_workspace(int64_t T, int d, int f, int E, int k, bool f32) {
    (void)d; (void)E;
    if (f32) return 0;
    const int64_t S = T * k;
    const int nparts = (f / CS::BN) * CS::WN;
    return (size_t)(S * nparts * (int64_t)sizeof(float));
}

hipError_t ffn_bwd(const FfnArgs& a, bool f32, hipStream_t st) {
    const int64_t S = a.T * a.k;
    if (f32) {
        hipLaunchKernelGGL(f32_g3, grid1d((int64_t)a.E * a.f * a.d, 256), dim3(256), 0, st,
                           (const float*)a.A, (const float*)a.B, (const float*)a.dy, a.gates,
                           a.offsets, a.eti, a.slot_src, a.d, a.f, a.E, a.dw2);
        hipLaunchKernelGGL(f32_g4, grid1d(S, 64), dim3(64), 0, st, (const float*)a.dy,
                           (const float*)a.w2, a.gates, a.offsets, a.eti, a.slot_src, S, a.d, a.f,
                           a.E, (float*)a.A, (float*)a.B, a.dgates);
        hipLaunchKernelGGL(f32_g5, grid1d((int64_t)a.E * a.d * a.f, 256), dim3(256), 0, st,
                           (const float*)a.x, (const float*)a.A, (const float*)a.B, a.offsets,
                           a.eti, a.d, a.f, a.E, a.dw1, a.dw3);
        hipLaunchKernelGGL(f32_g6, grid1d(S * a.d, 256), dim3(256), 0, st, (const float*)a.A,
                           (const float*)a.B, (const float*)a.w1, (const float*)a.w3, a.offsets,
                           S, a.d, a.f, a.E, (float*)a.dX);
        return hipGetLastError();
    }
    if (hipError_t e = set_lds_limits(); e != hipSuccess) return e;
    float* part = static_cast<float*>(a.ws);
    const int nparts = (a.f / CS::BN) * CS::WN;
    hipLaunchKernelGGL(g3_kernel, dim3(a.E * (a.f / CS::BM) * (a.d / CS::BN)), dim3(CS::THREADS),
                       CS::LDS, st, (const bf16_t*)a.A, (const bf16_t*)a.B, (const bf16_t*)a.dy,
                       a.gates, a.offsets, a.eti, a.slot_src, a.d, a.f, a.dw2);
    hipLaunchKernelGGL(g4_kernel, dim3(slot_grid(S, a.E, CS::BM, a.f / CS::BN)), dim3(CS::THREADS),
                       CS::LDS, st, (const bf16_t*)a.dy, (const bf16_t*)a.w2, a.gates, a.offsets,
                       a.eti, a.slot_src, a.d, a.f, a.E, (bf16_t*)a.A, (bf16_t*)a.B, part);
    hipLaunchKernelGGL(dgate_reduce, grid1d(S, 256), dim3(256), 0, st, part, nparts, a.slot_src,
                       S, a.dgates);
    hipLaunchKernelGGL(g5_kernel, dim3(a.E * (a.d / C1::BM) * (a.f / C1::BN)), dim3(C1::THREADS),
                       C1::LDS, st, (const bf16_t*)a.x, (const bf16_t*)a.A, (const bf16_t*)a.B,
                       a.offsets, a.eti, a.d, a.f, a.dw1, a.dw3);
    hipLaunchKernelGGL(g6_kernel, dim3(slot_grid(S, a.E, CS::BM, a.d / CS::BN)), dim3(CS::THREADS),
                       CS::LDS, st, (const bf16_t*)a.A, (const bf16_t*)a.B, (const bf16_t*)a.w1,
                       (const bf16_t*)a.w3, a.offsets, a.d, a.f, a.E, (bf16_t*)a.dX);
    return hipGetLastError();
}

}  // namespace moe
