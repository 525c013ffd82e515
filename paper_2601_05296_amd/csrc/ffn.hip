// ffn.hip -- expert FFN of the MoE layer (SwiGLU, or the non-gated SiLU / ReLU
// expert) as grouped GEMMs that read token rows through the dispatch index
// maps (MoEBlaze paper, Section 3 and Section 5, Algorithm 1), bf16 MFMA with
// float32 accumulation on gfx950.
//
// Forward (moe_ffn_fwd):
//   G1  A|B = x[eti] [W1|W3]      x rows gathered on load, both first-layer
//                                 projections from one x tile (Section 5.2);
//                                 A and B are the only saved activations. The
//                                 epilogue also writes h = SiLU(A)*B into a
//                                 transient buffer for G2.
//   G2  O = h W2                  (MOE_H_ON_LOAD: g2h_kernel forms h from A
//                                 and B as it loads them; no h buffer.)
// Backward (moe_ffn_bwd):
//   G4  u = dY[eti] W2^T, then in the epilogue: d_gate partials sum(u*h),
//       dA = g u B SiLU'(A), dB = g u SiLU(A) written over A and B, and g*h
//       into a transient buffer (h recomputed from A and B).
//   G3  dW2 = (g h)^T dY[eti]     dY rows gathered (the expert-summation
//                                 backward of Section 3.2). MOE_H_ON_LOAD:
//                                 g3h_kernel runs before G4 and forms g*h from
//                                 A, B and the gates on load; no g*h buffer.
//   G5  dW1 = x[eti]^T dA, dW3 = x[eti]^T dB   (one x tile, two products)
//   G6  dX_slot = [dA|dB] [W1|W3]^T             (both branches in one K loop)
// The token gradient is then a unit-weight combine (combine.hip). Forming h
// on load costs the second GEMMs a second operand stream and an in-LDS pass
// per K slice; it returns the same bits.
// The combined calls (moe_ffn_fwd_combine / moe_ffn_bwd_combine) run G2 and
// G6 over column strips, each followed by the ordered combine; with
// MOE_ATOMIC_COMBINE they run once, and the epilogue adds each slot row
// (times its gate in the forward) into the token's row of y or dx by
// packed-bf16 atomics (Section 3.1's reduction as the outputs are produced).
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
#include "gemm_rs.hpp"
#include "launch.hpp"
#include "probe.hpp"

namespace moe {
namespace {

// Tile configurations (gemm_rs.hpp): <BM, BN, WM, WN, NB>. 256-row tiles,
// 2x4 waves. Single right operand: each wave owns 128 x 64 outputs. Two right
// operands (G1: W1 and W3; G5: dA and dB): 128 x 32 of each.
using RD = rs::Cfg<256, 128, 2, 4, 2>;  // G1, G5
using RS = rs::Cfg<256, 256, 2, 4, 1>;  // G2, G3, G6
constexpr int RASTER_GM = 4;            // M tiles per raster group (find_slot_tile)

// ============================ epilogue helpers ===================================

__device__ __forceinline__ void store4_bf16(bf16_t* p, float a, float b, float c, float d) {
    *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf2(a, b), pack_bf2(c, d));
}
__device__ __forceinline__ float silu_bf(float a) { return a * sigmoidf_(a); }

// Expert activation: SwiGLU (gated, Section 5.1) or the non-gated SiLU / ReLU
// experts of Section 2.2, E(x) = W2 act(W1 x), whose only saved activation is
// A = x W1. ReLU'(0) is taken as 0.
enum : int { ACT_SWIGLU = 0, ACT_SILU = 1, ACT_RELU = 2 };
template <int ACT>
__device__ __forceinline__ float act_f(float a) {
    if constexpr (ACT == ACT_RELU) return a > 0.f ? a : 0.f;
    else return a * sigmoidf_(a);
}
template <int ACT>
__device__ __forceinline__ float act_d(float a) {
    if constexpr (ACT == ACT_RELU) return a > 0.f ? 1.f : 0.f;
    else {
        const float sg = sigmoidf_(a);
        return sg * (1.0f + a * (1.0f - sg));
    }
}
// tile configuration of the first-layer and dW1 GEMMs: two right operands
// when gated (W1|W3, dA|dB), one otherwise
template <int ACT> using CFirst = std::conditional_t<ACT == ACT_SWIGLU, RD, RS>;
// GEMMs with h (or g*h) formed on load: 128 x 512 tiles, so that each h
// element is formed once per 512 output columns rather than per 256 (forming
// it costs two transcendentals and some ten other vector operations, about
// as much vector-ALU time per slice as the slice's MFMAs take).
using RHW = rs::Cfg<128, 512, 2, 4, 1>;
static_assert(RD::THREADS == RS::THREADS && RD::LDS == RS::LDS, "RD and RS launch alike");
__device__ __forceinline__ void store8_bf16(bf16_t* p, const float (&v)[8]) { st16(p, pack8(v)); }

// ============================ kernels ==============================================

// G1: A = x[eti] W1[e], B = x[eti] W3[e]; also H = SiLU(A) * B (from the
// bf16-rounded A and B, exactly as the backward recomputes it). Non-gated:
// A = x[eti] W1[e] and H = act(A). H == NULL: A and B only (the backward's
// recompute under the full-recompute policy).
template <int ACT>
__global__ void __launch_bounds__(RD::THREADS)
g1_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ w1,
          const bf16_t* __restrict__ w3, const int32_t* __restrict__ offsets,
          const int32_t* __restrict__ eti, int d, int f, int E, bf16_t* __restrict__ A,
          bf16_t* __restrict__ B, bf16_t* __restrict__ H) {
    extern __shared__ __align__(16) char lds[];
    using C = CFirst<ACT>;
    SlotTile t;
    const int NT = (f + C::BN - 1) / C::BN;
    if (!find_slot_tile<C::THREADS>(reinterpret_cast<int*>(lds), offsets, E, C::BM, NT,
                                    xcd_remap(blockIdx.x, gridDim.x), C::BN,
                                    t, RASTER_GM))
        return;
    rs::GatherKC<C, C::BM> la;
    la.init(x, d, eti + t.off + t.m0, t.mrows);
    rs::DenseMC<C, C::BN> lb0;
    lb0.init(w1 + (int64_t)t.e * d * f, f, t.n0, f);
    rs::Acc<C> acc;
    if constexpr (ACT == ACT_SWIGLU) {
        rs::DenseMC<C, C::BN> lb1;
        lb1.init(w3 + (int64_t)t.e * d * f, f, t.n0, f);
        rs::mainloop<C>(la, lb0, lb1, d / rs::KS, lds, acc);
    } else {
        rs::NoLoader nl;
        rs::mainloop<C>(la, lb0, nl, d / rs::KS, lds, acc);
    }
    WaveCoord<C> wc;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        const int m = wc.row(i);
        if (m >= t.mrows) continue;
        const int64_t s = (int64_t)t.off + t.m0 + m;
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            float va[2][8], vb[2][8];
            frag_cols8(acc[0][i][j], va);
            if constexpr (ACT == ACT_SWIGLU) frag_cols8(acc[1][i][j], vb);
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                const int n = t.n0 + wc.col8(j, p);
                if (n >= f) continue;
                float a[8], b[8], h[8];
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    a[r] = bf2f(f2bf(va[p][r]));
                    if constexpr (ACT == ACT_SWIGLU) {
                        b[r] = bf2f(f2bf(vb[p][r]));
                        h[r] = silu_bf(a[r]) * b[r];
                    } else {
                        h[r] = act_f<ACT>(a[r]);
                    }
                }
                store8_bf16(A + s * f + n, a);
                if constexpr (ACT == ACT_SWIGLU) store8_bf16(B + s * f + n, b);
                if (H) store8_bf16(H + s * f + n, h);
            }
        }
    }
}

// Output rows of a slot tile (G2, G6), columns n < ncols of the tile's strip:
// slot row s goes to row s of O, rows ldo apart.
template <class C>
__device__ __forceinline__ void slot_rows_out(const rs::Acc<C>& acc, const SlotTile& t,
                                              int ncols, int64_t ldo, bf16_t* __restrict__ O) {
    WaveCoord<C> wc;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        const int m = wc.row(i);
        if (m >= t.mrows) continue;
        const int64_t s = (int64_t)t.off + t.m0 + m;
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            float v[2][8];
            frag_cols8(acc[0][i][j], v);
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                const int n = t.n0 + wc.col8(j, p);
                if (n < ncols) store8_bf16(O + s * ldo + n, v[p]);
            }
        }
    }
}

// The combine folded into the epilogue (Section 3.1): slot row s of the tile,
// times gs[s] (1 when gs is null), rounded to bf16, is added into row tok[s]
// of O (rows ldo apart) by packed-bf16 atomics, so that O receives the sum
// over a token's slots in whatever order the tiles finish. The tile goes
// through LDS first (free once the main loop is done), so that each atomic
// instruction of a wave covers 256 contiguous bytes of one row: 64 lanes, two
// columns each (straight from the fragments, a wave's atomics would touch 32
// rows 16 bytes apiece). 16-byte chunks are XOR-swizzled by row, so that both
// the fragment-ordered writes and the row-ordered reads are free of bank
// conflicts.
template <class C>
__device__ __forceinline__ void slot_rows_scatter(const rs::Acc<C>& acc, const SlotTile& t,
                                                  int ncols, int64_t ldo,
                                                  bf16_t* __restrict__ O,
                                                  const int32_t* __restrict__ tok,
                                                  const float* __restrict__ gs, char* lds) {
    constexpr int RB = C::BN * 2;      // bytes per tile row in LDS
    constexpr int CPR = C::BN / 8;     // 16-byte chunks per row
    static_assert(C::BM * RB <= C::LDS && CPR >= 32 && C::BN % 128 == 0, "scatter staging");
    const WaveCoord<C> wc;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        const int m = wc.row(i);
        const float g = (gs && m < t.mrows) ? gs[(int64_t)t.off + t.m0 + m] : 1.0f;
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            float v[2][8];
            frag_cols8(acc[0][i][j], v);
#pragma unroll
            for (int p = 0; p < 2; ++p) {
#pragma unroll
                for (int r = 0; r < 8; ++r) v[p][r] *= g;
                const int chunk = (wc.col8(j, p) >> 3) ^ (m & 31);
                *reinterpret_cast<uint4*>(lds + m * RB + chunk * 16) = pack8(v[p]);
            }
        }
    }
    __syncthreads();
    const int wv = wave_id();
    const int rows = min(C::BM, t.mrows);
    for (int r = wv; r < rows; r += C::NW) {
        bf16_t* dst = O + (int64_t)tok[(int64_t)t.off + t.m0 + r] * ldo + t.n0;
#pragma unroll
        for (int c = 0; c < C::BN / 128; ++c) {
            const int col = c * 128 + 2 * wc.lane;
            if (t.n0 + col >= ncols) continue;
            const int chunk = (col >> 3) ^ (r & 31);
            const uint32_t v =
                *reinterpret_cast<const uint32_t*>(lds + r * RB + chunk * 16 + (col & 7) * 2);
            __builtin_amdgcn_global_atomic_fadd_v2bf16(reinterpret_cast<bf16x2_t*>(dst + col),
                                                       __builtin_bit_cast(bf16x2_t, v));
        }
    }
}

// slot rows out, plain or (SCATTER) added into the token rows
template <bool SCATTER, class C>
__device__ __forceinline__ void slot_rows(const rs::Acc<C>& acc, const SlotTile& t, int ncols,
                                          int64_t ldo, bf16_t* __restrict__ O,
                                          const int32_t* __restrict__ tok,
                                          const float* __restrict__ gs, char* lds) {
    if constexpr (SCATTER) slot_rows_scatter<C>(acc, t, ncols, ldo, O, tok, gs, lds);
    else slot_rows_out<C>(acc, t, ncols, ldo, O);
}

// G2: O = H W2[e], output columns [n_base, n_base + ncols) of W2 into columns
// [0, ncols) of O, rows ldo apart (SCATTER: added into the token rows, see
// slot_rows_scatter)
template <bool SCATTER>
__global__ void __launch_bounds__(RS::THREADS)
g2_kernel(const bf16_t* __restrict__ H, const bf16_t* __restrict__ w2,
          const int32_t* __restrict__ offsets, int d, int f, int E, int n_base, int ncols,
          int64_t ldo, bf16_t* __restrict__ O, const int32_t* __restrict__ tok,
          const float* __restrict__ gs) {
    extern __shared__ __align__(16) char lds[];
    using C = RS;
    SlotTile t;
    const int NT = (ncols + C::BN - 1) / C::BN;
    if (!find_slot_tile<C::THREADS>(reinterpret_cast<int*>(lds), offsets, E, C::BM, NT,
                                    xcd_remap(blockIdx.x, gridDim.x), C::BN,
                                    t, RASTER_GM))
        return;
    rs::DenseKC2<C, C::BM> la;
    la.init(H, H, f, (int64_t)t.off + t.m0, t.mrows, f);
    rs::DenseMC<C, C::BN> lb;
    lb.init(w2 + (int64_t)t.e * f * d, d, n_base + t.n0, n_base + ncols);
    rs::NoLoader nl;
    rs::Acc<C> acc;
    rs::mainloop<C>(la, lb, nl, f / rs::KS, lds, acc);
    slot_rows<SCATTER, C>(acc, t, ncols, ldo, O, tok, gs, lds);
}

// h of one element from its (bf16-valued) A and B: the arithmetic of G1's
// epilogue, on the same values, so the result is bit-identical to the
// buffered h. Non-gated: act(A), B unused. With a gate g: g * h, the
// arithmetic of G4's epilogue for the dW2 GEMM's operand.
template <int ACT, bool GATE>
__device__ __forceinline__ float h_one(float a, float b, float g) {
    float h;
    if constexpr (ACT == ACT_SWIGLU) h = silu_bf(a) * b;
    else h = act_f<ACT>(a);
    if constexpr (GATE) h = g * h;
    return h;
}
// h of element pair dword p of (va, vb) as two transform pieces of one element
// each: piece 2p forms the low element into hl, piece 2p+1 the high one and
// packs the pair in place of va's dword (pieces of one element keep the
// vector work between two MFMAs short)
template <int ACT, bool GATE, int P>
__device__ __forceinline__ void h_piece(rs::u32x4& va, const rs::u32x4& vb, float g, float& hl) {
    constexpr int q = P >> 1;
    if constexpr ((P & 1) == 0) hl = h_one<ACT, GATE>(bf_lo(va[q]), bf_lo(vb[q]), g);
    else va[q] = pack_bf2(hl, h_one<ACT, GATE>(bf_hi(va[q]), bf_hi(vb[q]), g));
}

// Left operand of the second GEMM with h formed on load: KC tile of h rows
// row0 + r (r < rows, else row0) from the slot-ordered A (and B), h formed in
// registers between the loads and the LDS write (Section 3.1 keeps only the
// first MLP's output; Section 5.2 recomputes the activation).
template <int ACT, class C, int R>
struct HKC {
    static constexpr bool MC = false;
    using G = rs::KCGeom<C, R>;
    static constexpr int NCH = G::NCH;
    static constexpr bool GATED = ACT == ACT_SWIGLU;
    const bf16_t* pa;      // A + row0 * ld + this thread's chunk column
    int64_t dba;           // B - A, in elements
    int ld, rows;
    rs::u32x4 va[NCH], vb[NCH];
    __device__ void init(const bf16_t* A, const bf16_t* B, int ld_, int64_t row0, int rows_) {
        ld = ld_;
        rows = rows_;
        dba = GATED ? B - A : 0;
        pa = A + rs::roff(row0, ld) + G::chunk(0) * 8;
    }
    template <int i> __device__ void load(int kt) {
        int r = G::row(i);
        r = r < rows ? r : 0;
        const bf16_t* q = pa + rs::roff(r, ld) + kt * rs::KS;
        va[i] = rs::ldg16(q);
        if constexpr (GATED) vb[i] = rs::ldg16(q + dba);
    }
    // h of chunk i in place of A's, one element per piece
    static constexpr int NSUB = 8;
    float hl;
    template <int i, int p> __device__ void sub() { h_piece<ACT, false, p>(va[i], vb[i], 0.f, hl); }
    template <int i, bool TAIL> __device__ void store(char* tile) { rs::sts16(tile + G::lds(i), va[i]); }
};

// G2 with h formed on load: O = h W2[e] from the saved A (and B), no h buffer.
template <int ACT, bool SCATTER>
__global__ void __launch_bounds__(RHW::THREADS)
g2h_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ B,
           const bf16_t* __restrict__ w2, const int32_t* __restrict__ offsets, int d, int f,
           int E, int n_base, int ncols, int64_t ldo, bf16_t* __restrict__ O,
           const int32_t* __restrict__ tok, const float* __restrict__ gs) {
    extern __shared__ __align__(16) char lds[];
    using C = RHW;
    SlotTile t;
    const int NT = (ncols + C::BN - 1) / C::BN;
    if (!find_slot_tile<C::THREADS>(reinterpret_cast<int*>(lds), offsets, E, C::BM, NT,
                                        xcd_remap(blockIdx.x, gridDim.x), C::BN, t, RASTER_GM))
        return;
    HKC<ACT, C, C::BM> la;
    la.init(A, B, f, (int64_t)t.off + t.m0, t.mrows);
    rs::DenseMC<C, C::BN> lb;
    lb.init(w2 + (int64_t)t.e * f * d, d, n_base + t.n0, n_base + ncols);
    rs::NoLoader nl;
    rs::Acc<C> acc;
    rs::mainloop<C>(la, lb, nl, f / rs::KS, lds, acc);
    slot_rows<SCATTER, C>(acc, t, ncols, ldo, O, tok, gs, lds);
}

// G4: u = dY[eti] W2[e]^T; epilogue: d_gate partials sum(u*h), dA/dB over
// A/B, and HG = g * h (h recomputed from A, B) for G3. Non-gated: dA = g u
// act'(A) over A, h = act(A). gs: the gates in slot order (read when HG_OUT is
// false, i.e. with h on load, where G3 has built them already).
template <int ACT, bool HG_OUT>
__global__ void __launch_bounds__(RS::THREADS)
g4_kernel(const bf16_t* __restrict__ dy, const bf16_t* __restrict__ w2,
          const float* __restrict__ gates, const int32_t* __restrict__ offsets,
          const int32_t* __restrict__ eti, const int32_t* __restrict__ slot_src,
          const float* __restrict__ gs, int d, int f,
          int E, bf16_t* __restrict__ A, bf16_t* __restrict__ B, bf16_t* __restrict__ HG,
          float* __restrict__ part) {
    extern __shared__ __align__(16) char lds[];
    using C = RS;
    SlotTile t;
    const int NT = (f + C::BN - 1) / C::BN;
    if (!find_slot_tile<C::THREADS>(reinterpret_cast<int*>(lds), offsets, E, C::BM, NT,
                                    xcd_remap(blockIdx.x, gridDim.x), C::BN,
                                    t, RASTER_GM))
        return;
    rs::GatherKC<C, C::BM> la;
    la.init(dy, d, eti + t.off + t.m0, t.mrows);
    rs::DenseKC2<C, C::BN> lb;  // rows c of W2[e] ([f][d]), K = d
    const bf16_t* W2e = w2 + (int64_t)t.e * f * d;
    lb.init(W2e, W2e, d, t.n0, min(C::BN, f - t.n0), d);
    rs::NoLoader nl;
    const WaveCoord<C> wc;
    // The gate of this lane's row in every epilogue round. With h on load
    // (no HG output) they stand in slot order already (gs, for G3) and are
    // loaded before the main loop, whose waits cover them. Otherwise they
    // are gathered through slot_src after it. Either way they are waited for
    // (by a wait the compiler sees) before the epilogue's first copy: the
    // compiler does not see the copies, and a load of its own issued after
    // them would end in a wait for everything outstanding, copies included.
    float gr[C::FM];
    auto gate_row = [&](int i) {
        const int m = wc.row(i);
        return (int64_t)t.off + t.m0 + (m < t.mrows ? m : 0);
    };
    if constexpr (!HG_OUT) {
#pragma unroll
        for (int i = 0; i < C::FM; ++i) gr[i] = gs[gate_row(i)];
    }
    rs::Acc<C> acc;
    rs::mainloop<C>(la, lb, nl, d / rs::KS, lds, acc);
    if constexpr (HG_OUT) {
#pragma unroll
        for (int i = 0; i < C::FM; ++i) gr[i] = gates[slot_src[gate_row(i)]];
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    // ---- epilogue, one round per fragment row-block (64 rows of the tile) ----
    // The A and B rows of a round come into LDS by DMA (1 KB copies, many in
    // flight), two LDS buffers deep: the copies of round i+1 are issued as
    // round i starts and land while round i is computed and stored. Every
    // lane reads its values in LDS, writes dA and dB back in place, and the
    // rows then leave LDS as whole 512-byte runs. g*h goes out straight from
    // registers, 16 bytes per lane (staging it through LDS as well took two
    // more barriers per round and spilled registers: 4% slower). 16-byte
    // chunks are XOR-swizzled by row, so the fragment-ordered LDS accesses
    // (32 rows, one column) are conflict-free.
    constexpr int RR = C::WM * 32;       // rows per round
    constexpr int RB = C::BN * 2;        // bytes per row
    constexpr int CPR = RB / 16;         // 16-byte chunks per row (32)
    constexpr int ARR = RR * RB;         // bytes of one array in LDS
    constexpr int NARR = ACT == ACT_SWIGLU ? 2 : 1;   // A, B or A alone
    constexpr int BUF = 2 * ARR;         // one round's buffer (A and B)
    static_assert(CPR == 32 && 2 * BUF <= C::LDS, "G4 staging layout");
    const int nparts = NT * C::WN;
    const int pidx = (t.n0 / C::BN) * C::WN + wc.wn;
    const uint32_t lds_base = lds_offset(lds);
    const int wv = wave_id();
    auto tile_row = [&](int rr, int i) { return (rr / 32) * C::WTM + i * 32 + (rr & 31); };
    // DMA round i's A and B rows into buffer i & 1: copy q covers rows 2q',
    // 2q'+1 of array q / (ARR/1024)
    auto issue_round = [&](int i) {
#pragma unroll
        for (int c = 0; c < NARR * ARR / 1024 / C::NW; ++c) {
            const int q = wv + c * C::NW;
            const int arr = q / (ARR / 1024), qq = q % (ARR / 1024);
            const int rr = 2 * qq + (wc.lane >> 5);
            const int lc = (wc.lane & 31) ^ (rr & 31);
            int m = tile_row(rr, i);
            m = m < t.mrows ? m : 0;
            int n = t.n0 + lc * 8;
            n = n < f ? n : f - 8;
            const bf16_t* src = (arr ? B : A) + ((int64_t)t.off + t.m0 + m) * f + n;
            dma16(src, lds_base + (i & 1) * BUF + arr * ARR + qq * 1024);
        }
    };
    // Stores a round issues after the copies of the next round: the d_gate
    // partial, the dA (dB) row chunks, the g*h chunks.
    constexpr int NSTORE = 1 + NARR * RR * CPR / C::THREADS + (HG_OUT ? 2 * C::FN : 0);
    // In a full tile every one of them is issued by every wave (no lane
    // condition empties a wave's execution mask).
    const bool full = t.mrows >= C::BM && t.n0 + C::BN <= f;
    issue_round(0);
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
        // Round i's rows have landed. The wait counter counts vector-memory
        // operations down in issue order, so in a full tile, once at most
        // NSTORE remain, round i's copies (issued before round i-1's stores)
        // are done and the stores may still be in flight. Otherwise wait for
        // everything. Buffer (i+1) & 1 was last read by round i-1's stores,
        // before its closing barrier.
        if (i > 0 && full) wait_vmcnt<NSTORE>();
        else wait_vmcnt<0>();
        barrier_only();
        if (i + 1 < C::FM) issue_round(i + 1);
        char* const buf = lds + (i & 1) * BUF;
        // this lane's row of the round and its gate
        const int rr = wc.wm * 32 + (wc.lane & 31);
        const int m = wc.row(i);
        const bool valid = m < t.mrows;
        const int64_t s = (int64_t)t.off + t.m0 + (valid ? m : 0);
        const float g = gr[i];
        char* rowA = buf + rr * RB;
        char* rowB = buf + ARR + rr * RB;
        float dg = 0.f;
        uint4 hgv[C::FN][2];
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            float u8[2][8];
            frag_cols8(acc[0][i][j], u8);
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                const int cl = wc.col8(j, p);                       // tile column
                const int off = (((cl >> 3) ^ (rr & 31)) << 4);     // swizzled chunk
                const int n = t.n0 + cl;
                float a[8], b[8], da[8], db[8], hg[8];
                unpack8(*reinterpret_cast<const uint4*>(rowA + off), a);
                if constexpr (ACT == ACT_SWIGLU)
                    unpack8(*reinterpret_cast<const uint4*>(rowB + off), b);
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    const float u = u8[p][r];
                    const float dh = g * u;
                    float h;
                    if constexpr (ACT == ACT_SWIGLU) {
                        const float sg = sigmoidf_(a[r]);
                        const float sl = a[r] * sg;
                        h = sl * b[r];
                        da[r] = dh * b[r] * sg * (1.0f + a[r] * (1.0f - sg));
                        db[r] = dh * sl;
                    } else {
                        h = act_f<ACT>(a[r]);
                        da[r] = dh * act_d<ACT>(a[r]);
                    }
                    dg += n < f ? u * h : 0.f;
                    hg[r] = g * h;
                }
                *reinterpret_cast<uint4*>(rowA + off) = pack8(da);
                if constexpr (ACT == ACT_SWIGLU) *reinterpret_cast<uint4*>(rowB + off) = pack8(db);
                hgv[j][p] = pack8(hg);
            }
        }
        dg += __shfl_xor(dg, 32, 64);
        if (valid && wc.lane < 32) part[s * nparts + pidx] = dg;
        // rows out of LDS: chunk id -> (array, row, physical chunk)
        auto store_rows = [&](int narr, bf16_t* const* dst) {
#pragma unroll
            for (int ps = 0; ps < narr * RR * CPR / C::THREADS; ++ps) {
                const int cid = ps * C::THREADS + threadIdx.x;
                const int arr = cid / (RR * CPR);
                const int r2 = (cid / CPR) % RR, pc = cid % CPR;
                const int mm = tile_row(r2, i);
                const int n = t.n0 + ((pc ^ (r2 & 31)) << 3);
                const uint4 v = *reinterpret_cast<const uint4*>(buf + arr * ARR + r2 * RB + pc * 16);
                if (mm < t.mrows && n < f) st16_nt(dst[arr] + ((int64_t)t.off + t.m0 + mm) * f + n, v);
            }
        };
        lds_barrier();
        {
            bf16_t* const dst[2] = {A, B};
            store_rows(NARR, dst);
        }
        lds_barrier();
        if constexpr (HG_OUT) {   // false when G3 forms g*h itself (h on load)
            if (valid) {
#pragma unroll
                for (int j = 0; j < C::FN; ++j)
#pragma unroll
                    for (int p = 0; p < 2; ++p) {
                        const int n = t.n0 + wc.col8(j, p);
                        if (n < f) st16(HG + s * f + n, hgv[j][p]);
                    }
            }
        }
    }
}

// Weight gradients are written once and not read again by this layer:
// nontemporal stores keep them from displacing the operands in L2. With
// `add`, the tile is added to what the array holds (gradients of several
// token chunks).
__device__ __forceinline__ void st_nt(float* p, const f32x4& v) {
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(p));
}
__device__ __forceinline__ void st_dw(float* p, const f32x4& v, int add) {
    st_nt(p, add ? v + *reinterpret_cast<const f32x4*>(p) : v);
}

// G3: dW2[e] = sum_s HG[s]^T dY[eti[s]]   (M = f, N = d, K = slots of e)
__global__ void __launch_bounds__(RS::THREADS)
g3_kernel(const bf16_t* __restrict__ HG, const bf16_t* __restrict__ dy,
          const ExpertRank* __restrict__ rank, const int32_t* __restrict__ eti, int d, int f,
          int add, float* __restrict__ dw2) {
    extern __shared__ __align__(16) char lds[];
    using C = RS;
    const int MT = (f + C::BM - 1) / C::BM, NT = (d + C::BN - 1) / C::BN;
    ExpertRank er;
    int mt, nt;
    if (!wgrad_tile(rank, blockIdx.x, MT, NT, er, mt, nt)) return;
    const int e = er.e, off = er.off, cnt = er.cnt;
    const int m0 = mt * C::BM;
    const int n0 = nt * C::BN;
    rs::SlotMC<C, C::BM> la;
    rs::GatherMC<C, C::BN> lb;
    rs::NoLoader nl;
    if (cnt > 0) {
        la.init(HG, f, off, m0, f, cnt);
        lb.init(dy, d, n0, d, eti + off, cnt);
    }
    rs::Acc<C> acc;
    rs::mainloop<C>(la, lb, nl, rs::slices(cnt), lds, acc);
    float* out = dw2 + (int64_t)e * f * d;
    RowStage<C, 1>::run(acc, lds, [&](int, int r, int c, const f32x4& v) {
        const int m = m0 + r, n = n0 + c;
        if (m < f && n < d) st_dw(out + (int64_t)m * d + n, v, add);
    });
}


// Left operand of the dW2 GEMM with g*h formed on load: MC tile of g*h slot
// rows off + kr (K = the expert's slots) from the saved A (and B) and the
// slot-ordered gates gs. Rows at or past cnt are read from row cnt - 1 and
// stored as zeros.
template <int ACT, class C, int R>
struct GHMC {
    static constexpr bool MC = true;
    using G = rs::MCGeom<C, R>;
    static constexpr int NCH = G::NCH;
    static constexpr bool GATED = ACT == ACT_SWIGLU;
    const bf16_t* pa;      // A + off * ld + this thread's column
    int64_t dba;           // B - A, in elements
    const float* gsp;      // gates of slots off, off + 1, ...
    int ld, cnt;
    uint32_t zmask;
    rs::u32x4 va[NCH], vb[NCH];
    float g[NCH];
    __device__ void init(const bf16_t* A, const bf16_t* B, int ld_, int64_t off, int col0,
                         int ncols, int cnt_, const float* gs) {
        ld = ld_;
        cnt = cnt_;
        zmask = 0;
        dba = GATED ? B - A : 0;
        int c = col0 + G::col(0);
        c = c < ncols ? c : ncols - 8;
        pa = A + rs::roff(off, ld) + c;
        gsp = gs + off;
    }
    template <int i> __device__ void load(int kt) {
        int k = kt * rs::KS + G::krow(i);
        const bool past = k >= cnt;
        zmask = past ? (zmask | (1u << i)) : (zmask & ~(1u << i));
        k = past ? cnt - 1 : k;
        const bf16_t* q = pa + rs::roff(k, ld);
        va[i] = rs::ldg16(q);
        if constexpr (GATED) vb[i] = rs::ldg16(q + dba);
        g[i] = gsp[k];
    }
    // g * h of chunk i in place of A's, one element per piece
    static constexpr int NSUB = 8;
    float hl;
    template <int i, int p> __device__ void sub() { h_piece<ACT, true, p>(va[i], vb[i], g[i], hl); }
    template <int i, bool TAIL> __device__ void store(char* tile) {
        const rs::u32x4 z = {0u, 0u, 0u, 0u};
        if constexpr (TAIL) rs::sts16(tile + G::lds(i), (zmask >> i) & 1 ? z : va[i]);
        else rs::sts16(tile + G::lds(i), va[i]);
    }
};

// gs[s] = gates[slot_src[s]] for the filled slots s < offsets[E], 0 for the
// rest up to S (the gate of each slot in slot order, for the dW2 GEMM's
// left operand; fewer than S slots are filled only when the index build
// rejected choices)
__global__ void slot_gates(const float* __restrict__ gates, const int32_t* __restrict__ slot_src,
                           const int32_t* __restrict__ offsets, int E, int64_t S,
                           float* __restrict__ gs) {
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s < offsets[E]) gs[s] = gates[slot_src[s]];
    else if (s < S) gs[s] = 0.0f;
}

// gs[token_index_map[i]] = gates[i] for the accepted choices i < T*k: the
// gate of each filled slot in slot order, from the token-side map (the
// forward has no slot_src)
__global__ void fwd_slot_gates(const float* __restrict__ gates,
                                    const int32_t* __restrict__ tim, int64_t n,
                                    float* __restrict__ gs) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) {
        const int32_t s = tim[i];
        if (s >= 0) gs[s] = gates[i];
    }
}

// p[0..n) = 0 for n bf16 values, n a multiple of 8, p 16-byte aligned (a
// kernel rather than a memset, so that it can be captured in a graph)
__global__ void zero_bf16(bf16_t* __restrict__ p, int64_t n) {
    const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 8;
    if (i < n) st16(p + i, uint4{0u, 0u, 0u, 0u});
}

// G3 with g*h formed on load from the saved A (and B) and the slot-ordered
// gates gs: dW2[e] = sum_s (g h)[s]^T dY[eti[s]]. Runs before G4, which then
// writes dA, dB over A, B and no g*h.
template <int ACT>
__global__ void __launch_bounds__(RHW::THREADS)
g3h_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ B,
           const float* __restrict__ gs, const bf16_t* __restrict__ dy,
           const ExpertRank* __restrict__ rank, const int32_t* __restrict__ eti, int d, int f,
           int add, float* __restrict__ dw2) {
    extern __shared__ __align__(16) char lds[];
    using C = RHW;
    const int MT = (f + C::BM - 1) / C::BM, NT = (d + C::BN - 1) / C::BN;
    ExpertRank er;
    int mt, nt;
    if (!wgrad_tile(rank, blockIdx.x, MT, NT, er, mt, nt)) return;
    const int e = er.e, off = er.off, cnt = er.cnt;
    const int m0 = mt * C::BM;
    const int n0 = nt * C::BN;
    GHMC<ACT, C, C::BM> la;
    rs::GatherMC<C, C::BN> lb;
    rs::NoLoader nl;
    if (cnt > 0) {
        la.init(A, B, f, off, m0, f, cnt, gs);
        lb.init(dy, d, n0, d, eti + off, cnt);
    }
    rs::Acc<C> acc;
    rs::mainloop<C>(la, lb, nl, rs::slices(cnt), lds, acc);
    float* out = dw2 + (int64_t)e * f * d;
    RowStage<C, 1>::run(acc, lds, [&](int, int r, int c, const f32x4& v) {
        const int m = m0 + r, n = n0 + c;
        if (m < f && n < d) st_dw(out + (int64_t)m * d + n, v, add);
    });
}

// G5: dW1[e] = x[eti]^T dA, dW3[e] = x[eti]^T dB   (M = d, N = f, K = slots of e)
// (non-gated: dW1 alone)
template <int ACT>
__global__ void __launch_bounds__(RD::THREADS)
g5_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ dA,
          const bf16_t* __restrict__ dB, const ExpertRank* __restrict__ rank,
          const int32_t* __restrict__ eti, int d, int f, int add, float* __restrict__ dw1,
          float* __restrict__ dw3) {
    extern __shared__ __align__(16) char lds[];
    using C = CFirst<ACT>;
    const int MT = (d + C::BM - 1) / C::BM, NT = (f + C::BN - 1) / C::BN;
    ExpertRank er;
    int mt, nt;
    if (!wgrad_tile(rank, blockIdx.x, MT, NT, er, mt, nt)) return;
    const int e = er.e, off = er.off, cnt = er.cnt;
    const int m0 = mt * C::BM;
    const int n0 = nt * C::BN;
    rs::GatherMC<C, C::BM> la;
    rs::SlotMC<C, C::BN> lb0;
    std::conditional_t<ACT == ACT_SWIGLU, rs::SlotMC<C, C::BN>, rs::NoLoader> lb1;
    if (cnt > 0) {
        la.init(x, d, m0, d, eti + off, cnt);
        lb0.init(dA, f, off, n0, f, cnt);
        if constexpr (ACT == ACT_SWIGLU) lb1.init(dB, f, off, n0, f, cnt);
    }
    rs::Acc<C> acc;
    rs::mainloop<C>(la, lb0, lb1, rs::slices(cnt), lds, acc);
    float* o1 = dw1 + (int64_t)e * d * f;
    float* o3 = ACT == ACT_SWIGLU ? dw3 + (int64_t)e * d * f : o1;  // dw3 is NULL when non-gated
    RowStage<C, ACT == ACT_SWIGLU ? 2 : 1>::run(acc, lds, [&](int b, int r, int c, const f32x4& v) {
        const int m = m0 + r, n = n0 + c;
        if (m < d && n < f) st_dw((b ? o3 : o1) + (int64_t)m * f + n, v, add);
    });
}

// G6: dX_slot = dA W1[e]^T + dB W3[e]^T, output columns [n_base, n_base + ncols)
// into rows ldo apart   (K = 2f; non-gated: dA W1[e]^T, K = f,
// called with dB = dA and W3 = W1, whose second halves are then never reached)
template <bool SCATTER>
__global__ void __launch_bounds__(RS::THREADS)
g6_kernel(const bf16_t* __restrict__ dA, const bf16_t* __restrict__ dB,
          const bf16_t* __restrict__ w1, const bf16_t* __restrict__ w3,
          const int32_t* __restrict__ offsets, int d, int f, int E, int kslices, int n_base,
          int ncols, int64_t ldo, bf16_t* __restrict__ dX, const int32_t* __restrict__ tok) {
    extern __shared__ __align__(16) char lds[];
    using C = RS;
    SlotTile t;
    const int NT = (ncols + C::BN - 1) / C::BN;
    if (!find_slot_tile<C::THREADS>(reinterpret_cast<int*>(lds), offsets, E, C::BM, NT,
                                    xcd_remap(blockIdx.x, gridDim.x), C::BN,
                                    t, RASTER_GM))
        return;
    rs::DenseKC2<C, C::BM> la;
    la.init(dA, dB, f, (int64_t)t.off + t.m0, t.mrows, f);
    rs::DenseKC2<C, C::BN> lb;  // rows i of W1[e] / W3[e] ([d][f]), K = f then f
    lb.init(w1 + (int64_t)t.e * d * f, w3 + (int64_t)t.e * d * f, f, n_base + t.n0,
            min(C::BN, ncols - t.n0), f);
    rs::NoLoader nl;
    rs::Acc<C> acc;
    rs::mainloop<C>(la, lb, nl, kslices, lds, acc);
    slot_rows<SCATTER, C>(acc, t, ncols, ldo, dX, tok, nullptr, lds);
}

// rank[r] = (expert, first slot, slot count) of the expert of rank r by slot
// count, descending, ties to the lower index: the order in which the
// weight-gradient GEMMs take the experts (wgrad_tile). One workgroup, one
// thread per expert.
__global__ void __launch_bounds__(256)
expert_ranks(const int32_t* __restrict__ offsets, int E, ExpertRank* __restrict__ rank) {
    __shared__ int cnt[256];
    const int t = threadIdx.x;
    if (t < E) cnt[t] = offsets[t + 1] - offsets[t];
    __syncthreads();
    if (t >= E) return;
    const int c = cnt[t];
    int r = 0;
    for (int u = 0; u < E; ++u) {
        const int cu = cnt[u];
        r += (cu > c) | ((cu == c) & (u < t));
    }
    rank[r] = ExpertRank{t, offsets[t], c, 0};
}

// d_gates[slot_src[s]] = sum of the G4 partials of slot s (fixed order)
// (16-byte loads when a slot's nparts partials fill whole 16-byte vectors;
// the sum runs in order p = 0..nparts-1 either way)
__global__ void dgate_reduce(const float* __restrict__ part, int nparts,
                             const int32_t* __restrict__ slot_src,
                             const int32_t* __restrict__ offsets, int E, int64_t S,
                             float* __restrict__ dgates) {
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= S || s >= offsets[E]) return;
    const float* row = part + s * nparts;
    float acc = 0.f;
    if ((nparts & 3) == 0) {
        for (int p = 0; p < nparts; p += 4) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(row + p);
            acc += v[0]; acc += v[1]; acc += v[2]; acc += v[3];
        }
    } else {
        for (int p = 0; p < nparts; ++p) acc += row[p];
    }
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

// h and its derivatives from the first-layer outputs (b unused when non-gated)
template <int ACT>
__device__ float f32_h(float a, float b) {
    if constexpr (ACT == ACT_SWIGLU) return silu32(a) * b;
    else if constexpr (ACT == ACT_RELU) return a > 0.f ? a : 0.f;
    else return silu32(a);
}

template <int ACT>
__global__ void f32_g1(const float* x, const float* w1, const float* w3, const int32_t* offsets,
                       const int32_t* eti, int64_t S, int d, int f, int E, float* A, float* B) {
    const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= S * f) return;
    const int64_t s = id / f;
    const int n = (int)(id % f);
    if (s >= offsets[E]) return;
    const int e = expert_of(offsets, E, s);
    const float* xr = x + (int64_t)eti[s] * d;
    float a = 0.f, b = 0.f;
    for (int i = 0; i < d; ++i) {
        a = fmaf(xr[i], w1[((int64_t)e * d + i) * f + n], a);
        if constexpr (ACT == ACT_SWIGLU) b = fmaf(xr[i], w3[((int64_t)e * d + i) * f + n], b);
    }
    A[id] = a;
    if constexpr (ACT == ACT_SWIGLU) B[id] = b;
}

template <int ACT>
__global__ void f32_g2(const float* A, const float* B, const float* w2, const int32_t* offsets,
                       int64_t S, int d, int f, int E, float* O) {
    const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= S * d) return;
    const int64_t s = id / d;
    const int n = (int)(id % d);
    const int e = expert_of(offsets, E, s);
    float o = 0.f;
    for (int c = 0; c < f; ++c)
        o = fmaf(f32_h<ACT>(A[s * f + c], ACT == ACT_SWIGLU ? B[s * f + c] : 0.f),
                 w2[((int64_t)e * f + c) * d + n], o);
    O[id] = o;
}

template <int ACT>
__global__ void f32_g3(const float* A, const float* B, const float* dy, const float* gates,
                       const int32_t* offsets, const int32_t* eti, const int32_t* slot_src,
                       int d, int f, int E, int add, float* dw2) {
    const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= (int64_t)E * f * d) return;
    const int e = (int)(id / ((int64_t)f * d));
    const int c = (int)((id / d) % f);
    const int n = (int)(id % d);
    float acc = 0.f;
    for (int s = offsets[e]; s < offsets[e + 1]; ++s) {
        const float h = f32_h<ACT>(A[(int64_t)s * f + c],
                                   ACT == ACT_SWIGLU ? B[(int64_t)s * f + c] : 0.f);
        acc = fmaf(gates[slot_src[s]] * h, dy[(int64_t)eti[s] * d + n], acc);
    }
    dw2[id] = add ? dw2[id] + acc : acc;
}

// one thread per slot: u, d_gate, dA, dB (in place)
template <int ACT>
__global__ void f32_g4(const float* dy, const float* w2, const float* gates,
                       const int32_t* offsets, const int32_t* eti, const int32_t* slot_src,
                       int64_t S, int d, int f, int E, float* A, float* B, float* dgates) {
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= S || s >= offsets[E]) return;
    const int e = expert_of(offsets, E, s);
    const float* dyr = dy + (int64_t)eti[s] * d;
    const float g = gates[slot_src[s]];
    float dg = 0.f;
    for (int c = 0; c < f; ++c) {
        float u = 0.f;
        const float* wr = w2 + ((int64_t)e * f + c) * d;
        for (int n = 0; n < d; ++n) u = fmaf(dyr[n], wr[n], u);
        const float a = A[s * f + c];
        const float dh = g * u;
        if constexpr (ACT == ACT_SWIGLU) {
            const float b = B[s * f + c];
            const float sg = 1.0f / (1.0f + __expf(-a));
            dg = fmaf(u, a * sg * b, dg);
            A[s * f + c] = dh * b * sg * (1.0f + a * (1.0f - sg));
            B[s * f + c] = dh * a * sg;
        } else if constexpr (ACT == ACT_RELU) {
            dg = fmaf(u, a > 0.f ? a : 0.f, dg);
            A[s * f + c] = a > 0.f ? dh : 0.f;
        } else {
            const float sg = 1.0f / (1.0f + __expf(-a));
            dg = fmaf(u, a * sg, dg);
            A[s * f + c] = dh * sg * (1.0f + a * (1.0f - sg));
        }
    }
    dgates[slot_src[s]] = dg;
}

template <int ACT>
__global__ void f32_g5(const float* x, const float* dA, const float* dB, const int32_t* offsets,
                       const int32_t* eti, int d, int f, int E, int add, float* dw1, float* dw3) {
    const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= (int64_t)E * d * f) return;
    const int e = (int)(id / ((int64_t)d * f));
    const int i = (int)((id / f) % d);
    const int c = (int)(id % f);
    float a1 = 0.f, a3 = 0.f;
    for (int s = offsets[e]; s < offsets[e + 1]; ++s) {
        const float xv = x[(int64_t)eti[s] * d + i];
        a1 = fmaf(xv, dA[(int64_t)s * f + c], a1);
        if constexpr (ACT == ACT_SWIGLU) a3 = fmaf(xv, dB[(int64_t)s * f + c], a3);
    }
    dw1[id] = add ? dw1[id] + a1 : a1;
    if constexpr (ACT == ACT_SWIGLU) dw3[id] = add ? dw3[id] + a3 : a3;
}

template <int ACT>
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
        if constexpr (ACT == ACT_SWIGLU) acc = fmaf(dB[s * f + c], r3[c], acc);
    }
    dX[id] = acc;
}

inline dim3 grid1d(int64_t n, int bs) { return dim3((unsigned)((n + bs - 1) / bs)); }

// number of workgroups for a row-wise grouped GEMM (upper bound on tiles)
inline unsigned slot_grid(int64_t S, int E, int BM, int NT) {
    return (unsigned)(((S + BM - 1) / BM + E) * NT);
}
inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// Raise the dynamic LDS limit of the GEMM kernels once per process.
hipError_t set_lds_limits() {
    static hipError_t status = [] {
        hipError_t e = hipSuccess;
        auto set = [&](const void* fn, int bytes) {
            if (e == hipSuccess)
                e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
        };
        auto per_act = [&](auto act) {
            constexpr int ACT = decltype(act)::value;
            set(reinterpret_cast<const void*>(g1_kernel<ACT>), CFirst<ACT>::LDS);
            set(reinterpret_cast<const void*>(g4_kernel<ACT, true>), RS::LDS);
            set(reinterpret_cast<const void*>(g4_kernel<ACT, false>), RS::LDS);
            set(reinterpret_cast<const void*>(g5_kernel<ACT>), CFirst<ACT>::LDS);
            set(reinterpret_cast<const void*>(g2h_kernel<ACT, false>), RHW::LDS);
            set(reinterpret_cast<const void*>(g2h_kernel<ACT, true>), RHW::LDS);
            set(reinterpret_cast<const void*>(g3h_kernel<ACT>), RHW::LDS);
        };
        per_act(std::integral_constant<int, ACT_SWIGLU>{});
        per_act(std::integral_constant<int, ACT_SILU>{});
        per_act(std::integral_constant<int, ACT_RELU>{});
        set(reinterpret_cast<const void*>(g2_kernel<false>), RS::LDS);
        set(reinterpret_cast<const void*>(g2_kernel<true>), RS::LDS);
        set(reinterpret_cast<const void*>(g3_kernel), RS::LDS);
        set(reinterpret_cast<const void*>(g6_kernel<false>), RS::LDS);
        set(reinterpret_cast<const void*>(g6_kernel<true>), RS::LDS);
        return e;
    }();
    return status;
}

inline size_t align256(size_t b) { return (b + 255) / 256 * 256; }
inline int g4_nparts(int f) { return cdiv(f, RS::BN) * RS::WN; }
// Column strip of the expert output (or of dX_slot) when the combine follows
// strip by strip. Narrow strips save memory, but a launch needs enough tiles
// (here about six waves of 256) or its last partial wave leaves CUs idle, so
// the strips are about as narrow as that allows, in whole tiles of the GEMM
// that produces them (BM x BN): with 256 x 256 tiles about 1024 columns for
// 98k slots and 64 experts, 2048 for 65k slots and 8 experts, 256 for 524k
// slots. `narrow`: round the number of strips up rather than down (the last
// strip may then be narrower), for the memory-lean h-on-load policy.
inline int strip_width(int64_t S, int E, int d, int BM, int BN, bool narrow) {
    const int64_t mtiles = (S + BM - 1) / BM + E / 2;   // tiles per column of tiles
    const int64_t want = 6 * 256;
    int64_t w = (int64_t)BN * ((want + mtiles - 1) / mtiles);
    w = w < d ? w : d;
    const int n = (int)(narrow ? (d + w - 1) / w : d / w);   // strips
    const int width = ((d + n - 1) / n + BN - 1) / BN * BN;
    return width < d ? width : d;
}
// strips of the forward's second GEMM (h on load: its 128 x 512 tiles) and of
// the backward's dX GEMM
inline int fwd_strip(int64_t S, int E, int d, bool h_on_load) {
    return h_on_load ? strip_width(S, E, d, RHW::BM, RHW::BN, true)
                     : strip_width(S, E, d, RS::BM, RS::BN, false);
}
inline int bwd_strip(int64_t S, int E, int d) { return strip_width(S, E, d, RS::BM, RS::BN, false); }

}  // namespace

size_t ffn_fwd_workspace(int64_t T, int d, int f, int E, int k, bool f32, bool combined,
                         bool h_on_load, bool scatter) {
    const size_t S = (size_t)T * k;
    if (f32) return combined ? align256(S * d * sizeof(float)) : 0;  // O
    const size_t h = h_on_load ? 0 : align256(S * f * sizeof(bf16_t));   // H
    if (!combined) return h;
    if (scatter) return h + align256(S * sizeof(float));                  // slot gates
    return h + align256(S * fwd_strip(S, E, d, h_on_load) * sizeof(bf16_t));
}

namespace {

template <int ACT>
hipError_t ffn_fwd_act(const FfnArgs& a, bool f32, hipStream_t st) {
    const int64_t S = a.T * a.k;
    if (f32) {
        hipLaunchKernelGGL(f32_g1<ACT>, grid1d(S * a.f, 256), dim3(256), 0, st,
                           (const float*)a.x, (const float*)a.w1, (const float*)a.w3, a.offsets,
                           a.eti, S, a.d, a.f, a.E, (float*)a.A, (float*)a.B);
        probe::mark("f32_g1", st);
        float* O = a.y ? static_cast<float*>(a.ws) : (float*)a.O;
        hipLaunchKernelGGL(f32_g2<ACT>, grid1d(S * a.d, 256), dim3(256), 0, st,
                           (const float*)a.A, (const float*)a.B, (const float*)a.w2, a.offsets, S,
                           a.d, a.f, a.E, O);
        probe::mark("f32_g2", st);
        if (a.y) return combine(O, a.gates, a.tim, a.T, a.d, a.k, true, false, a.y, st);
        return hipGetLastError();
    }
    if (hipError_t e = set_lds_limits(); e != hipSuccess) return e;
    using C1 = CFirst<ACT>;
    using C2H = RHW;
    // h buffered between the GEMMs, or (h_on_load) formed again from A, B
    bf16_t* H = a.h_on_load ? nullptr : static_cast<bf16_t*>(a.ws);
    hipLaunchKernelGGL(g1_kernel<ACT>, dim3(slot_grid(S, a.E, C1::BM, cdiv(a.f, C1::BN))),
                       dim3(C1::THREADS), C1::LDS, st, (const bf16_t*)a.x, (const bf16_t*)a.w1,
                       (const bf16_t*)a.w3, a.offsets, a.eti, a.d, a.f, a.E, (bf16_t*)a.A,
                       (bf16_t*)a.B, H);
    probe::mark("g1_kernel", st);
    // the second GEMM over columns [c0, c0 + nc): slot rows into out (ldo
    // apart), or with gs (scatter) added into the token rows of out
    auto second = [&](int c0, int nc, int64_t ldo, bf16_t* out, const float* gs) {
        if (a.h_on_load) {
            auto g2h = gs ? g2h_kernel<ACT, true> : g2h_kernel<ACT, false>;
            hipLaunchKernelGGL(g2h, dim3(slot_grid(S, a.E, C2H::BM, cdiv(nc, C2H::BN))),
                               dim3(C2H::THREADS), C2H::LDS, st, (const bf16_t*)a.A,
                               (const bf16_t*)a.B, (const bf16_t*)a.w2, a.offsets, a.d, a.f, a.E,
                               c0, nc, ldo, out, a.eti, gs);
            probe::mark("g2h_kernel", st);
        } else {
            auto g2 = gs ? g2_kernel<true> : g2_kernel<false>;
            hipLaunchKernelGGL(g2, dim3(slot_grid(S, a.E, RS::BM, cdiv(nc, RS::BN))),
                               dim3(RS::THREADS), RS::LDS, st, (const bf16_t*)H,
                               (const bf16_t*)a.w2, a.offsets, a.d, a.f, a.E, c0, nc, ldo, out,
                               a.eti, gs);
            probe::mark("g2_kernel", st);
        }
    };
    if (!a.y) {   // O [S, d] for the caller's combine
        second(0, a.d, (int64_t)a.d, (bf16_t*)a.O, nullptr);
        return hipGetLastError();
    }
    if (a.scatter) {   // y = 0, then every slot row times its gate added into y
        float* gs = reinterpret_cast<float*>(
            static_cast<char*>(a.ws) + (a.h_on_load ? 0 : align256((size_t)S * a.f * sizeof(bf16_t))));
        hipLaunchKernelGGL(fwd_slot_gates, grid1d(S, 256), dim3(256), 0, st, a.gates, a.tim,
                           S, gs);
        probe::mark("fwd_slot_gates", st);
        hipLaunchKernelGGL(zero_bf16, grid1d(a.T * a.d / 8, 256), dim3(256), 0, st,
                           static_cast<bf16_t*>(a.y), a.T * a.d);
        probe::mark("zero_bf16", st);
        second(0, a.d, (int64_t)a.d, static_cast<bf16_t*>(a.y), gs);
        return hipGetLastError();
    }
    // combined: one column strip of O at a time, straight into y
    const int sw = fwd_strip(S, a.E, a.d, a.h_on_load);
    bf16_t* strip = reinterpret_cast<bf16_t*>(
        static_cast<char*>(a.ws) + (a.h_on_load ? 0 : align256((size_t)S * a.f * sizeof(bf16_t))));
    for (int c0 = 0; c0 < a.d; c0 += sw) {
        const int nc = min(sw, a.d - c0);
        second(c0, nc, (int64_t)nc, strip, nullptr);
        if (hipError_t e = combine_cols(strip, nc, a.gates, a.tim, a.T, nc, a.k, false, false,
                                        static_cast<bf16_t*>(a.y) + c0, a.d, st);
            e != hipSuccess)
            return e;
    }
    return hipGetLastError();
}

template <int ACT>
hipError_t ffn_first_act(const FfnArgs& a, bool f32, hipStream_t st) {
    const int64_t S = a.T * a.k;
    if (f32) {
        hipLaunchKernelGGL(f32_g1<ACT>, grid1d(S * a.f, 256), dim3(256), 0, st,
                           (const float*)a.x, (const float*)a.w1, (const float*)a.w3, a.offsets,
                           a.eti, S, a.d, a.f, a.E, (float*)a.A, (float*)a.B);
        probe::mark("f32_g1", st);
        return hipGetLastError();
    }
    if (hipError_t e = set_lds_limits(); e != hipSuccess) return e;
    using C1 = CFirst<ACT>;
    hipLaunchKernelGGL(g1_kernel<ACT>, dim3(slot_grid(S, a.E, C1::BM, cdiv(a.f, C1::BN))),
                       dim3(C1::THREADS), C1::LDS, st, (const bf16_t*)a.x, (const bf16_t*)a.w1,
                       (const bf16_t*)a.w3, a.offsets, a.eti, a.d, a.f, a.E, (bf16_t*)a.A,
                       (bf16_t*)a.B, (bf16_t*)nullptr);
    probe::mark("g1_kernel", st);
    return hipGetLastError();
}

}  // namespace

hipError_t ffn_first(const FfnArgs& a, bool f32, hipStream_t st) {
    switch (a.act) {
    case ACT_SILU: return ffn_first_act<ACT_SILU>(a, f32, st);
    case ACT_RELU: return ffn_first_act<ACT_RELU>(a, f32, st);
    default: return ffn_first_act<ACT_SWIGLU>(a, f32, st);
    }
}

hipError_t ffn_fwd(const FfnArgs& a, bool f32, hipStream_t st) {
    switch (a.act) {
    case ACT_SILU: return ffn_fwd_act<ACT_SILU>(a, f32, st);
    case ACT_RELU: return ffn_fwd_act<ACT_RELU>(a, f32, st);
    default: return ffn_fwd_act<ACT_SWIGLU>(a, f32, st);
    }
}

// bytes of the backward workspace before the expert rank table
inline size_t bwd_main_bytes(size_t S, int d, int f, int E, bool combined, bool h_on_load) {
    // combined: the dX strips (none when they are scattered into dx)
    const size_t part = align256(S * g4_nparts(f) * sizeof(float));  // d_gate partials
    const size_t strip = combined ? S * bwd_strip(S, E, d) * sizeof(bf16_t) : 0;
    if (h_on_load) {   // slot-ordered gates for G3, then (same space) the dX strip
        const size_t gs = S * sizeof(float);
        return part + align256(gs > strip ? gs : strip);
    }
    const size_t hg = S * f * sizeof(bf16_t);                         // g*h, then dX strips
    return part + align256(hg > strip ? hg : strip);
}

size_t ffn_bwd_workspace(int64_t T, int d, int f, int E, int k, bool f32, bool combined,
                         bool h_on_load, bool scatter) {
    const size_t S = (size_t)T * k;
    if (f32) return combined ? align256(S * d * sizeof(float)) : 0;  // dX_slot
    return bwd_main_bytes(S, d, f, E, combined && !scatter, h_on_load) +
           align256(E * sizeof(ExpertRank));
}

namespace {

template <int ACT>
hipError_t ffn_bwd_act(const FfnArgs& a, bool f32, hipStream_t st) {
    const int64_t S = a.T * a.k;
    constexpr bool GATED = ACT == ACT_SWIGLU;
    if (f32) {
        hipLaunchKernelGGL(f32_g3<ACT>, grid1d((int64_t)a.E * a.f * a.d, 256), dim3(256), 0, st,
                           (const float*)a.A, (const float*)a.B, (const float*)a.dy, a.gates,
                           a.offsets, a.eti, a.slot_src, a.d, a.f, a.E, (int)a.accumulate_dw, a.dw2);
        probe::mark("f32_g3", st);
        hipLaunchKernelGGL(f32_g4<ACT>, grid1d(S, 64), dim3(64), 0, st, (const float*)a.dy,
                           (const float*)a.w2, a.gates, a.offsets, a.eti, a.slot_src, S, a.d, a.f,
                           a.E, (float*)a.A, (float*)a.B, a.dgates);
        probe::mark("f32_g4", st);
        hipLaunchKernelGGL(f32_g5<ACT>, grid1d((int64_t)a.E * a.d * a.f, 256), dim3(256), 0, st,
                           (const float*)a.x, (const float*)a.A, (const float*)a.B, a.offsets,
                           a.eti, a.d, a.f, a.E, (int)a.accumulate_dw, a.dw1, a.dw3);
        probe::mark("f32_g5", st);
        float* dX = a.y ? static_cast<float*>(a.ws) : (float*)a.dX;
        hipLaunchKernelGGL(f32_g6<ACT>, grid1d(S * a.d, 256), dim3(256), 0, st, (const float*)a.A,
                           (const float*)a.B, (const float*)a.w1, (const float*)a.w3, a.offsets,
                           S, a.d, a.f, a.E, dX);
        probe::mark("f32_g6", st);
        if (a.y) return combine(dX, nullptr, a.tim, a.T, a.d, a.k, true, a.accumulate, a.y, st);
        return hipGetLastError();
    }
    if (hipError_t e = set_lds_limits(); e != hipSuccess) return e;
    using C5 = CFirst<ACT>;
    using C3H = RHW;
    const int nparts = g4_nparts(a.f);
    float* part = static_cast<float*>(a.ws);
    char* const ws2 = static_cast<char*>(a.ws) + align256((size_t)S * nparts * sizeof(float));
    // default: g*h [S, f] from G4's epilogue for G3; h on load: slot-ordered
    // gates, and G3 (run first, before G4 overwrites A and B) forms g*h itself.
    // Either is finished with before the dX strips reuse the space.
    float* gs = a.h_on_load ? reinterpret_cast<float*>(ws2) : nullptr;
    bf16_t* HG = a.h_on_load ? nullptr : reinterpret_cast<bf16_t*>(ws2);
    bf16_t* strip = reinterpret_cast<bf16_t*>(ws2);
    ExpertRank* rank = reinterpret_cast<ExpertRank*>(
        static_cast<char*>(a.ws) +
        bwd_main_bytes(S, a.d, a.f, a.E, a.y != nullptr && !a.scatter, a.h_on_load));
    hipLaunchKernelGGL(expert_ranks, dim3(1), dim3(256), 0, st, a.offsets, a.E, rank);
    probe::mark("expert_ranks", st);
    // non-gated: the second operand of the two-branch kernels is the first again
    const void* Bx = GATED ? a.B : a.A;
    const void* w3x = GATED ? a.w3 : a.w1;
    if (a.h_on_load) {
        hipLaunchKernelGGL(slot_gates, grid1d(S, 256), dim3(256), 0, st, a.gates,
                           a.slot_src, a.offsets, a.E, S, gs);
        probe::mark("slot_gates", st);
        hipLaunchKernelGGL(g3h_kernel<ACT>, dim3(wgrad_grid(a.E, cdiv(a.f, C3H::BM), cdiv(a.d, C3H::BN))),
                           dim3(C3H::THREADS), C3H::LDS, st, (const bf16_t*)a.A,
                           (const bf16_t*)Bx, (const float*)gs, (const bf16_t*)a.dy, rank,
                           a.eti, a.d, a.f, (int)a.accumulate_dw, a.dw2);
        probe::mark("g3h_kernel", st);
    }
    auto g4 = a.h_on_load ? g4_kernel<ACT, false> : g4_kernel<ACT, true>;
    hipLaunchKernelGGL(g4, dim3(slot_grid(S, a.E, RS::BM, cdiv(a.f, RS::BN))),
                       dim3(RS::THREADS), RS::LDS, st, (const bf16_t*)a.dy, (const bf16_t*)a.w2,
                       a.gates, a.offsets, a.eti, a.slot_src, (const float*)gs, a.d, a.f, a.E,
                       (bf16_t*)a.A, (bf16_t*)a.B, HG, part);
    probe::mark("g4_kernel", st);
    hipLaunchKernelGGL(dgate_reduce, grid1d(S, 256), dim3(256), 0, st, part, nparts, a.slot_src,
                       a.offsets, a.E, S, a.dgates);
    probe::mark("dgate_reduce", st);
    if (!a.h_on_load) {
        hipLaunchKernelGGL(g3_kernel, dim3(wgrad_grid(a.E, cdiv(a.f, RS::BM), cdiv(a.d, RS::BN))),
                           dim3(RS::THREADS), RS::LDS, st, (const bf16_t*)HG, (const bf16_t*)a.dy,
                           rank, a.eti, a.d, a.f, (int)a.accumulate_dw, a.dw2);
        probe::mark("g3_kernel", st);
    }
    hipLaunchKernelGGL(g5_kernel<ACT>, dim3(wgrad_grid(a.E, cdiv(a.d, C5::BM), cdiv(a.f, C5::BN))),
                       dim3(C5::THREADS), C5::LDS, st, (const bf16_t*)a.x, (const bf16_t*)a.A,
                       (const bf16_t*)a.B, rank, a.eti, a.d, a.f, (int)a.accumulate_dw,
                       a.dw1, a.dw3);
    probe::mark("g5_kernel", st);
    const int kslices = (GATED ? 2 : 1) * a.f / rs::KS;
    if (!a.y) {   // dX_slot [S, d] for the caller's combine
        hipLaunchKernelGGL(g6_kernel<false>, dim3(slot_grid(S, a.E, RS::BM, cdiv(a.d, RS::BN))),
                           dim3(RS::THREADS), RS::LDS, st, (const bf16_t*)a.A, (const bf16_t*)Bx,
                           (const bf16_t*)a.w1, (const bf16_t*)w3x, a.offsets, a.d, a.f, a.E,
                           kslices, 0, a.d, (int64_t)a.d, (bf16_t*)a.dX, a.eti);
        probe::mark("g6_kernel", st);
        return hipGetLastError();
    }
    if (a.scatter) {   // every dX_slot row added into dx (cleared first unless accumulating)
        if (!a.accumulate) {
            hipLaunchKernelGGL(zero_bf16, grid1d(a.T * a.d / 8, 256), dim3(256), 0, st,
                               static_cast<bf16_t*>(a.y), a.T * a.d);
            probe::mark("zero_bf16", st);
        }
        hipLaunchKernelGGL(g6_kernel<true>, dim3(slot_grid(S, a.E, RS::BM, cdiv(a.d, RS::BN))),
                           dim3(RS::THREADS), RS::LDS, st, (const bf16_t*)a.A, (const bf16_t*)Bx,
                           (const bf16_t*)a.w1, (const bf16_t*)w3x, a.offsets, a.d, a.f, a.E,
                           kslices, 0, a.d, (int64_t)a.d, static_cast<bf16_t*>(a.y), a.eti);
        probe::mark("g6_kernel", st);
        return hipGetLastError();
    }
    // combined: one column strip of dX_slot at a time, summed straight into dx;
    // by default the strip reuses g*h's workspace, which G3 has finished with
    const int sw = bwd_strip(S, a.E, a.d);
    for (int c0 = 0; c0 < a.d; c0 += sw) {
        const int nc = min(sw, a.d - c0);
        hipLaunchKernelGGL(g6_kernel<false>, dim3(slot_grid(S, a.E, RS::BM, cdiv(nc, RS::BN))),
                           dim3(RS::THREADS), RS::LDS, st, (const bf16_t*)a.A, (const bf16_t*)Bx,
                           (const bf16_t*)a.w1, (const bf16_t*)w3x, a.offsets, a.d, a.f, a.E,
                           kslices, c0, nc, (int64_t)nc, strip, a.eti);
        probe::mark("g6_kernel", st);
        if (hipError_t e = combine_cols(strip, nc, nullptr, a.tim, a.T, nc, a.k, false,
                                        a.accumulate, static_cast<bf16_t*>(a.y) + c0, a.d, st);
            e != hipSuccess)
            return e;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t ffn_bwd(const FfnArgs& a, bool f32, hipStream_t st) {
    switch (a.act) {
    case ACT_SILU: return ffn_bwd_act<ACT_SILU>(a, f32, st);
    case ACT_RELU: return ffn_bwd_act<ACT_RELU>(a, f32, st);
    default: return ffn_bwd_act<ACT_SWIGLU>(a, f32, st);
    }
}

}  // namespace moe
