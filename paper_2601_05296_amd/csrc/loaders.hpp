// loaders.hpp -- operand loaders of the grouped GEMM core (gemm.hpp).
//
// Each loader issues the 1 KB global->LDS copies of one operand tile for one
// K slice, in the LDS layout the core expects (KC or MC). Rows or columns at
// or beyond the operand's extent are clamped to valid memory; the epilogues
// never store the outputs that depend on them.
#pragma once

#include "gemm.hpp"

namespace moe {

template <class C, int R>
struct KCBase {
    static constexpr bool MC = false;
    static constexpr int NQ = R * GBK * 2 / 1024 / C::NW;  // copies per wave per slice
    __device__ static int q(int i) { return wave_id() + i * C::NW; }
};

// KC rows gathered through an index list: row r -> base[idx[r]] (rows at or
// beyond `rows` read row 0).
template <class C, int R>
struct GatherKC : KCBase<C, R> {
    using KCBase<C, R>::NQ;
    const bf16_t* p[NQ];
    __device__ void init(const bf16_t* base, int ld, const int32_t* idx, int rows) {
        const int lane = threadIdx.x & 63;
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
            const int q = this->q(i);
            int r = KCDma::row(q, lane);
            r = r < rows ? r : 0;
            p[i] = base + (int64_t)idx[r] * ld + KCDma::kcol(q, lane);
        }
    }
    __device__ void issue(int kt, uint32_t t) {
#pragma unroll
        for (int i = 0; i < NQ; ++i) dma16(p[i] + kt * GBK, t + this->q(i) * 1024u);
    }
};

// KC rows row0 + r (r < rows, else row0) of a dense row-major matrix, K split
// over two sources: k < ksplit from src0, k >= ksplit from src1 (same ld).
template <class C, int R>
struct DenseKC2 : KCBase<C, R> {
    using KCBase<C, R>::NQ;
    const bf16_t* p0[NQ];
    const bf16_t* p1[NQ];
    int kst;  // K slices served by src0
    __device__ void init(const bf16_t* src0, const bf16_t* src1, int ld, int64_t row0, int rows,
                         int ksplit) {
        const int lane = threadIdx.x & 63;
        kst = ksplit / GBK;
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
            const int q = this->q(i);
            int r = KCDma::row(q, lane);
            r = r < rows ? r : 0;
            const int64_t o = (row0 + r) * (int64_t)ld + KCDma::kcol(q, lane);
            p0[i] = src0 + o;
            p1[i] = src1 + o - (int64_t)ksplit;
        }
    }
    __device__ void issue(int kt, uint32_t t) {
        const bool first = kt < kst;
#pragma unroll
        for (int i = 0; i < NQ; ++i)
            dma16((first ? p0[i] : p1[i]) + kt * GBK, t + this->q(i) * 1024u);
    }
};

// Two KC tiles of the same rows row0 + r (r < rows, else row0) from two
// row-major matrices of equal shape: src0 into the left operand's tile, src1
// into the extra tile after it (GemmCfg XA = 1).
template <class C, int R>
struct PairKC : KCBase<C, R> {
    static constexpr int NQ1 = KCBase<C, R>::NQ;
    static constexpr int NQ = 2 * NQ1;   // copies per wave per slice, both tiles
    static_assert(C::XA == 1 && R == C::BM, "pair tiles fill the left operand and its extra tile");
    const bf16_t* p0[NQ1];
    const bf16_t* p1[NQ1];
    __device__ void init(const bf16_t* src0, const bf16_t* src1, int ld, int64_t row0, int rows) {
        const int lane = threadIdx.x & 63;
#pragma unroll
        for (int i = 0; i < NQ1; ++i) {
            const int q = this->q(i);
            int r = KCDma::row(q, lane);
            r = r < rows ? r : 0;
            const int64_t o = (row0 + r) * (int64_t)ld + KCDma::kcol(q, lane);
            p0[i] = src0 + o;
            p1[i] = src1 + o;
        }
    }
    __device__ void issue(int kt, uint32_t t) {
#pragma unroll
        for (int i = 0; i < NQ1; ++i) {
            dma16(p0[i] + kt * GBK, t + this->q(i) * 1024u);
            dma16(p1[i] + kt * GBK, t + C::A_BYTES + this->q(i) * 1024u);
        }
    }
};

template <class C, int R>
struct MCBase {
    static constexpr bool MC = true;
    using D = MCDma<R>;
    static constexpr int NQ = GBK * R * 2 / 1024 / C::NW;
    __device__ static int q(int i) { return wave_id() + i * C::NW; }
    // column of copy i for this lane, clamped into [0, ncols)
    __device__ static int colc(int i, int col0, int ncols) {
        const int c = col0 + D::col(q(i), threadIdx.x & 63);
        return c < ncols ? c : ncols - 8;
    }
    __device__ static int krow(int i) { return D::krow(q(i), threadIdx.x & 63); }
};

// MC tile of a dense row-major [K][ncols] matrix, columns col0..
template <class C, int R>
struct DenseMC : MCBase<C, R> {
    using MCBase<C, R>::NQ;
    const bf16_t* p[NQ];
    int64_t step;
    __device__ void init(const bf16_t* W, int ld, int col0, int ncols) {
        step = (int64_t)GBK * ld;
#pragma unroll
        for (int i = 0; i < NQ; ++i)
            p[i] = W + (int64_t)this->krow(i) * ld + this->colc(i, col0, ncols);
    }
    __device__ void issue(int kt, uint32_t t) {
#pragma unroll
        for (int i = 0; i < NQ; ++i) dma16(p[i] + kt * step, t + this->q(i) * 1024u);
    }
};

// ---- loaders whose K is the slot dimension of one expert (weight gradients) ----
// K row kr (0 <= kr < cnt) is slot off + kr; rows at or past cnt are clamped to
// row cnt - 1 (the main loop zeroes them in the left operand).

// MC rows gathered through eti: row kr -> base[eti[off + kr]] (x or dY).
// The k rows covered by one copy are the same for the whole wave (KPK of
// them, one per group of R/8 lanes), so their indices are read with scalar
// loads, one slice ahead of the copies that use them.
template <class C, int R>
struct GatherMC : MCBase<C, R> {
    using MCBase<C, R>::NQ;
    using D = MCDma<R>;
    const bf16_t* base[NQ];
    const int32_t* idx;  // eti + off
    int ld, cnt;
    int nidx[NQ][D::KPK];
    __device__ void load_idx(int kt) {
#pragma unroll
        for (int i = 0; i < NQ; ++i)
#pragma unroll
            for (int h = 0; h < D::KPK; ++h) {
                int kr = kt * GBK + this->q(i) * D::KPK + h;
                kr = kr < cnt ? kr : cnt - 1;
                // constant address space: a uniform address becomes a scalar load
                nidx[i][h] = ((const __attribute__((address_space(4))) int32_t*)(idx))[kr];
            }
    }
    __device__ void init(const bf16_t* b, int ld_, int col0, int ncols, const int32_t* ix,
                         int cnt_) {
        ld = ld_;
        idx = ix;
        cnt = cnt_;
#pragma unroll
        for (int i = 0; i < NQ; ++i) base[i] = b + this->colc(i, col0, ncols);
        load_idx(0);
    }
    __device__ void issue(int kt, uint32_t t) {
        const int h = (threadIdx.x & 63) / D::CPR;
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
            int row = nidx[i][0];
#pragma unroll
            for (int hh = 1; hh < D::KPK; ++hh) row = h == hh ? nidx[i][hh] : row;
            dma16(base[i] + (int64_t)row * ld, t + this->q(i) * 1024u);
        }
        load_idx(kt + 1);
    }
};

// MC rows of a slot-ordered matrix (g*h, dA or dB): row kr -> src[off + kr].
template <class C, int R>
struct SlotMC : MCBase<C, R> {
    using MCBase<C, R>::NQ;
    const bf16_t* base[NQ];
    int ld, cnt;
    __device__ void init(const bf16_t* src, int ld_, int64_t off, int col0, int ncols, int cnt_) {
        ld = ld_;
        cnt = cnt_;
#pragma unroll
        for (int i = 0; i < NQ; ++i) base[i] = src + off * ld_ + this->colc(i, col0, ncols);
    }
    __device__ void issue(int kt, uint32_t t) {
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
            int kr = kt * GBK + this->krow(i);
            kr = kr < cnt ? kr : cnt - 1;
            dma16(base[i] + (int64_t)kr * ld, t + this->q(i) * 1024u);
        }
    }
};


// MC tile of a [K][ncols] matrix whose K rows come from two row ranges of the
// same matrix: k < ksplit -> row k, k >= ksplit -> row k - ksplit; rows at or
// beyond nrows are clamped (the other operand is zero there).
// MC tiles of slot rows off + kr (kr < cnt, else cnt - 1) of one or two
// row-major [S][ld] matrices (NSRC = 2: the second into the extra tile,
// GemmCfg XA = 1), and the slice's 32 per-slot gates (float32, slot order,
// padded with zeros past the last slot) into a 128-byte slot of the gate
// array that follows the LDS ring. Every wave copies the same gate bytes, so
// that all waves count the same number of copies per slice.
template <class C, int R, int NSRC>
struct SlotMCG : MCBase<C, R> {
    static constexpr int NQ1 = MCBase<C, R>::NQ;
    static constexpr int NQ = NSRC * NQ1 + 1;
    static_assert(NSRC == 1 + C::XA && R == C::BM, "one tile per source, left operand shape");
    const bf16_t* base0[NQ1];
    const bf16_t* base1[NQ1];
    const float* gs;        // gates of slots off, off + 1, ...
    int ld, cnt;
    uint32_t gate_lds;      // LDS offset of the gate array (NST slots of 128 bytes)
    __device__ void init(const bf16_t* src0, const bf16_t* src1, int ld_, int64_t off, int col0,
                         int ncols, int cnt_, const float* gates_slot, uint32_t gate_lds_) {
        ld = ld_;
        cnt = cnt_;
        gs = gates_slot + off;
        gate_lds = gate_lds_;
#pragma unroll
        for (int i = 0; i < NQ1; ++i) {
            base0[i] = src0 + off * ld_ + this->colc(i, col0, ncols);
            base1[i] = src1 + off * ld_ + this->colc(i, col0, ncols);
        }
    }
    __device__ void issue(int kt, uint32_t t) {
#pragma unroll
        for (int i = 0; i < NQ1; ++i) {
            int kr = kt * GBK + this->krow(i);
            kr = kr < cnt ? kr : cnt - 1;
            dma16(base0[i] + (int64_t)kr * ld, t + this->q(i) * 1024u);
            if constexpr (NSRC == 2)
                dma16(base1[i] + (int64_t)kr * ld, t + C::A_BYTES + this->q(i) * 1024u);
        }
        const int lane = threadIdx.x & 63;
        if (lane < GBK) dma4(gs + kt * GBK + lane, gate_lds + (kt % NST) * 128u);
    }
};

template <class C, int R>
struct SplitRowsMC : MCBase<C, R> {
    using MCBase<C, R>::NQ;
    const bf16_t* base[NQ];
    int ld, ksplit, nrows;
    __device__ void init(const bf16_t* W, int ld_, int col0, int ncols, int ksplit_, int nrows_) {
        ld = ld_;
        ksplit = ksplit_;
        nrows = nrows_;
#pragma unroll
        for (int i = 0; i < NQ; ++i) base[i] = W + this->colc(i, col0, ncols);
    }
    __device__ void issue(int kt, uint32_t t) {
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
            int k = kt * GBK + this->krow(i);
            k = k < ksplit ? k : k - ksplit;
            k = k < nrows ? k : nrows - 1;
            dma16(base[i] + (int64_t)k * ld, t + this->q(i) * 1024u);
        }
    }
};

// k rows of the last slice at or beyond a K extent of cnt rows (GBK: none)
__device__ __forceinline__ int tail_from(int cnt) {
    const int r = cnt % GBK;
    return r == 0 ? GBK : r;
}

}  // namespace moe
