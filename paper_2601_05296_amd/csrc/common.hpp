// common.hpp -- device helpers shared by the gfx950 kernels of the MoE layer.
//
// bfloat16 values travel as raw 16-bit patterns (uint16_t in memory, 8 of
// them per 16-byte vector). Matrix-core work uses the gfx950 instruction
// v_mfma_f32_16x16x32_bf16 with float32 accumulation.
//
// MFMA 16x16x32 operand layout (wave64), verified on gfx950: for D = P * Q,
// lane L supplies P[L%16][8*(L/16) + 0..7] and Q[8*(L/16) + 0..7][L%16], and
// receives D[4*(L/16) + r][L%16] for r = 0..3. The GEMM kernels call it with
// P = a tile of the right operand (rows = output columns n) and Q = a tile of
// the left operand (columns = output rows m), so that lane L ends up holding
// output row m = L%16 at the four consecutive columns n = 4*(L/16) + r.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;  // storage pattern

constexpr int WAVE = 64;

// ---- bfloat16 <-> float32 ---------------------------------------------------
__device__ __forceinline__ float bf2f(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round to nearest even (NaN stays NaN) with gfx950's v_cvt_pk_bf16_f32, one
// instruction per pair. Checked on the device against the integer form
// (u + 0x7fff + lsb) >> 16 over all 2^32 float32 bit patterns: equal for every
// non-NaN input.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
    const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ uint32_t f2bf(float f) { return pack_bf2(f, 0.0f) & 0xffffu; }

// unpack 8 bf16 (one 16-byte vector) to float
__device__ __forceinline__ void unpack8(const uint4& v, float (&o)[8]) {
    o[0] = bf_lo(v.x); o[1] = bf_hi(v.x); o[2] = bf_lo(v.y); o[3] = bf_hi(v.y);
    o[4] = bf_lo(v.z); o[5] = bf_hi(v.z); o[6] = bf_lo(v.w); o[7] = bf_hi(v.w);
}
__device__ __forceinline__ uint4 pack8(const float (&o)[8]) {
    uint4 v;
    v.x = pack_bf2(o[0], o[1]); v.y = pack_bf2(o[2], o[3]);
    v.z = pack_bf2(o[4], o[5]); v.w = pack_bf2(o[6], o[7]);
    return v;
}

// Inclusive prefix sum over the 64 lanes of a wave, by DPP lane moves: a
// Hillis-Steele scan inside each row of 16 lanes (row_shr 1, 2, 4, 8; a lane
// whose source lies before its row's start adds 0), then the last lane of row
// 0 and of row 2 added into rows 1 and 3 (row_bcast:15, row mask 0b1010) and
// the last lane of row 1 into rows 2 and 3 (row_bcast:31, row mask 0b1100).
__device__ __forceinline__ int wave_incl_scan(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);   // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);   // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);   // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);   // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);   // row_bcast:15
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);   // row_bcast:31
    return v;
}

// ---- activation -------------------------------------------------------------
// logistic function with the hardware reciprocal (v_rcp_f32, about 1 ulp)
// instead of a correctly rounded divide, which takes some ten instructions
__device__ __forceinline__ float sigmoidf_(float u) {
    return __builtin_amdgcn_rcpf(1.0f + __expf(-u));
}

// ---- memory helpers -----------------------------------------------------------
__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ void st16(void* p, const uint4& v) { *reinterpret_cast<uint4*>(p) = v; }
// streaming store of 16 bytes to global memory; only for stores that cover
// whole 128-byte lines (partial-line nontemporal stores measured slower than
// plain ones). The pointer is cast to the global address space: where the
// compiler cannot infer it, it would otherwise emit a flat store, which also
// counts as an LDS access for the wait counters.
__device__ __forceinline__ void st16_nt(void* p, const uint4& v) {
    typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(1))) u32x4_t* gptr_t;
    __builtin_nontemporal_store(u32x4_t{v.x, v.y, v.z, v.w}, (gptr_t)p);
}
__device__ __forceinline__ uint4 zero16() { return make_uint4(0u, 0u, 0u, 0u); }

// ---- MFMA ---------------------------------------------------------------------
__device__ __forceinline__ f32x4 mfma16x16x32(const bf16x8& p, const bf16x8& q, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(p, q, c, 0, 0, 0);
}

// ---- XCD-aware block order ------------------------------------------------------
// Consecutive hardware workgroup ids are dealt round-robin to the 8 XCDs (each
// with its own L2). Renumber so that every XCD works on one contiguous range of
// logical tiles, which keeps neighbouring tiles (sharing operand panels) in the
// same L2. Bijective for any grid size.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
    const int q = nblocks >> 3, r = nblocks & 7;
    const int x = bid & 7, i = bid >> 3;
    return x * q + (x < r ? x : r) + i;
}

// ---- wave reductions ------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, WAVE);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, WAVE));
    return v;
}

}  // namespace moe
