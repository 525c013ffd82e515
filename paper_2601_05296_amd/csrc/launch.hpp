// launch.hpp -- internal launchers behind the C ABI (arguments already
// validated by api.hip). Each returns hipSuccess or the launch error.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace moe {

// ---- dispatch index build ----
size_t build_index_workspace(int64_t T, int E, int k);
hipError_t build_index(const int32_t* ids, int64_t T, int E, int k, int32_t* counts,
                       int32_t* offsets, int32_t* eti, int32_t* tim, int32_t* slot_src,
                       void* ws, hipStream_t st);
// device address and size of the static scratch of the no-allocation index
// build on the current device (looked up once per device)
hipError_t noalloc_scratch(void** ptr, size_t* bytes);

// ---- routing ----
hipError_t route(const void* x, const void* wg, const float* bias, int64_t T, int d, int E,
                 int k, bool f32, bool renorm, int32_t* ids, float* gates, float* logits,
                 hipStream_t st);
size_t route_bwd_workspace(int64_t T, int d, int E, int k, bool f32);
hipError_t route_bwd(const float* dgates, const float* logits, const int32_t* ids,
                     const float* gates, const void* x, const void* wg, int64_t T, int d,
                     int E, int k, bool f32, bool renorm, bool accumulate, float* dwg,
                     void* dx, void* ws, hipStream_t st);

// ---- combine ----
hipError_t combine(const void* src, const float* w, const int32_t* tim, int64_t T, int d,
                   int k, bool f32, bool accumulate, void* out, hipStream_t st);
// the same on one column strip: ncols columns of source rows src_ld elements
// apart into output rows out_ld elements apart
hipError_t combine_cols(const void* src, int64_t src_ld, const float* w, const int32_t* tim,
                        int64_t T, int ncols, int k, bool f32, bool accumulate, void* out,
                        int64_t out_ld, hipStream_t st);

// ---- expert FFN ----
struct FfnArgs {
    const void* x; const void* w1; const void* w3; const void* w2;
    const int32_t* offsets; const int32_t* eti; const int32_t* slot_src;
    const float* gates; const void* dy;
    void* A; void* B; void* O; void* dX;
    float* dw1; float* dw3; float* dw2; float* dgates;
    int64_t T; int d, f, E, k;
    int act;  // 0 SwiGLU (gated), 1 SiLU, 2 ReLU (non-gated: w3, B, dw3 unused)
    void* ws;
    // combined calls: y (forward) or dx (backward) [T, d] written through
    // token_index_map instead of O / dX_slot; accumulate adds into dx
    void* y; const int32_t* tim; bool accumulate;
    // h is not buffered: the second GEMM forms it again from A (and B) on load
    bool h_on_load;
    // backward: add the weight gradients into dw1, dw3, dw2
    bool accumulate_dw;
    // combined calls: the second GEMM (forward) or the dX GEMM (backward) adds
    // its rows into y / dx with atomics instead of strips and a gather-reduce
    bool scatter;
};
size_t ffn_fwd_workspace(int64_t T, int d, int f, int E, int k, bool f32, bool combined,
                         bool h_on_load, bool scatter);
hipError_t ffn_fwd(const FfnArgs& a, bool f32, hipStream_t st);
// first layer only: A (and B) from x, nothing else
hipError_t ffn_first(const FfnArgs& a, bool f32, hipStream_t st);
size_t ffn_bwd_workspace(int64_t T, int d, int f, int E, int k, bool f32, bool combined,
                         bool h_on_load, bool scatter);
hipError_t ffn_bwd(const FfnArgs& a, bool f32, hipStream_t st);

}  // namespace moe
