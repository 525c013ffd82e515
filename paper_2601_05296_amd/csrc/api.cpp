// api.cpp -- the extern "C" entry points of libmoeblaze.so: argument
// validation (before anything is enqueued), then the internal launchers.
#include <stdarg.h>
#include <stdio.h>

#include "../../include/moeblaze.h"
#include "launch.hpp"
#include "probe.hpp"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQUIRE_PTR(p)                                                                 \
    do {                                                                               \
        if (!(p)) return fail(MOE_ERR_INVALID_ARG, "%s: %s is NULL", fn, #p);          \
        if (!aligned16(p)) return fail(MOE_ERR_INVALID_ARG, "%s: %s is not 16-byte aligned", fn, #p); \
    } while (0)
#define OPT_PTR(p)                                                                     \
    do {                                                                               \
        if ((p) && !aligned16(p))                                                      \
            return fail(MOE_ERR_INVALID_ARG, "%s: %s is not 16-byte aligned", fn, #p); \
    } while (0)

const unsigned KNOWN_FLAGS = MOE_F32 | MOE_RENORM | MOE_ACCUMULATE | MOE_ACT_SILU |
                             MOE_ACT_RELU | MOE_H_ON_LOAD | MOE_ACCUMULATE_DW |
                             MOE_ATOMIC_COMBINE;
const unsigned ACT_FLAGS = MOE_ACT_SILU | MOE_ACT_RELU;
// meaningful to the FFN calls only
const unsigned FFN_ONLY = ACT_FLAGS | MOE_H_ON_LOAD | MOE_ACCUMULATE_DW | MOE_ATOMIC_COMBINE;

// MOE_ATOMIC_COMBINE: combined bf16 calls only
int check_scatter(const char* fn, bool combined, unsigned flags) {
    if (!(flags & MOE_ATOMIC_COMBINE)) return MOE_OK;
    if (!combined)
        return fail(MOE_ERR_INVALID_ARG, "%s: MOE_ATOMIC_COMBINE applies to the combined calls only", fn);
    if (flags & MOE_F32)
        return fail(MOE_ERR_UNSUPPORTED, "%s: MOE_ATOMIC_COMBINE is bfloat16 only", fn);
    return MOE_OK;
}

// expert activation code of the FFN calls (0 SwiGLU, 1 SiLU, 2 ReLU), or -1
int act_of(unsigned flags) {
    const unsigned a = flags & ACT_FLAGS;
    return a == 0 ? 0 : a == MOE_ACT_SILU ? 1 : a == MOE_ACT_RELU ? 2 : -1;
}

int check_common(const char* fn, int64_t T, int E, int k, unsigned flags) {
    if (T < 0) return fail(MOE_ERR_INVALID_ARG, "%s: T = %lld < 0", fn, (long long)T);
    if (E < 1) return fail(MOE_ERR_INVALID_ARG, "%s: E = %d < 1", fn, E);
    if (k < 1) return fail(MOE_ERR_INVALID_ARG, "%s: k = %d < 1", fn, k);
    if (k > E) return fail(MOE_ERR_INVALID_ARG, "%s: k = %d > E = %d", fn, k, E);
    if (flags & ~KNOWN_FLAGS) return fail(MOE_ERR_INVALID_ARG, "%s: unknown flag bits 0x%x", fn, flags);
    if (E > 256) return fail(MOE_ERR_UNSUPPORTED, "%s: E = %d > 256", fn, E);
    if (k > 16) return fail(MOE_ERR_UNSUPPORTED, "%s: k = %d > 16", fn, k);
    if (T * (int64_t)k >= (int64_t(1) << 31))
        return fail(MOE_ERR_UNSUPPORTED, "%s: T*k = %lld does not fit int32 slots", fn,
                    (long long)(T * k));
    return MOE_OK;
}

int check_dim(const char* fn, const char* name, int v) {
    if (v < 1) return fail(MOE_ERR_INVALID_ARG, "%s: %s = %d < 1", fn, name, v);
    if (v % 64) return fail(MOE_ERR_UNSUPPORTED, "%s: %s = %d is not a multiple of 64", fn, name, v);
    return MOE_OK;
}

int hip_status(const char* fn, hipError_t e) {
    if (e != hipSuccess) return fail(MOE_ERR_HIP, "%s: %s", fn, hipGetErrorString(e));
    return MOE_OK;
}

}  // namespace

namespace {

// moe_ffn_fwd and moe_ffn_fwd_combine: O (plain) or y via gates and
// token_index_map (combined)
int ffn_fwd_impl(const char* fn, bool combined, const void* x, const void* w1, const void* w3,
                 const void* w2, const int32_t* offsets, const int32_t* expert_token_indices,
                 const float* gates, const int32_t* token_index_map, int64_t T, int d, int f,
                 int E, int k, unsigned flags, void* A, void* B, void* out, void* workspace,
                 size_t workspace_bytes, hipStream_t stream) {
    int r;
    if ((r = check_common(fn, T, E, k, flags)) || (r = check_dim(fn, "d", d)) ||
        (r = check_dim(fn, "f", f)))
        return r;
    if (flags & (MOE_RENORM | MOE_ACCUMULATE | MOE_ACCUMULATE_DW))
        return fail(MOE_ERR_INVALID_ARG, "%s: only MOE_F32 / MOE_BF16, an activation flag, MOE_H_ON_LOAD and (combined) MOE_ATOMIC_COMBINE are valid", fn);
    if ((r = check_scatter(fn, combined, flags))) return r;
    const int act = act_of(flags);
    if (act < 0) return fail(MOE_ERR_INVALID_ARG, "%s: MOE_ACT_SILU and MOE_ACT_RELU both set", fn);
    if (T == 0) return MOE_OK;
    REQUIRE_PTR(x); REQUIRE_PTR(w1); REQUIRE_PTR(w2); REQUIRE_PTR(offsets);
    REQUIRE_PTR(expert_token_indices); REQUIRE_PTR(A);
    if (combined) {
        const void* y = out;
        REQUIRE_PTR(gates); REQUIRE_PTR(token_index_map); REQUIRE_PTR(y);
    } else {
        const void* O = out;
        REQUIRE_PTR(O);
    }
    if (act == 0) { REQUIRE_PTR(w3); REQUIRE_PTR(B); }
    else { OPT_PTR(w3); OPT_PTR(B); }
    const size_t need =
        moe::ffn_fwd_workspace(T, d, f, E, k, flags & MOE_F32, combined, flags & MOE_H_ON_LOAD,
                               flags & MOE_ATOMIC_COMBINE);
    if (need && (!workspace || workspace_bytes < need))
        return fail(MOE_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, workspace_bytes, need);
    OPT_PTR(workspace);
    moe::FfnArgs a{};
    a.x = x; a.w1 = w1; a.w3 = w3; a.w2 = w2; a.offsets = offsets; a.eti = expert_token_indices;
    a.A = A; a.B = B; a.T = T; a.d = d; a.f = f; a.E = E; a.k = k; a.ws = workspace;
    a.act = act;
    a.h_on_load = flags & MOE_H_ON_LOAD;
    a.scatter = flags & MOE_ATOMIC_COMBINE;
    if (combined) { a.y = out; a.gates = gates; a.tim = token_index_map; }
    else a.O = out;
    moe::probe::begin(stream);
    return hip_status(fn, moe::ffn_fwd(a, flags & MOE_F32, stream));
}

}  // namespace

namespace {

// moe_ffn_bwd and moe_ffn_bwd_combine: dX_slot (plain) or dx through
// token_index_map (combined; MOE_ACCUMULATE adds into dx)
int ffn_bwd_impl(const char* fn, bool combined, const void* dy, const void* x, const void* w1,
                 const void* w3, const void* w2, const float* gates, const int32_t* offsets,
                 const int32_t* expert_token_indices, const int32_t* slot_src,
                 const int32_t* token_index_map, void* A, void* B, int64_t T, int d, int f,
                 int E, int k, unsigned flags, float* dw1, float* dw3, float* dw2,
                 float* d_gates, void* out, void* workspace, size_t workspace_bytes,
                 hipStream_t stream) {
    int r;
    if ((r = check_common(fn, T, E, k, flags)) || (r = check_dim(fn, "d", d)) ||
        (r = check_dim(fn, "f", f)))
        return r;
    if ((flags & MOE_RENORM) || (!combined && (flags & MOE_ACCUMULATE)))
        return fail(MOE_ERR_INVALID_ARG, "%s: flag not valid here", fn);
    if ((r = check_scatter(fn, combined, flags))) return r;
    const int act = act_of(flags);
    if (act < 0) return fail(MOE_ERR_INVALID_ARG, "%s: MOE_ACT_SILU and MOE_ACT_RELU both set", fn);
    if (T == 0) return MOE_OK;
    REQUIRE_PTR(dy); REQUIRE_PTR(x); REQUIRE_PTR(w1); REQUIRE_PTR(w2);
    REQUIRE_PTR(gates); REQUIRE_PTR(offsets); REQUIRE_PTR(expert_token_indices);
    REQUIRE_PTR(slot_src); REQUIRE_PTR(A); REQUIRE_PTR(dw1);
    REQUIRE_PTR(dw2); REQUIRE_PTR(d_gates);
    if (combined) {
        const void* dx = out;
        REQUIRE_PTR(token_index_map); REQUIRE_PTR(dx);
    } else {
        const void* dX_slot = out;
        REQUIRE_PTR(dX_slot);
    }
    if (act == 0) { REQUIRE_PTR(w3); REQUIRE_PTR(B); REQUIRE_PTR(dw3); }
    else { OPT_PTR(w3); OPT_PTR(B); OPT_PTR(dw3); }
    const size_t need =
        moe::ffn_bwd_workspace(T, d, f, E, k, flags & MOE_F32, combined, flags & MOE_H_ON_LOAD,
                               flags & MOE_ATOMIC_COMBINE);
    if (need && (!workspace || workspace_bytes < need))
        return fail(MOE_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, workspace_bytes, need);
    OPT_PTR(workspace);
    moe::FfnArgs a{};
    a.x = x; a.w1 = w1; a.w3 = w3; a.w2 = w2; a.offsets = offsets; a.eti = expert_token_indices;
    a.slot_src = slot_src; a.gates = gates; a.dy = dy; a.A = A; a.B = B;
    a.dw1 = dw1; a.dw3 = dw3; a.dw2 = dw2; a.dgates = d_gates; a.T = T; a.d = d; a.f = f;
    a.E = E; a.k = k; a.ws = workspace; a.act = act;
    a.h_on_load = flags & MOE_H_ON_LOAD;
    a.accumulate_dw = flags & MOE_ACCUMULATE_DW;
    a.scatter = flags & MOE_ATOMIC_COMBINE;
    if (combined) { a.y = out; a.tim = token_index_map; a.accumulate = flags & MOE_ACCUMULATE; }
    else a.dX = out;
    moe::probe::begin(stream);
    return hip_status(fn, moe::ffn_bwd(a, flags & MOE_F32, stream));
}

}  // namespace

extern "C" {

const char* moe_strerror(int status) {
    switch (status) {
        case MOE_OK: return "MOE_OK";
        case MOE_ERR_INVALID_ARG: return "MOE_ERR_INVALID_ARG";
        case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED";
        case MOE_ERR_WORKSPACE: return "MOE_ERR_WORKSPACE";
        case MOE_ERR_HIP: return "MOE_ERR_HIP";
        default: return "unknown status";
    }
}

const char* moe_last_error(void) { return g_err; }

int moe_probe_enable(int capacity) {
    if (capacity < 1) return fail(MOE_ERR_INVALID_ARG, "moe_probe_enable: capacity %d < 1", capacity);
    if (moe::probe::enable(capacity) != 0)
        return fail(MOE_ERR_HIP, "moe_probe_enable: hipEventCreate failed");
    return MOE_OK;
}

void moe_probe_disable(void) { moe::probe::disable(); }

int moe_probe_count(void) { return moe::probe::count(); }

int moe_probe_dropped(void) { return moe::probe::dropped(); }

int moe_probe_get(int index, const char** kernel_name, float* ms) {
    if (!kernel_name || !ms) return fail(MOE_ERR_INVALID_ARG, "moe_probe_get: NULL output");
    if (moe::probe::get(index, kernel_name, ms) != 0)
        return fail(MOE_ERR_INVALID_ARG, "moe_probe_get: no record %d", index);
    return MOE_OK;
}

int moe_route(const void* x, const void* w_gate, const float* bias, int64_t T, int d, int E,
              int k, unsigned flags, int32_t* topk_ids, float* gates, float* logits,
              hipStream_t stream) {
    const char* fn = "moe_route";
    int r;
    if ((r = check_common(fn, T, E, k, flags)) || (r = check_dim(fn, "d", d))) return r;
    if (flags & FFN_ONLY) return fail(MOE_ERR_INVALID_ARG, "%s: activation, h-on-load and weight-gradient accumulation flags apply to the FFN calls only", fn);
    if (flags & MOE_ACCUMULATE) return fail(MOE_ERR_INVALID_ARG, "%s: MOE_ACCUMULATE not valid here", fn);
    if (T == 0) return MOE_OK;
    REQUIRE_PTR(x); REQUIRE_PTR(w_gate); OPT_PTR(bias); REQUIRE_PTR(topk_ids); REQUIRE_PTR(gates);
    OPT_PTR(logits);
    moe::probe::begin(stream);
    return hip_status(fn, moe::route(x, w_gate, bias, T, d, E, k, flags & MOE_F32,
                                     flags & MOE_RENORM, topk_ids, gates, logits, stream));
}

size_t moe_build_index_workspace_size(int64_t T, int E, int k) {
    if (T <= 0 || E < 1 || k < 1) return 0;
    return moe::build_index_workspace(T, E, k);
}

int moe_build_index(const int32_t* topk_ids, int64_t T, int E, int k, int32_t* counts,
                    int32_t* offsets, int32_t* expert_token_indices, int32_t* token_index_map,
                    int32_t* slot_src, void* workspace, size_t workspace_bytes,
                    hipStream_t stream) {
    const char* fn = "moe_build_index";
    int r;
    if ((r = check_common(fn, T, E, k, 0))) return r;
    if (T == 0) return MOE_OK;
    REQUIRE_PTR(topk_ids); REQUIRE_PTR(counts); REQUIRE_PTR(offsets);
    REQUIRE_PTR(expert_token_indices); REQUIRE_PTR(token_index_map); REQUIRE_PTR(slot_src);
    const size_t need = moe::build_index_workspace(T, E, k);
    if (!workspace || workspace_bytes < need)
        return fail(MOE_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, workspace_bytes, need);
    REQUIRE_PTR(workspace);
    moe::probe::begin(stream);
    return hip_status(fn, moe::build_index(topk_ids, T, E, k, counts, offsets, expert_token_indices,
                                           token_index_map, slot_src, workspace, stream));
}

int moe_build_index_noalloc(const int32_t* topk_ids, int64_t T, int E, int k, int32_t* counts,
                            int32_t* offsets, int32_t* expert_token_indices,
                            int32_t* token_index_map, int32_t* slot_src, hipStream_t stream) {
    const char* fn = "moe_build_index_noalloc";
    int r;
    if ((r = check_common(fn, T, E, k, 0))) return r;
    if (T == 0) return MOE_OK;
    REQUIRE_PTR(topk_ids); REQUIRE_PTR(counts); REQUIRE_PTR(offsets);
    REQUIRE_PTR(expert_token_indices); REQUIRE_PTR(token_index_map); REQUIRE_PTR(slot_src);
    void* ws = nullptr;
    size_t have = 0;
    if (hipError_t e = moe::noalloc_scratch(&ws, &have); e != hipSuccess)
        return fail(MOE_ERR_HIP, "%s: scratch address lookup failed: %s", fn, hipGetErrorString(e));
    const size_t need = moe::build_index_workspace(T, E, k);
    if (need > have)
        return fail(MOE_ERR_UNSUPPORTED, "%s: needs %zu bytes of scratch, the static scratch holds %zu",
                    fn, need, have);
    moe::probe::begin(stream);
    return hip_status(fn, moe::build_index(topk_ids, T, E, k, counts, offsets, expert_token_indices,
                                           token_index_map, slot_src, ws, stream));
}

size_t moe_ffn_fwd_workspace_size(int64_t T, int d, int f, int E, int k, unsigned flags) {
    if (T <= 0 || d < 1 || f < 1 || E < 1 || k < 1) return 0;
    return moe::ffn_fwd_workspace(T, d, f, E, k, flags & MOE_F32, false, flags & MOE_H_ON_LOAD,
                                  false);
}

int moe_ffn_fwd(const void* x, const void* w1, const void* w3, const void* w2,
                const int32_t* offsets, const int32_t* expert_token_indices, int64_t T, int d,
                int f, int E, int k, unsigned flags, void* A, void* B, void* O, void* workspace,
                size_t workspace_bytes, hipStream_t stream) {
    return ffn_fwd_impl("moe_ffn_fwd", false, x, w1, w3, w2, offsets, expert_token_indices,
                        nullptr, nullptr, T, d, f, E, k, flags, A, B, O, workspace,
                        workspace_bytes, stream);
}

int moe_ffn_recompute(const void* x, const void* w1, const void* w3,
                      const int32_t* offsets, const int32_t* expert_token_indices, int64_t T,
                      int d, int f, int E, int k, unsigned flags, void* A, void* B,
                      hipStream_t stream) {
    const char* fn = "moe_ffn_recompute";
    int r;
    if ((r = check_common(fn, T, E, k, flags)) || (r = check_dim(fn, "d", d)) ||
        (r = check_dim(fn, "f", f)))
        return r;
    if (flags & (MOE_RENORM | MOE_ACCUMULATE | MOE_ACCUMULATE_DW | MOE_ATOMIC_COMBINE))
        return fail(MOE_ERR_INVALID_ARG, "%s: only MOE_F32 / MOE_BF16, an activation flag and MOE_H_ON_LOAD are valid", fn);
    const int act = act_of(flags);
    if (act < 0) return fail(MOE_ERR_INVALID_ARG, "%s: MOE_ACT_SILU and MOE_ACT_RELU both set", fn);
    if (T == 0) return MOE_OK;
    REQUIRE_PTR(x); REQUIRE_PTR(w1); REQUIRE_PTR(offsets); REQUIRE_PTR(expert_token_indices);
    REQUIRE_PTR(A);
    if (act == 0) { REQUIRE_PTR(w3); REQUIRE_PTR(B); }
    else { OPT_PTR(w3); OPT_PTR(B); }
    moe::FfnArgs a{};
    a.x = x; a.w1 = w1; a.w3 = w3; a.offsets = offsets; a.eti = expert_token_indices;
    a.A = A; a.B = B; a.T = T; a.d = d; a.f = f; a.E = E; a.k = k; a.act = act;
    moe::probe::begin(stream);
    return hip_status(fn, moe::ffn_first(a, flags & MOE_F32, stream));
}

size_t moe_ffn_fwd_combine_workspace_size(int64_t T, int d, int f, int E, int k, unsigned flags) {
    if (T <= 0 || d < 1 || f < 1 || E < 1 || k < 1) return 0;
    return moe::ffn_fwd_workspace(T, d, f, E, k, flags & MOE_F32, true, flags & MOE_H_ON_LOAD,
                                  flags & MOE_ATOMIC_COMBINE);
}

int moe_ffn_fwd_combine(const void* x, const void* w1, const void* w3, const void* w2,
                        const int32_t* offsets, const int32_t* expert_token_indices,
                        const float* gates, const int32_t* token_index_map, int64_t T, int d,
                        int f, int E, int k, unsigned flags, void* A, void* B, void* y,
                        void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return ffn_fwd_impl("moe_ffn_fwd_combine", true, x, w1, w3, w2, offsets,
                        expert_token_indices, gates, token_index_map, T, d, f, E, k, flags, A, B,
                        y, workspace, workspace_bytes, stream);
}

int moe_combine(const void* src, const float* weights, const int32_t* token_index_map,
                int64_t T, int d, int k, unsigned flags, void* out, hipStream_t stream) {
    const char* fn = "moe_combine";
    int r;
    if ((r = check_common(fn, T, k, k, flags)) || (r = check_dim(fn, "d", d))) return r;
    if (flags & FFN_ONLY) return fail(MOE_ERR_INVALID_ARG, "%s: activation, h-on-load and weight-gradient accumulation flags apply to the FFN calls only", fn);
    if (flags & MOE_RENORM) return fail(MOE_ERR_INVALID_ARG, "%s: MOE_RENORM not valid here", fn);
    if (T == 0) return MOE_OK;
    REQUIRE_PTR(src); OPT_PTR(weights); REQUIRE_PTR(token_index_map); REQUIRE_PTR(out);
    moe::probe::begin(stream);
    return hip_status(fn, moe::combine(src, weights, token_index_map, T, d, k, flags & MOE_F32,
                                       flags & MOE_ACCUMULATE, out, stream));
}


size_t moe_ffn_bwd_workspace_size(int64_t T, int d, int f, int E, int k, unsigned flags) {
    if (T <= 0 || d < 1 || f < 1 || E < 1 || k < 1) return 0;
    return moe::ffn_bwd_workspace(T, d, f, E, k, flags & MOE_F32, false, flags & MOE_H_ON_LOAD,
                                  false);
}

int moe_ffn_bwd(const void* dy, const void* x, const void* w1, const void* w3, const void* w2,
                const float* gates, const int32_t* offsets, const int32_t* expert_token_indices,
                const int32_t* slot_src, void* A, void* B, int64_t T, int d, int f, int E, int k,
                unsigned flags, float* dw1, float* dw3, float* dw2, float* d_gates,
                void* dX_slot, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return ffn_bwd_impl("moe_ffn_bwd", false, dy, x, w1, w3, w2, gates, offsets,
                        expert_token_indices, slot_src, nullptr, A, B, T, d, f, E, k, flags, dw1,
                        dw3, dw2, d_gates, dX_slot, workspace, workspace_bytes, stream);
}

size_t moe_ffn_bwd_combine_workspace_size(int64_t T, int d, int f, int E, int k, unsigned flags) {
    if (T <= 0 || d < 1 || f < 1 || E < 1 || k < 1) return 0;
    return moe::ffn_bwd_workspace(T, d, f, E, k, flags & MOE_F32, true, flags & MOE_H_ON_LOAD,
                                  flags & MOE_ATOMIC_COMBINE);
}

int moe_ffn_bwd_combine(const void* dy, const void* x, const void* w1, const void* w3,
                        const void* w2, const float* gates, const int32_t* offsets,
                        const int32_t* expert_token_indices, const int32_t* slot_src,
                        const int32_t* token_index_map, void* A, void* B, int64_t T, int d,
                        int f, int E, int k, unsigned flags, float* dw1, float* dw3, float* dw2,
                        float* d_gates, void* dx, void* workspace, size_t workspace_bytes,
                        hipStream_t stream) {
    return ffn_bwd_impl("moe_ffn_bwd_combine", true, dy, x, w1, w3, w2, gates, offsets,
                        expert_token_indices, slot_src, token_index_map, A, B, T, d, f, E, k,
                        flags, dw1, dw3, dw2, d_gates, dx, workspace, workspace_bytes, stream);
}

size_t moe_route_bwd_workspace_size(int64_t T, int d, int E, int k, unsigned flags) {
    if (T <= 0 || d < 1 || E < 1 || k < 1) return 0;
    return moe::route_bwd_workspace(T, d, E, k, flags & MOE_F32);
}

int moe_route_bwd(const float* d_gates, const float* logits, const int32_t* topk_ids,
                  const float* gates, const void* x, const void* w_gate, int64_t T, int d, int E,
                  int k, unsigned flags, float* dw_gate, void* dx, void* workspace,
                  size_t workspace_bytes, hipStream_t stream) {
    const char* fn = "moe_route_bwd";
    int r;
    if ((r = check_common(fn, T, E, k, flags)) || (r = check_dim(fn, "d", d))) return r;
    if (flags & FFN_ONLY) return fail(MOE_ERR_INVALID_ARG, "%s: activation, h-on-load and weight-gradient accumulation flags apply to the FFN calls only", fn);
    if (T == 0) return MOE_OK;
    REQUIRE_PTR(d_gates); REQUIRE_PTR(logits); REQUIRE_PTR(topk_ids); REQUIRE_PTR(gates);
    REQUIRE_PTR(x); REQUIRE_PTR(w_gate); REQUIRE_PTR(dw_gate); REQUIRE_PTR(dx);
    const size_t need = moe::route_bwd_workspace(T, d, E, k, flags & MOE_F32);
    if (!workspace || workspace_bytes < need)
        return fail(MOE_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, workspace_bytes, need);
    REQUIRE_PTR(workspace);
    moe::probe::begin(stream);
    return hip_status(fn, moe::route_bwd(d_gates, logits, topk_ids, gates, x, w_gate, T, d, E, k,
                                         flags & MOE_F32, flags & MOE_RENORM,
                                         flags & MOE_ACCUMULATE, dw_gate, dx, workspace, stream));
}

}  // extern "C"
