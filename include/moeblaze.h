/*
 * moeblaze.h -- C ABI of the MI355X (gfx950) MoEBlaze MoE-layer library.
 *
 * One MoE block, forward and backward, on one GPU, as described in the
 * MoEBlaze paper (arXiv 2601.05296): top-k softmax gating (Section 2.1),
 * buffer-free dispatch through index maps (Sections 3.1 and 4), SwiGLU expert
 * FFNs computed as grouped GEMMs that gather token rows on load, with SiLU
 * recomputed instead of stored (Section 5, Algorithm 1), and the gate-weighted
 * combine (Section 2.3).
 *
 * Conventions shared by every call:
 *  - All tensor arguments are DEVICE pointers owned by the caller. The library
 *    never allocates or frees device memory and never synchronises with the
 *    host: each call validates its arguments, enqueues kernels on `stream`
 *    and returns. Results are ready when the stream reaches that point.
 *  - Validation happens before any launch. On a non-zero return nothing has
 *    been enqueued and no output has been written (except MOE_ERR_HIP, which
 *    reports a failed launch).
 *  - Layouts are row-major and dense. Row-vector convention: x[1,d] W[d,f].
 *      x        [T, d]         token activations
 *      w_gate   [E, d]         router weights
 *      w1, w3   [E, d, f]      expert first layer: SiLU branch, linear branch
 *      w2       [E, f, d]      expert down projection
 *    Element type of x, w_gate, w1, w3, w2, dy, A, B, O, dX_slot and the
 *    y / dx outputs: bfloat16 (MOE_BF16, the default) or float32 (MOE_F32,
 *    a debug mode). Gates, logits, gate gradients and weight gradients are
 *    float32 in both modes; index arrays are int32.
 *  - A slot is one (token, chosen expert) pair; there are S = T*k slots,
 *    grouped by expert and, inside an expert, by ascending token id.
 *  - Limits: 1 <= k <= min(E, 16), 1 <= E <= 256, d and f multiples of 64,
 *    T*k < 2^31. T == 0 is a no-op returning MOE_OK. All pointers must be
 *    16-byte aligned.
 *  - Calls that share output or workspace buffers must be ordered on one
 *    stream; concurrent calls on different streams must use disjoint buffers.
 */
#ifndef MOEBLAZE_H
#define MOEBLAZE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define MOE_OK               0
#define MOE_ERR_INVALID_ARG  (-1)  /* null pointer, bad size, k > E, ... */
#define MOE_ERR_UNSUPPORTED  (-2)  /* valid but outside the limits above */
#define MOE_ERR_WORKSPACE    (-3)  /* workspace null or smaller than queried */
#define MOE_ERR_HIP          (-4)  /* a kernel launch failed */

/* flags (bitwise or) */
#define MOE_BF16        0u   /* bfloat16 activations and weights (default) */
#define MOE_F32         1u   /* float32 activations and weights (debug mode) */
#define MOE_RENORM      2u   /* moe_route / moe_route_bwd: renormalise the k gates */
#define MOE_ACCUMULATE  4u   /* moe_combine / moe_route_bwd: add into the output */
/* moe_ffn_fwd / moe_ffn_bwd: expert activation. Default (neither flag): the
 * gated SwiGLU expert of Section 5.1. MOE_ACT_SILU / MOE_ACT_RELU select the
 * non-gated expert of Section 2.2, E(x) = w2 act(x w1) (ReLU and SiLU are the
 * activations of the experiments, Section 6): w3, B and dw3 are then unused
 * and may be NULL, A = x w1 is the only saved activation and act is
 * recomputed from it in the backward. ReLU'(0) is taken as 0. At most one of
 * the two may be set (else MOE_ERR_INVALID_ARG). */
#define MOE_ACT_SILU    8u
#define MOE_ACT_RELU    16u
/* The FFN calls and their workspace queries: buffer no h = SiLU(A) * B.
 * Forward: the second GEMM forms h again from A and B as it loads them
 * (Section 3.1 keeps only the first MLP's output; Section 5.2 recomputes the
 * activation). Backward: the dW2 GEMM runs first and forms g*h from A, B and
 * the gates as it loads them, before dA and dB overwrite A and B. Every result
 * is bit-identical to the default path; the forward workspace drops S*f*2
 * bytes (h; the combined call's strip is rounded to the 512-column tiles of
 * the GEMM that forms h) and the backward's the same (g*h), at the cost of
 * those two GEMMs reading A and B instead of one buffer. moe_ffn_recompute accepts and ignores
 * it; route, build, combine and route_bwd reject it (MOE_ERR_INVALID_ARG). */
#define MOE_H_ON_LOAD   32u
/* moe_ffn_bwd / moe_ffn_bwd_combine: add the weight gradients into dw1, dw3
 * and dw2 instead of overwriting them (the gradient of a layer whose tokens
 * are processed in several chunks is the sum of the chunks' gradients). Every
 * other call rejects it (MOE_ERR_INVALID_ARG). */
#define MOE_ACCUMULATE_DW 64u
/* moe_ffn_fwd_combine / moe_ffn_bwd_combine and their workspace queries: the
 * combine is folded into the epilogue of the GEMM that produces the slot rows
 * (Section 3.1: the expert outputs are reduced as they are produced). Each
 * slot row, times its gate in the forward, is rounded to bfloat16 and added
 * into its token's row of y (dx) by packed-bf16 atomic adds, so no [T*k, d]
 * output nor any strip of it is held: the forward workspace drops the strip
 * and holds T*k float32 slot gates instead, the backward's drops the strip.
 * y (dx, unless MOE_ACCUMULATE) is cleared first. Each atomic add rounds to
 * bfloat16, so a token's k terms are rounded k times, not once (the error
 * grows with k: about 3x the ordered combine's at k = 15), and for k > 2
 * (or with MOE_ACCUMULATE) the result depends on the order in which tiles
 * finish: it is not deterministic bit for bit. With k <= 2 and no
 * MOE_ACCUMULATE it is (bfloat16 addition of two terms onto zero does not
 * depend on their order). bfloat16 only: with MOE_F32, MOE_ERR_UNSUPPORTED.
 * Every other call rejects it (MOE_ERR_INVALID_ARG). */
#define MOE_ATOMIC_COMBINE 128u

/* Human-readable name of a status code (static storage). */
const char* moe_strerror(int status);

/* Detail of the last non-OK status returned on the calling thread. */
const char* moe_last_error(void);

/*
 * moe_route -- top-k softmax gating (Section 2.1: TopK(softmax(W_g x))).
 *   logits[t,e] = x[t] . w_gate[e] (+ bias[e]),  p = softmax over e,
 *   topk_ids[t, 0..k-1] = the k experts with the largest logits, in
 *   decreasing order (equal logits: lower id first),
 *   gates[t,j] = p[t, topk_ids[t,j]]  (MOE_RENORM: divided by the sum of the
 *   k selected probabilities).
 * In:  x [T,d], w_gate [E,d] (element type per flags), bias [E] float32 or
 *      NULL (added before the softmax; -INFINITY excludes an expert).
 * Out: topk_ids [T,k] int32, gates [T,k] float32, logits [T,E] float32
 *      (may be NULL; moe_route_bwd needs it).
 * Logits accumulate in float32; selection is made on the float32 logits.
 */
int moe_route(const void* x, const void* w_gate, const float* bias,
              int64_t T, int d, int E, int k, unsigned flags,
              int32_t* topk_ids, float* gates, float* logits, hipStream_t stream);

/*
 * moe_build_index -- dispatch index maps (Section 4.1 definitions, built
 * without global atomics as in Section 4.2: per-tile expert counts, one
 * prefix sum, then a stable in-tile rank and scatter).
 * In:  topk_ids [T,k] int32, each row k distinct ids in [0,E), as moe_route
 *      writes them.
 * Out: counts [E]                        tokens routed to each expert
 *      offsets [E+1]                     exclusive prefix sum of counts
 *                                        (expert_token_offsets)
 *      expert_token_indices [T*k]        token ids grouped by expert,
 *                                        ascending inside an expert
 *      token_index_map [T,k]             slot of (t,j):
 *                                        expert_token_indices[token_index_map[t,j]] == t
 *      slot_src [T*k]                    t*k + j of each slot (inverse map)
 * workspace: moe_build_index_workspace_size(T,E,k) bytes of device memory.
 * Deterministic: identical inputs give bit-identical outputs.
 * Other ids are rejected on the device, not reported: a choice whose id is
 * outside [0,E) or repeats an earlier id of its row gets no slot and a
 * token_index_map entry of -1, and counts / offsets leave it out, so that
 * offsets[E] < T*k. The maps stay consistent (slots [0, offsets[E]) each
 * written once), and every later call stays inside its buffers: moe_combine
 * adds nothing for a -1 entry, the FFN calls write only slot rows below
 * offsets[E] and no d_gates entry of a rejected choice, and moe_route_bwd
 * ignores ids outside [0,E). The router gradients of a token with a rejected
 * choice are then unspecified.
 */
size_t moe_build_index_workspace_size(int64_t T, int E, int k);
int moe_build_index(const int32_t* topk_ids, int64_t T, int E, int k,
                    int32_t* counts, int32_t* offsets, int32_t* expert_token_indices,
                    int32_t* token_index_map, int32_t* slot_src,
                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * moe_build_index_noalloc -- moe_build_index for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation): the same kernels and outputs, with the per-tile
 * counts in a static 1 MiB device array of the library instead of a caller
 * workspace. No memory is allocated or freed. Arguments, outputs and errors
 * as moe_build_index, plus MOE_ERR_UNSUPPORTED if the counts would not fit
 * the array (never within the limits above: E <= 256 and at most 1024 tiles)
 * and MOE_ERR_HIP if the array's device address cannot be found. Every call
 * on one GPU uses that GPU's single array: calls that overlap on one GPU (on
 * different streams, or from different host threads) race and must not be
 * made.
 */
int moe_build_index_noalloc(const int32_t* topk_ids, int64_t T, int E, int k,
                            int32_t* counts, int32_t* offsets, int32_t* expert_token_indices,
                            int32_t* token_index_map, int32_t* slot_src, hipStream_t stream);

/*
 * moe_ffn_fwd -- expert forward without a routed-token buffer (Section 3.1,
 * Algorithm 1 forward). For each slot s of expert e with token
 * t = expert_token_indices[s] (x rows are gathered while loading):
 *   A[s] = x[t] w1[e],   B[s] = x[t] w3[e]           (saved for backward)
 *   h[s] = SiLU(A[s]) * B[s]                         (formed in the epilogue of
 *                                                     the first GEMM from the
 *                                                     stored A, B; transient)
 *   O[s] = h[s] w2[e]
 * In:  x, w1, w3, w2, offsets [E+1], expert_token_indices [T*k] (from
 *      moe_build_index).
 * Out: A, B [T*k, f], O [T*k, d] (element type per flags).
 * Non-gated (MOE_ACT_SILU / MOE_ACT_RELU): A[s] = x[t] w1[e], h[s] = act(A[s]),
 *      O[s] = h[s] w2[e]; w3 and B are not touched.
 * workspace: moe_ffn_fwd_workspace_size(T,d,f,E,k,flags) bytes (holds h
 *      between the two GEMMs; 0 in MOE_F32 mode, where NULL is accepted).
 */
size_t moe_ffn_fwd_workspace_size(int64_t T, int d, int f, int E, int k, unsigned flags);
int moe_ffn_fwd(const void* x, const void* w1, const void* w3, const void* w2,
                const int32_t* offsets, const int32_t* expert_token_indices,
                int64_t T, int d, int f, int E, int k, unsigned flags,
                void* A, void* B, void* O, void* workspace, size_t workspace_bytes,
                hipStream_t stream);

/*
 * moe_combine -- gate-weighted aggregation (Section 2.3) through the
 * per-token slot list (Section 3.1), and, with weights == NULL, the token
 * gradient accumulation of the backward pass (Section 3.2, step 3):
 *   out[t] = sum_{j<k} weights[t,j] * src[token_index_map[t,j]]
 * The k terms are added in order j = 0..k-1 in float32; a token_index_map
 * entry of -1 (a choice moe_build_index rejected) adds nothing.
 * MOE_ACCUMULATE: out[t] += (the sum) instead of overwriting.
 * In:  src [T*k, d], weights [T,k] float32 or NULL (all ones),
 *      token_index_map [T,k].
 * Out: out [T, d] (element type per flags).
 */
int moe_combine(const void* src, const float* weights, const int32_t* token_index_map,
                int64_t T, int d, int k, unsigned flags, void* out, hipStream_t stream);

/*
 * moe_ffn_bwd -- expert backward (Section 3.2, Algorithm 1 backward).
 * Per slot s of expert e, token t, gate g = gates[slot_src[s]]; dY rows are
 * gathered on load (the expert-summation backward never materialises g*dY:
 * g is applied in the epilogue of u and carried in g*h); h = SiLU(A) * B is
 * recomputed from the saved A, B in the epilogue of the u GEMM:
 *   dw2[e]         = sum_s h[s]^T (g dY[t])
 *   u              = dY[t] w2[e]^T
 *   d_gates[t,j]   = sum_f u * h           (= <dY[t], O[s]>)
 *   dA = g u * B * SiLU'(A),   dB = g u * SiLU(A)      (written over A, B)
 *   dw1[e] = sum_s x[t]^T dA[s],   dw3[e] = sum_s x[t]^T dB[s]
 *   dX_slot[s] = dA[s] w1[e]^T + dB[s] w3[e]^T
 * The token gradient is then moe_combine(dX_slot, NULL, token_index_map).
 * In:  dy [T,d], x, w1, w3, w2, gates [T,k], offsets, expert_token_indices,
 *      slot_src; A, B [T*k,f] as written by moe_ffn_fwd.
 * Non-gated (MOE_ACT_SILU / MOE_ACT_RELU): h = act(A), dA = g u act'(A)
 *      (written over A), dw1 and dX_slot from dA alone; w3, B, dw3 unused.
 * Out: A, B overwritten with dA, dB; dw1, dw3 [E,d,f], dw2 [E,f,d] float32
 *      (overwritten, zero for experts with no tokens; with MOE_ACCUMULATE_DW
 *      added to); d_gates [T,k] float32; dX_slot [T*k, d].
 * workspace: moe_ffn_bwd_workspace_size(T,d,f,E,k,flags) bytes (gate-gradient
 *      partial sums, g*h for the dw2 GEMM, and the experts ordered by token
 *      count, which the weight-gradient GEMMs take longest first; 0 in
 *      MOE_F32 mode).
 */
size_t moe_ffn_bwd_workspace_size(int64_t T, int d, int f, int E, int k, unsigned flags);
int moe_ffn_bwd(const void* dy, const void* x, const void* w1, const void* w3, const void* w2,
                const float* gates, const int32_t* offsets,
                const int32_t* expert_token_indices, const int32_t* slot_src,
                void* A, void* B, int64_t T, int d, int f, int E, int k, unsigned flags,
                float* dw1, float* dw3, float* dw2, float* d_gates, void* dX_slot,
                void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * moe_ffn_recompute -- the first-layer outputs alone: A[s] = x[t] w1[e] and
 * B[s] = x[t] w3[e] (non-gated: A alone), bit-identical to what moe_ffn_fwd
 * writes. It serves a full-recompute checkpoint policy (Section 5.2 carried
 * one step further): the forward keeps only the routing decision and the
 * dispatch maps, and the backward recomputes A and B with this call before
 * moe_ffn_bwd, for 2*T*k*d*f (non-gated: T*k*d*f) extra multiply-adds.
 * In:  x, w1, w3, offsets, expert_token_indices as moe_ffn_fwd.
 * Out: A, B [T*k, f]. No workspace.
 */
int moe_ffn_recompute(const void* x, const void* w1, const void* w3,
                      const int32_t* offsets, const int32_t* expert_token_indices,
                      int64_t T, int d, int f, int E, int k, unsigned flags,
                      void* A, void* B, hipStream_t stream);

/*
 * moe_ffn_fwd_combine -- moe_ffn_fwd followed by moe_combine(O, gates,
 * token_index_map) without the [T*k, d] expert-output buffer: the second GEMM
 * runs one column strip of O at a time (512 columns) into the workspace and
 * each strip is combined into y before the next one is computed (Section 2.3
 * aggregation, Section 3.1). Same arithmetic and summation order as the two
 * separate calls, so the result is identical and deterministic.
 * MOE_ATOMIC_COMBINE instead folds the combine into the second GEMM's
 * epilogue (no strip; see the flag).
 * In:  as moe_ffn_fwd, plus gates [T,k] float32 and token_index_map [T,k].
 * Out: A, B as moe_ffn_fwd; y [T,d] (element type per flags).
 * workspace: moe_ffn_fwd_combine_workspace_size(T,d,f,E,k,flags) bytes (h and
 *      one [T*k, 512] strip; in MOE_F32 mode the whole [T*k, d] output).
 */
size_t moe_ffn_fwd_combine_workspace_size(int64_t T, int d, int f, int E, int k, unsigned flags);
int moe_ffn_fwd_combine(const void* x, const void* w1, const void* w3, const void* w2,
                        const int32_t* offsets, const int32_t* expert_token_indices,
                        const float* gates, const int32_t* token_index_map,
                        int64_t T, int d, int f, int E, int k, unsigned flags,
                        void* A, void* B, void* y, void* workspace, size_t workspace_bytes,
                        hipStream_t stream);

/*
 * moe_ffn_bwd_combine -- moe_ffn_bwd followed by the token gradient
 * accumulation moe_combine(dX_slot, NULL, token_index_map) of Section 3.2
 * step 3, without the [T*k, d] dX_slot buffer: dX_slot is produced one column
 * strip at a time in the workspace (reusing the space of g*h, which the dw2
 * GEMM has consumed by then) and each strip is summed into dx. Identical to
 * the two separate calls. MOE_ATOMIC_COMBINE instead adds the dX_slot rows
 * into dx from the dX GEMM's epilogue (no strip; see the flag).
 * In:  as moe_ffn_bwd, plus token_index_map [T,k].
 * Out: as moe_ffn_bwd, with dx [T,d] in place of dX_slot; MOE_ACCUMULATE adds
 *      into dx instead of overwriting it.
 * workspace: moe_ffn_bwd_combine_workspace_size(T,d,f,E,k,flags) bytes.
 */
size_t moe_ffn_bwd_combine_workspace_size(int64_t T, int d, int f, int E, int k, unsigned flags);
int moe_ffn_bwd_combine(const void* dy, const void* x, const void* w1, const void* w3,
                        const void* w2, const float* gates, const int32_t* offsets,
                        const int32_t* expert_token_indices, const int32_t* slot_src,
                        const int32_t* token_index_map, void* A, void* B, int64_t T, int d,
                        int f, int E, int k, unsigned flags, float* dw1, float* dw3, float* dw2,
                        float* d_gates, void* dx, void* workspace, size_t workspace_bytes,
                        hipStream_t stream);

/*
 * moe_route_bwd -- router backward. The paper does not state it; this is the
 * closed form of the gating Jacobian for the forward of moe_route:
 *   without MOE_RENORM: dl = p * (dp - <p, dp>), dp[e] = d_gates[t,j] where
 *                       topk_ids[t,j] == e, else 0 (p = softmax(logits));
 *   with MOE_RENORM:    dl[topk_ids[t,j]] = g_j (d_gates[t,j] - sum_j' g_j'
 *                       d_gates[t,j']), zero for unselected experts.
 *   dw_gate = dl^T x   (float32 [E,d], overwritten),
 *   dx      = dl w_gate (written, or added with MOE_ACCUMULATE).
 * The bias receives no gradient.
 * In:  d_gates [T,k], logits [T,E], topk_ids [T,k], gates [T,k] (from
 *      moe_route), x [T,d], w_gate [E,d].
 * workspace: moe_route_bwd_workspace_size(T,d,E,k,flags) bytes.
 */
size_t moe_route_bwd_workspace_size(int64_t T, int d, int E, int k, unsigned flags);
int moe_route_bwd(const float* d_gates, const float* logits, const int32_t* topk_ids,
                  const float* gates, const void* x, const void* w_gate,
                  int64_t T, int d, int E, int k, unsigned flags,
                  float* dw_gate, void* dx, void* workspace, size_t workspace_bytes,
                  hipStream_t stream);

/*
 * Kernel timing probe (diagnostics; not needed for computing anything, and
 * the one part of this library that waits on the host: moe_probe_get
 * synchronises with the event it reads).
 * moe_probe_enable(capacity) creates `capacity` HIP events and starts
 * recording: each entry point then records an event on its stream before its
 * first kernel and one after every kernel it launches. Record i (0-based,
 * counting kernel records only) is the time between the kernel's preceding
 * event and its own, i.e. that kernel's duration on the stream. Once the
 * events run out nothing more is recorded; moe_probe_dropped returns how
 * many records were lost that way since moe_probe_enable (a caller that
 * needs every launch must check it is 0). moe_probe_get waits for record i
 * and returns the kernel's name (static storage) and its duration in ms.
 * moe_probe_disable destroys the events. Not thread-safe; single stream.
 */
int moe_probe_enable(int capacity);
void moe_probe_disable(void);
int moe_probe_count(void);
int moe_probe_dropped(void);
int moe_probe_get(int index, const char** kernel_name, float* ms);

#ifdef __cplusplus
}
#endif
#endif /* MOEBLAZE_H */
