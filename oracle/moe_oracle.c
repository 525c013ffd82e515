/*
 * moe_oracle.c -- plain, slow CPU oracle for one MoEBlaze MoE layer.
 *
 * TEST INFRASTRUCTURE ONLY. This file is compiled into liboracle.so, which
 * only the test suite, the package's smoke check and the CPU-baseline leg of
 * the benchmark load. The product path (the HIP library) never links, loads or
 * calls it, and the two share no source.
 *
 * Everything is computed in double precision with straightforward loops, in
 * the order the paper states the operations. Inputs are double arrays holding
 * exactly the values the device sees (bf16 values widened without change).
 * OpenMP splits only independent output rows (or whole experts for weight
 * gradients), so every sum has one fixed order and results do not depend on
 * the thread count.
 *
 * Notation (row-vector convention, x[1,d] times W[d,f]):
 *   x [T,d], w_gate [E,d], bias [E] (optional), w1, w3 [E,d,f], w2 [E,f,d].
 *   Slot s in [0, T*k) is one (token, expert) assignment; slots are grouped by
 *   expert, ascending token id inside an expert.
 *
 * Readings of the paper used here (each also listed in the design notes):
 *   - Gating (Section 2.1): softmax over all E logits, then the k largest.
 *     Selection is made on the logits (softmax is monotone); the decision is
 *     taken on the logits rounded to float32, the precision the device uses;
 *     equal values go to the lower expert id. Slot j of a token holds its
 *     j-th largest logit.
 *   - Gates (Section 2.3): g[t,j] = p[t, ids[t,j]]; with renorm, divided by
 *     the sum of the token's k selected probabilities.
 *   - SwiGLU (Section 5.1): h = SiLU(x W1) * (x W3), o = h W2, SiLU(u) = u
 *     sigmoid(u). W3 is the linear branch, W2 the down projection.
 *   - Backward (Section 3.2, Algorithm 1): dY is mapped to slots through the
 *     index maps, the expert backward uses the saved first-layer outputs A, B
 *     with SiLU recomputed, and token gradients sum the k slot gradients.
 *   - Router backward: the paper gives none; the closed form of the softmax
 *     (or renormalised softmax) Jacobian is used.
 *   - Non-gated experts (Section 2.2, E_i(x) = W2 act(W1 x); the experiments
 *     of Section 6 use ReLU and SiLU): a = x W1 is the one saved activation,
 *     act is recomputed from it in the backward (the checkpoint of Section
 *     5.2 applied to a single projection). ReLU'(0) is taken as 0.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_API __attribute__((visibility("default")))

#include <omp.h>

/* threads the OpenMP loops of this file run with (for reporting only) */
ORACLE_API int oracle_threads(void) { return omp_get_max_threads(); }

static double sigmoid(double u) { return 1.0 / (1.0 + exp(-u)); }
static double silu(double u) { return u * sigmoid(u); }

/* activation codes of the non-gated experts */
enum { ACT_SILU = 1, ACT_RELU = 2 };
static double act_f(int act, double u) { return act == ACT_RELU ? (u > 0.0 ? u : 0.0) : silu(u); }
static double act_d(int act, double u)
{
    if (act == ACT_RELU) return u > 0.0 ? 1.0 : 0.0;
    const double sg = sigmoid(u);
    return sg * (1.0 + u * (1.0 - sg));
}

/* ---------------------------------------------------------------------------
 * Gating (Section 2.1): logits = x W_g^T (+ bias), p = softmax(logits),
 * topk_experts = TopK(p).  Outputs: ids [T,k], gates [T,k], logits [T,E],
 * probs [T,E] (nullable).
 * ------------------------------------------------------------------------- */
ORACLE_API void oracle_route(const double* x, const double* w_gate, const double* bias,
                             int64_t T, int d, int E, int k, int renorm,
                             int32_t* ids, double* gates, double* logits, double* probs)
{
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        const double* xt = x + t * d;
        double* lt = logits + t * E;
        for (int e = 0; e < E; ++e) {
            double acc = 0.0;
            for (int i = 0; i < d; ++i) acc += xt[i] * w_gate[(int64_t)e * d + i];
            if (bias) acc += bias[e];
            lt[e] = acc;
        }
        /* softmax over all experts, max-subtracted */
        double mx = -INFINITY;
        for (int e = 0; e < E; ++e) if (lt[e] > mx) mx = lt[e];
        double* p = (double*)malloc(sizeof(double) * (size_t)E);
        double z = 0.0;
        for (int e = 0; e < E; ++e) { p[e] = exp(lt[e] - mx); z += p[e]; }
        for (int e = 0; e < E; ++e) p[e] /= z;
        if (probs) memcpy(probs + t * E, p, sizeof(double) * (size_t)E);
        /* top-k by repeated selection of the largest remaining float32 logit */
        unsigned char* taken = (unsigned char*)calloc((size_t)E, 1);
        double gsum = 0.0;
        for (int j = 0; j < k; ++j) {
            int best = -1;
            float bestv = 0.0f;
            for (int e = 0; e < E; ++e) {
                if (taken[e]) continue;
                float v = (float)lt[e];
                if (best < 0 || v > bestv) { best = e; bestv = v; }
            }
            taken[best] = 1;
            ids[t * k + j] = best;
            gates[t * k + j] = p[best];
            gsum += p[best];
        }
        if (renorm)
            for (int j = 0; j < k; ++j) gates[t * k + j] /= gsum;
        free(taken);
        free(p);
    }
}

/* ---------------------------------------------------------------------------
 * Dispatch index maps (Section 4.1 definitions):
 *   counts[e]        number of (token, slot) pairs routed to e
 *   offsets[E+1]     exclusive prefix sum of counts
 *   eti[S]           expert_token_indices: token ids grouped by expert,
 *                    ascending token id within an expert (worked example)
 *   tim[T,k]         token_index_map: eti[tim[t,j]] == t
 *   slot_src[S]      t*k + j of the slot, i.e. the inverse of tim
 * Written straight from the definitions: visit experts in order and, for each,
 * tokens in ascending order.
 * ------------------------------------------------------------------------- */
ORACLE_API void oracle_build_index(const int32_t* ids, int64_t T, int E, int k,
                                   int32_t* counts, int32_t* offsets, int32_t* eti,
                                   int32_t* tim, int32_t* slot_src)
{
    for (int e = 0; e < E; ++e) counts[e] = 0;
    for (int64_t t = 0; t < T; ++t)
        for (int j = 0; j < k; ++j) counts[ids[t * k + j]] += 1;
    offsets[0] = 0;
    for (int e = 0; e < E; ++e) offsets[e + 1] = offsets[e] + counts[e];
    #pragma omp parallel for schedule(dynamic, 1)
    for (int e = 0; e < E; ++e) {
        int64_t pos = offsets[e];
        for (int64_t t = 0; t < T; ++t)
            for (int j = 0; j < k; ++j)
                if (ids[t * k + j] == e) {
                    eti[pos] = (int32_t)t;
                    tim[t * k + j] = (int32_t)pos;
                    slot_src[pos] = (int32_t)(t * k + j);
                    ++pos;
                }
    }
}

/* expert owning slot s (offsets is nondecreasing, offsets[E] = S) */
static int expert_of_slot(const int32_t* offsets, int E, int64_t s)
{
    int e = 0;
    while (e < E - 1 && s >= offsets[e + 1]) ++e;
    return e;
}

/* ---------------------------------------------------------------------------
 * Expert forward (Section 3.1 and Algorithm 1, forward procedure): for every
 * slot s of expert e with token t = eti[s], gathered straight from x:
 *   A[s] = x[t] W1[e],  B[s] = x[t] W3[e],  h = SiLU(A) * B,  O[s] = h W2[e].
 * A and B are the saved activations; O is the per-slot expert output.
 * ------------------------------------------------------------------------- */
ORACLE_API void oracle_ffn_fwd(const double* x, const double* w1, const double* w3,
                               const double* w2, const int32_t* offsets, const int32_t* eti,
                               int64_t T, int d, int f, int E, int k,
                               double* A, double* B, double* O)
{
    const int64_t S = T * k;
    #pragma omp parallel for schedule(static)
    for (int64_t s = 0; s < S; ++s) {
        const int e = expert_of_slot(offsets, E, s);
        const double* xt = x + (int64_t)eti[s] * d;
        const double* W1 = w1 + (int64_t)e * d * f;
        const double* W3 = w3 + (int64_t)e * d * f;
        const double* W2 = w2 + (int64_t)e * f * d;
        double* a = A + s * f;
        double* b = B + s * f;
        double* o = O + s * d;
        for (int n = 0; n < f; ++n) { a[n] = 0.0; b[n] = 0.0; }
        for (int i = 0; i < d; ++i) {
            const double xi = xt[i];
            for (int n = 0; n < f; ++n) {
                a[n] += xi * W1[(int64_t)i * f + n];
                b[n] += xi * W3[(int64_t)i * f + n];
            }
        }
        for (int n = 0; n < d; ++n) o[n] = 0.0;
        for (int c = 0; c < f; ++c) {
            const double h = silu(a[c]) * b[c];
            for (int n = 0; n < d; ++n) o[n] += h * W2[(int64_t)c * d + n];
        }
    }
}

/* ---------------------------------------------------------------------------
 * Output aggregation (Section 2.3), driven by token_index_map (Section 3.1):
 *   out[t] = sum_j w[t,j] * src[tim[t,j]]   (w == NULL means all ones).
 * With w == NULL this is also the token gradient accumulation of Section 3.2
 * step 3 (sum of the k slot gradients of a token).
 * ------------------------------------------------------------------------- */
ORACLE_API void oracle_combine(const double* src, const double* w, const int32_t* tim,
                               int64_t T, int d, int k, double* out)
{
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        double* yt = out + t * d;
        for (int n = 0; n < d; ++n) yt[n] = 0.0;
        for (int j = 0; j < k; ++j) {
            const double g = w ? w[t * k + j] : 1.0;
            const double* o = src + (int64_t)tim[t * k + j] * d;
            for (int n = 0; n < d; ++n) yt[n] += g * o[n];
        }
    }
}

/* ---------------------------------------------------------------------------
 * Expert backward (Section 3.2, Algorithm 1 backward procedure), per slot s
 * of expert e, token t = eti[s], gate g = gates[slot_src[s]]:
 *   expert-summation backward:  dO = g * dY[t]            (never stored)
 *   gate gradient:              d_gates[slot_src[s]] = <dY[t], O[s]>,
 *                               O[s] = h W2[e] recomputed here
 *   final projection:           dW2[e] += h^T dO,   dh = dO W2[e]^T
 *   recompute SiLU(A) and       dA = dh * B * SiLU'(A),   dB = dh * SiLU(A)
 *   first layer:                dW1[e] += x[t]^T dA,  dW3[e] += x[t]^T dB
 *                               dX_slot[s] = dA W1[e]^T + dB W3[e]^T
 * SiLU'(u) = sigmoid(u) * (1 + u * (1 - sigmoid(u))).
 * Weight gradients are summed over the expert's slots in slot order.
 * ------------------------------------------------------------------------- */
ORACLE_API void oracle_ffn_bwd(const double* dy, const double* x, const double* w1,
                               const double* w3, const double* w2, const double* gates,
                               const int32_t* offsets, const int32_t* eti,
                               const int32_t* slot_src, const double* A, const double* B,
                               int64_t T, int d, int f, int E, int k,
                               double* dA, double* dB, double* dw1, double* dw3,
                               double* dw2, double* d_gates, double* dX_slot)
{
    const int64_t S = T * k;
    /* per-slot quantities */
    #pragma omp parallel for schedule(static)
    for (int64_t s = 0; s < S; ++s) {
        const int e = expert_of_slot(offsets, E, s);
        const int64_t t = eti[s];
        const double g = gates[slot_src[s]];
        const double* W1 = w1 + (int64_t)e * d * f;
        const double* W3 = w3 + (int64_t)e * d * f;
        const double* W2 = w2 + (int64_t)e * f * d;
        const double* a = A + s * f;
        const double* b = B + s * f;
        const double* dyt = dy + t * d;
        /* gate gradient from the recomputed expert output O[s] = h W2[e] */
        double* o = (double*)calloc((size_t)d, sizeof(double));
        for (int c = 0; c < f; ++c) {
            const double h = silu(a[c]) * b[c];
            for (int n = 0; n < d; ++n) o[n] += h * W2[(int64_t)c * d + n];
        }
        double dg = 0.0;
        for (int n = 0; n < d; ++n) dg += dyt[n] * o[n];
        free(o);
        d_gates[slot_src[s]] = dg;
        /* dh = (g dY[t]) W2^T, then the SwiGLU derivative */
        for (int c = 0; c < f; ++c) {
            double dh = 0.0;
            for (int n = 0; n < d; ++n) dh += g * dyt[n] * W2[(int64_t)c * d + n];
            const double sg = sigmoid(a[c]);
            dA[s * f + c] = dh * b[c] * sg * (1.0 + a[c] * (1.0 - sg));
            dB[s * f + c] = dh * a[c] * sg;
        }
        /* slot input gradient */
        double* dxs = dX_slot + s * d;
        for (int i = 0; i < d; ++i) {
            double acc = 0.0;
            for (int c = 0; c < f; ++c)
                acc += dA[s * f + c] * W1[(int64_t)i * f + c] + dB[s * f + c] * W3[(int64_t)i * f + c];
            dxs[i] = acc;
        }
    }
    /* weight gradients: one expert per thread, slots in order */
    #pragma omp parallel for schedule(dynamic, 1)
    for (int e = 0; e < E; ++e) {
        double* DW1 = dw1 + (int64_t)e * d * f;
        double* DW3 = dw3 + (int64_t)e * d * f;
        double* DW2 = dw2 + (int64_t)e * f * d;
        memset(DW1, 0, sizeof(double) * (size_t)d * f);
        memset(DW3, 0, sizeof(double) * (size_t)d * f);
        memset(DW2, 0, sizeof(double) * (size_t)f * d);
        for (int64_t s = offsets[e]; s < offsets[e + 1]; ++s) {
            const int64_t t = eti[s];
            const double g = gates[slot_src[s]];
            const double* xt = x + t * d;
            const double* dyt = dy + t * d;
            for (int c = 0; c < f; ++c) {
                const double h = silu(A[s * f + c]) * B[s * f + c];
                for (int n = 0; n < d; ++n) DW2[(int64_t)c * d + n] += h * g * dyt[n];
            }
            for (int i = 0; i < d; ++i) {
                const double xi = xt[i];
                for (int c = 0; c < f; ++c) {
                    DW1[(int64_t)i * f + c] += xi * dA[s * f + c];
                    DW3[(int64_t)i * f + c] += xi * dB[s * f + c];
                }
            }
        }
    }
}

/* ---------------------------------------------------------------------------
 * Router backward (not given in the paper; closed form of the gating
 * Jacobian). From the gate gradients d_gates [T,k]:
 *   no renorm: g_j = p[ids_j];  dl = p * (dp - <p, dp>), dp[e] = d_gates[t,j]
 *              where ids[t,j] == e, else 0.
 *   renorm:    g = softmax of the selected logits; dl[ids_j] = g_j (dg_j -
 *              sum_j' g_j' dg_j'), zero for unselected experts.
 *   dW_g = dl^T x,   dx_router[t] = dl[t] W_g.   The bias gets no gradient.
 * p and g are recomputed from the saved logits.
 * ------------------------------------------------------------------------- */
ORACLE_API void oracle_route_bwd(const double* d_gates, const double* logits,
                                 const int32_t* ids, const double* x, const double* w_gate,
                                 int64_t T, int d, int E, int k, int renorm,
                                 double* dlogits, double* dw_gate, double* dx_router)
{
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        const double* lt = logits + t * E;
        double* dl = dlogits + t * E;
        double mx = -INFINITY;
        for (int e = 0; e < E; ++e) if (lt[e] > mx) mx = lt[e];
        double* p = (double*)malloc(sizeof(double) * (size_t)E);
        double z = 0.0;
        for (int e = 0; e < E; ++e) { p[e] = exp(lt[e] - mx); z += p[e]; }
        for (int e = 0; e < E; ++e) p[e] /= z;
        for (int e = 0; e < E; ++e) dl[e] = 0.0;
        if (!renorm) {
            double pdp = 0.0;
            for (int j = 0; j < k; ++j) pdp += p[ids[t * k + j]] * d_gates[t * k + j];
            for (int e = 0; e < E; ++e) {
                double dp = 0.0;
                for (int j = 0; j < k; ++j) if (ids[t * k + j] == e) dp = d_gates[t * k + j];
                dl[e] = p[e] * (dp - pdp);
            }
        } else {
            double psel = 0.0;
            for (int j = 0; j < k; ++j) psel += p[ids[t * k + j]];
            double gdg = 0.0;
            for (int j = 0; j < k; ++j) gdg += (p[ids[t * k + j]] / psel) * d_gates[t * k + j];
            for (int j = 0; j < k; ++j) {
                const double gj = p[ids[t * k + j]] / psel;
                dl[ids[t * k + j]] = gj * (d_gates[t * k + j] - gdg);
            }
        }
        free(p);
        double* dxt = dx_router + t * d;
        for (int i = 0; i < d; ++i) dxt[i] = 0.0;
        for (int e = 0; e < E; ++e) {
            const double c = dl[e];
            for (int i = 0; i < d; ++i) dxt[i] += c * w_gate[(int64_t)e * d + i];
        }
    }
    #pragma omp parallel for schedule(static)
    for (int e = 0; e < E; ++e) {
        double* dw = dw_gate + (int64_t)e * d;
        for (int i = 0; i < d; ++i) dw[i] = 0.0;
        for (int64_t t = 0; t < T; ++t) {
            const double c = dlogits[t * E + e];
            for (int i = 0; i < d; ++i) dw[i] += c * x[t * d + i];
        }
    }
}

/* ---------------------------------------------------------------------------
 * Non-gated expert forward (Section 2.2): per slot s of expert e, token
 * t = eti[s]:  a = x[t] W1[e],  h = act(a),  o = h W2[e].
 * Outputs A [S,f] (the saved pre-activation) and O [S,d].
 * ------------------------------------------------------------------------- */
ORACLE_API void oracle_ffn_fwd_act(const double* x, const double* w1, const double* w2,
                                   const int32_t* offsets, const int32_t* eti, int64_t T,
                                   int d, int f, int E, int k, int act, double* A, double* O)
{
    const int64_t S = T * k;
    #pragma omp parallel for schedule(static)
    for (int64_t s = 0; s < S; ++s) {
        const int e = expert_of_slot(offsets, E, s);
        const double* xt = x + (int64_t)eti[s] * d;
        const double* W1 = w1 + (int64_t)e * d * f;
        const double* W2 = w2 + (int64_t)e * f * d;
        double* a = A + s * f;
        double* o = O + s * d;
        for (int n = 0; n < f; ++n) a[n] = 0.0;
        for (int i = 0; i < d; ++i) {
            const double xi = xt[i];
            for (int n = 0; n < f; ++n) a[n] += xi * W1[(int64_t)i * f + n];
        }
        for (int n = 0; n < d; ++n) o[n] = 0.0;
        for (int c = 0; c < f; ++c) {
            const double h = act_f(act, a[c]);
            for (int n = 0; n < d; ++n) o[n] += h * W2[(int64_t)c * d + n];
        }
    }
}

/* ---------------------------------------------------------------------------
 * Non-gated expert backward (Section 3.2 with the expert of Section 2.2), per
 * slot s of expert e, token t, gate g = gates[slot_src[s]]:
 *   d_gates[slot_src[s]] = <dY[t], O[s]>,  O[s] = act(A[s]) W2[e] recomputed
 *   dh = (g dY[t]) W2[e]^T,   dA = dh * act'(A)
 *   dW2[e] += act(A)^T (g dY[t]),   dW1[e] += x[t]^T dA,   dX_slot[s] = dA W1[e]^T
 * Weight gradients are summed over the expert's slots in slot order.
 * ------------------------------------------------------------------------- */
ORACLE_API void oracle_ffn_bwd_act(const double* dy, const double* x, const double* w1,
                                   const double* w2, const double* gates,
                                   const int32_t* offsets, const int32_t* eti,
                                   const int32_t* slot_src, const double* A, int64_t T, int d,
                                   int f, int E, int k, int act, double* dA, double* dw1,
                                   double* dw2, double* d_gates, double* dX_slot)
{
    const int64_t S = T * k;
    #pragma omp parallel for schedule(static)
    for (int64_t s = 0; s < S; ++s) {
        const int e = expert_of_slot(offsets, E, s);
        const int64_t t = eti[s];
        const double g = gates[slot_src[s]];
        const double* W1 = w1 + (int64_t)e * d * f;
        const double* W2 = w2 + (int64_t)e * f * d;
        const double* a = A + s * f;
        const double* dyt = dy + t * d;
        double* o = (double*)calloc((size_t)d, sizeof(double));
        for (int c = 0; c < f; ++c) {
            const double h = act_f(act, a[c]);
            for (int n = 0; n < d; ++n) o[n] += h * W2[(int64_t)c * d + n];
        }
        double dg = 0.0;
        for (int n = 0; n < d; ++n) dg += dyt[n] * o[n];
        free(o);
        d_gates[slot_src[s]] = dg;
        for (int c = 0; c < f; ++c) {
            double dh = 0.0;
            for (int n = 0; n < d; ++n) dh += g * dyt[n] * W2[(int64_t)c * d + n];
            dA[s * f + c] = dh * act_d(act, a[c]);
        }
        double* dxs = dX_slot + s * d;
        for (int i = 0; i < d; ++i) {
            double acc = 0.0;
            for (int c = 0; c < f; ++c) acc += dA[s * f + c] * W1[(int64_t)i * f + c];
            dxs[i] = acc;
        }
    }
    #pragma omp parallel for schedule(dynamic, 1)
    for (int e = 0; e < E; ++e) {
        double* DW1 = dw1 + (int64_t)e * d * f;
        double* DW2 = dw2 + (int64_t)e * f * d;
        memset(DW1, 0, sizeof(double) * (size_t)d * f);
        memset(DW2, 0, sizeof(double) * (size_t)f * d);
        for (int64_t s = offsets[e]; s < offsets[e + 1]; ++s) {
            const int64_t t = eti[s];
            const double g = gates[slot_src[s]];
            const double* xt = x + t * d;
            const double* dyt = dy + t * d;
            for (int c = 0; c < f; ++c) {
                const double h = act_f(act, A[s * f + c]);
                for (int n = 0; n < d; ++n) DW2[(int64_t)c * d + n] += h * g * dyt[n];
            }
            for (int i = 0; i < d; ++i) {
                const double xi = xt[i];
                for (int c = 0; c < f; ++c) DW1[(int64_t)i * f + c] += xi * dA[s * f + c];
            }
        }
    }
}
