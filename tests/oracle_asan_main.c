/* Drives every function of oracle/moe_oracle.c once on small seeded inputs
 * (one full layer forward and backward, gated and non-gated, including an
 * expert that receives no token and a single-token case), so that a build
 * with AddressSanitizer and UndefinedBehaviorSanitizer checks the oracle's
 * memory accesses and integer arithmetic. Built and run by
 * tests/test_oracle_asan.py; prints "ok" and exits 0 when every call
 * returned. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void oracle_route(const double*, const double*, const double*, int64_t, int, int, int, int,
                  int32_t*, double*, double*, double*);
void oracle_build_index(const int32_t*, int64_t, int, int, int32_t*, int32_t*, int32_t*,
                        int32_t*, int32_t*);
void oracle_ffn_fwd(const double*, const double*, const double*, const double*, const int32_t*,
                    const int32_t*, int64_t, int, int, int, int, double*, double*, double*);
void oracle_combine(const double*, const double*, const int32_t*, int64_t, int, int, double*);
void oracle_ffn_bwd(const double*, const double*, const double*, const double*, const double*,
                    const double*, const int32_t*, const int32_t*, const int32_t*,
                    const double*, const double*, int64_t, int, int, int, int, double*, double*,
                    double*, double*, double*, double*, double*);
void oracle_route_bwd(const double*, const double*, const int32_t*, const double*,
                      const double*, int64_t, int, int, int, int, double*, double*, double*);
void oracle_ffn_fwd_act(const double*, const double*, const double*, const int32_t*,
                        const int32_t*, int64_t, int, int, int, int, int, double*, double*);
void oracle_ffn_bwd_act(const double*, const double*, const double*, const double*,
                        const double*, const int32_t*, const int32_t*, const int32_t*,
                        const double*, int64_t, int, int, int, int, int, double*, double*,
                        double*, double*, double*);

static uint64_t rng = 88172645463325252ull;
static double urand(void) {   /* xorshift64, uniform in [-1, 1) */
    rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
    return (double)(rng >> 11) / (double)(1ull << 52) - 1.0;
}
static double* vec(size_t n, double scale) {
    double* p = malloc(n * sizeof(double));
    if (!p) { fprintf(stderr, "out of memory\n"); exit(2); }
    for (size_t i = 0; i < n; ++i) p[i] = scale * urand();
    return p;
}
static void* zalloc(size_t n, size_t sz) {
    void* p = calloc(n ? n : 1, sz);
    if (!p) { fprintf(stderr, "out of memory\n"); exit(2); }
    return p;
}

static void layer(int64_t T, int d, int f, int E, int k, int renorm, int act) {
    const int64_t S = T * k;
    double *x = vec(T * d, 1.0), *wg = vec((size_t)E * d, 0.1), *bias = vec(E, 0.5);
    double *w1 = vec((size_t)E * d * f, 0.1), *w3 = vec((size_t)E * d * f, 0.1);
    double *w2 = vec((size_t)E * f * d, 0.1), *dy = vec(T * d, 1.0);
    bias[E - 1] = -1e30;   /* the last expert receives no token */
    int32_t* ids = zalloc(S, 4);
    double *gates = zalloc(S, 8), *logits = zalloc(T * E, 8), *probs = zalloc(T * E, 8);
    oracle_route(x, wg, bias, T, d, E, k, renorm, ids, gates, logits, probs);
    int32_t *counts = zalloc(E, 4), *offsets = zalloc(E + 1, 4), *eti = zalloc(S, 4);
    int32_t *tim = zalloc(S, 4), *slot_src = zalloc(S, 4);
    oracle_build_index(ids, T, E, k, counts, offsets, eti, tim, slot_src);
    double *A = zalloc(S * f, 8), *B = zalloc(S * f, 8), *O = zalloc(S * d, 8);
    double *y = zalloc(T * d, 8);
    double *dA = zalloc(S * f, 8), *dB = zalloc(S * f, 8), *dX = zalloc(S * d, 8);
    double *dw1 = zalloc((size_t)E * d * f, 8), *dw3 = zalloc((size_t)E * d * f, 8);
    double *dw2 = zalloc((size_t)E * f * d, 8), *dg = zalloc(S, 8), *dx = zalloc(T * d, 8);
    double *dl = zalloc(T * E, 8), *dwg = zalloc((size_t)E * d, 8), *dxr = zalloc(T * d, 8);
    if (act == 0) {
        oracle_ffn_fwd(x, w1, w3, w2, offsets, eti, T, d, f, E, k, A, B, O);
        oracle_combine(O, gates, tim, T, d, k, y);
        oracle_ffn_bwd(dy, x, w1, w3, w2, gates, offsets, eti, slot_src, A, B, T, d, f, E, k,
                       dA, dB, dw1, dw3, dw2, dg, dX);
    } else {
        oracle_ffn_fwd_act(x, w1, w2, offsets, eti, T, d, f, E, k, act, A, O);
        oracle_combine(O, gates, tim, T, d, k, y);
        oracle_ffn_bwd_act(dy, x, w1, w2, gates, offsets, eti, slot_src, A, T, d, f, E, k, act,
                           dA, dw1, dw2, dg, dX);
    }
    oracle_combine(dX, NULL, tim, T, d, k, dx);
    oracle_route_bwd(dg, logits, ids, x, wg, T, d, E, k, renorm, dl, dwg, dxr);
    void* all[] = {x, wg, bias, w1, w3, w2, dy, ids, gates, logits, probs, counts, offsets, eti,
                   tim, slot_src, A, B, O, y, dA, dB, dX, dw1, dw3, dw2, dg, dx, dl, dwg, dxr};
    for (size_t i = 0; i < sizeof(all) / sizeof(all[0]); ++i) free(all[i]);
}

int main(void) {
    layer(37, 16, 24, 5, 2, 0, 0);    /* gated, plain gates */
    layer(29, 8, 16, 6, 3, 1, 0);     /* gated, renormalised */
    layer(1, 8, 8, 3, 2, 1, 0);       /* a single token */
    layer(21, 16, 8, 4, 2, 0, 1);     /* non-gated SiLU */
    layer(17, 8, 16, 5, 4, 1, 2);     /* non-gated ReLU */
    printf("ok\n");
    return 0;
}
