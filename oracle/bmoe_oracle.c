/*
 * CPU oracle for the grouped ("full-brownout") MoE layer forward.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may link, load or
 * call this file; it is used by the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark. It shares no code, header or table with
 * the HIP library.
 *
 * What it computes (paper, Sec. 2.1 and Sec. 4.2 / Eq. 1-2, Sec. 4.3 closing
 * paragraphs, Sec. 4.4 closing paragraph):
 *   - an MoE layer computes h_t = sum over the top-K experts of
 *     g_i(x_t) * FFN_i(x_t) (Sec. 2.1);
 *   - grouping is a map g from the E experts to G groups (Eq. 2); under full
 *     brownout the gate still chooses each token's experts and every chosen
 *     expert is served by the united expert of its group (Sec. 4.3, last
 *     paragraph before Algorithm 1; Sec. 4.4, last paragraph).
 * The readings taken where the paper is silent are:
 *   - the gate is a linear router (plus an additive per-expert bias) followed
 *     by a softmax over all E experts; top-k selection is on the logits,
 *     descending, ties to the lower expert index; optional renormalisation of
 *     the k weights;
 *   - two chosen experts of one token that share a group make ONE call of that
 *     united expert with the sum of their weights (equal to two calls by
 *     linearity); the merged weight sits in the group's first slot, later
 *     duplicate slots carry group -1 and weight 0;
 *   - rows of a group are ordered by token index (stable counting sort);
 *   - every expert FFN is SwiGLU: y = W_down (silu(W_gate a) * (W_up a)),
 *     silu(v) = v / (1 + exp(-v)); weights in [out, in] layout;
 *   - shared experts are always on with weight 1.
 *
 * Arithmetic: every sum, product, exp and division is done in double, in
 * ascending index order; stage outputs are rounded once to float (the
 * interface precision). Router logits are also available in double, and
 * selection uses the double logits.
 *
 * Parity pins (checked by the CPU test-suite against things other than this
 * file): identity map with G=E equals the ungrouped layer of Sec. 2.1; G=1
 * equals top-k mass times one dense SwiGLU (textbook, library matmul);
 * merged and unmerged united-expert calls agree; top-k set equals the best
 * k-subset by brute force; token-order invariance; group weights sum to the
 * top-k mass; counting-sort bijection and stability.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads the following calls may use (timing runs only; no effect on results). */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------------ */
/* Gate logits (Sec. 2.1 "gating function"; linear router reading).
 * z[t*E+e] = sum_j x[t*d+j] * w[e*d+j]  (+ bias[e]), double, ascending j.   */
void oracle_router_logits(const float* x, const float* w, const float* bias,
                          int T, int d, int E, double* z) {
#pragma omp parallel for schedule(static)
    for (int t = 0; t < T; ++t) {
        const float* xt = x + (size_t)t * d;
        for (int e = 0; e < E; ++e) {
            const float* we = w + (size_t)e * d;
            double acc = 0.0;
            for (int j = 0; j < d; ++j) acc += (double)xt[j] * (double)we[j];
            if (bias) acc += (double)bias[e];
            z[(size_t)t * E + e] = acc;
        }
    }
}

/* Selection, gate weights and the expert-to-group substitution for one token.
 * z: E logits; e2g: map of Eq. 2 (0-based).                                  */
static void route_one(const double* z, const int32_t* e2g, int E, int k, int norm_topk,
                      int32_t* idx, float* w_out, int32_t* sgroup, float* sgate) {
    /* softmax over all experts */
    double m = z[0];
    for (int e = 1; e < E; ++e) if (z[e] > m) m = z[e];
    double s = 0.0;
    for (int e = 0; e < E; ++e) s += exp(z[e] - m);

    /* top-k: k passes of "largest not yet taken", first index wins ties */
    unsigned char taken[1024];
    memset(taken, 0, (size_t)E);
    double w[64];
    int pick[64];
    for (int i = 0; i < k; ++i) {
        int best = -1;
        for (int e = 0; e < E; ++e) {
            if (taken[e]) continue;
            if (best < 0 || z[e] > z[best]) best = e;
        }
        taken[best] = 1;
        pick[i] = best;
        w[i] = exp(z[best] - m) / s;
    }
    if (norm_topk) {
        double tot = 0.0;
        for (int i = 0; i < k; ++i) tot += w[i];
        for (int i = 0; i < k; ++i) w[i] = w[i] / tot;
    }
    /* substitution by united experts, one call per distinct group */
    for (int i = 0; i < k; ++i) {
        idx[i] = pick[i];
        w_out[i] = (float)w[i];
        int r = e2g[pick[i]];
        int first = 1;
        for (int j = 0; j < i; ++j) if (e2g[pick[j]] == r) first = 0;
        if (first) {
            double g = 0.0;
            for (int j = i; j < k; ++j) if (e2g[pick[j]] == r) g += w[j];
            sgroup[i] = r;
            sgate[i] = (float)g;
        } else {
            sgroup[i] = -1;
            sgate[i] = 0.0f;
        }
    }
}

/* Route every token from double logits z[T*E]. Outputs are [T*k]. */
void oracle_route_from_logits(const double* z, const int32_t* e2g, int T, int E, int k,
                              int norm_topk, int32_t* topk_idx, float* topk_w,
                              int32_t* slot_group, float* slot_gate) {
#pragma omp parallel for schedule(static)
    for (int t = 0; t < T; ++t)
        route_one(z + (size_t)t * E, e2g, E, k, norm_topk, topk_idx + (size_t)t * k,
                  topk_w + (size_t)t * k, slot_group + (size_t)t * k, slot_gate + (size_t)t * k);
}

/* Same from float logits (the selection then runs on those exact values). */
void oracle_route_from_logits_f32(const float* zf, const int32_t* e2g, int T, int E, int k,
                                  int norm_topk, int32_t* topk_idx, float* topk_w,
                                  int32_t* slot_group, float* slot_gate) {
#pragma omp parallel for schedule(static)
    for (int t = 0; t < T; ++t) {
        double z[1024];
        for (int e = 0; e < E; ++e) z[e] = (double)zf[(size_t)t * E + e];
        route_one(z, e2g, E, k, norm_topk, topk_idx + (size_t)t * k, topk_w + (size_t)t * k,
                  slot_group + (size_t)t * k, slot_gate + (size_t)t * k);
    }
}

/* ------------------------------------------------------------------------ */
/* Dispatch: per-group row counts, their exclusive prefix, and the stable
 * permutation of (token, group) pairs (group-major, token-minor).
 * counts[G], offsets[G+1], perm_token[N], slot_row[T*k] (-1 where merged).
 * Returns N = offsets[G].                                                    */
int oracle_dispatch(const int32_t* slot_group, int T, int k, int G, int32_t* counts,
                    int32_t* offsets, int32_t* perm_token, int32_t* slot_row) {
    for (int r = 0; r < G; ++r) counts[r] = 0;
    for (int i = 0; i < T * k; ++i) {
        slot_row[i] = -1;
        if (slot_group[i] >= 0) counts[slot_group[i]] += 1;
    }
    offsets[0] = 0;
    for (int r = 0; r < G; ++r) offsets[r + 1] = offsets[r] + counts[r];
    int pos = 0;
    for (int r = 0; r < G; ++r) {
        for (int t = 0; t < T; ++t) {
            for (int i = 0; i < k; ++i) {
                if (slot_group[(size_t)t * k + i] == r) {
                    perm_token[pos] = t;
                    slot_row[(size_t)t * k + i] = pos;
                    ++pos;
                }
            }
        }
    }
    return pos;
}

/* Row gather: x_perm[row] = x[perm_token[row]] for row < N. */
void oracle_gather_rows(const float* x, const int32_t* perm_token, int N, int d, float* x_perm) {
    for (int r = 0; r < N; ++r)
        memcpy(x_perm + (size_t)r * d, x + (size_t)perm_token[r] * d, sizeof(float) * (size_t)d);
}

/* ------------------------------------------------------------------------ */
/* Grouped SwiGLU FFN. Segment s covers rows [offsets[s], offsets[s+1]) of a
 * and uses w_gate[s], w_up[s] ([d_ff, d]) and w_down[s] ([d, d_ff]).
 * y[row] = W_down (silu(W_gate a) * (W_up a)); h (optional) gets the hidden
 * activation.                                                                */
void oracle_ffn(int n_seg, const int32_t* offsets, int d, int d_ff, const float* a,
                const float* w_gate, const float* w_up, const float* w_down,
                float* h_out, float* y) {
    int N = offsets[n_seg];
    int* seg_of = (int*)malloc(sizeof(int) * (size_t)(N > 0 ? N : 1));
    for (int s = 0; s < n_seg; ++s)
        for (int r = offsets[s]; r < offsets[s + 1]; ++r) seg_of[r] = s;
#pragma omp parallel
    {
        double* hbuf = (double*)malloc(sizeof(double) * (size_t)d_ff);
#pragma omp for schedule(dynamic, 1)
        for (int r = 0; r < N; ++r) {
            int s = seg_of[r];
            const float* ar = a + (size_t)r * d;
            const float* wg = w_gate + (size_t)s * d_ff * d;
            const float* wu = w_up + (size_t)s * d_ff * d;
            const float* wd = w_down + (size_t)s * d * d_ff;
            for (int j = 0; j < d_ff; ++j) {
                double g = 0.0, u = 0.0;
                const float* gj = wg + (size_t)j * d;
                const float* uj = wu + (size_t)j * d;
                for (int c = 0; c < d; ++c) {
                    g += (double)gj[c] * (double)ar[c];
                    u += (double)uj[c] * (double)ar[c];
                }
                double silu = g / (1.0 + exp(-g));
                hbuf[j] = silu * u;
                if (h_out) h_out[(size_t)r * d_ff + j] = (float)hbuf[j];
            }
            for (int i = 0; i < d; ++i) {
                const float* di = wd + (size_t)i * d_ff;
                double acc = 0.0;
                for (int j = 0; j < d_ff; ++j) acc += (double)di[j] * hbuf[j];
                y[(size_t)r * d + i] = (float)acc;
            }
        }
        free(hbuf);
    }
    free(seg_of);
}

/* ------------------------------------------------------------------------ */
/* Combine: out[t] = sum over slots i of t with slot_row >= 0 (ascending i) of
 * slot_gate[t,i] * y[slot_row[t,i]], plus y_shared[t] when given.            */
void oracle_combine(const int32_t* slot_row, const float* slot_gate, const float* y,
                    const float* y_shared, int T, int k, int d, float* out) {
#pragma omp parallel for schedule(static)
    for (int t = 0; t < T; ++t) {
        for (int c = 0; c < d; ++c) {
            double acc = 0.0;
            for (int i = 0; i < k; ++i) {
                int row = slot_row[(size_t)t * k + i];
                if (row >= 0) acc += (double)slot_gate[(size_t)t * k + i] * (double)y[(size_t)row * d + c];
            }
            if (y_shared) acc += (double)y_shared[(size_t)t * d + c];
            out[(size_t)t * d + c] = (float)acc;
        }
    }
}
