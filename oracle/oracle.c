/*
 * Oracle for the message-passing propagate path of PyTorch Geometric
 * (Fey & Lenssen, "Fast Graph Representation Learning with PyTorch
 * Geometric", ICLR-W 2019).
 *
 * TEST INFRASTRUCTURE. This file is the plain, slow, obviously correct CPU
 * definition that the HIP library is checked against. Only the test suite,
 * the smoke check and the benchmark's cpu_baseline leg may load it; the
 * library never calls it. It shares no source, header, table or helper with
 * the HIP library.
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared (no fast-math, no OpenMP).
 * On x86-64 float arithmetic is IEEE single precision with no excess
 * precision, so a C `float` product or difference is one correctly rounded
 * fp32 operation.
 *
 * Conventions (readings of the paper, Section 2):
 *  - A graph is G = (X, (I, E)); X is [N, F] row-major fp32, I is the COO
 *    index matrix stored as int64 [2, E] row-major.
 *  - Row 0 of I is the source j, row 1 the target i: Eq. (1) aggregates
 *    phi(x_i, x_j, e_{j,i}) over j in N(i), i.e. along edges j -> i.
 *  - Multi-edges count with multiplicity (multiset semantics).
 *  - An empty neighbourhood aggregates to 0; its argmax is the sentinel E
 *    (propagate) or N (pooling).
 *  - max: messages are compared in fp32 after mapping -0.0 to +0.0; among
 *    equal maxima the lowest edge id (first in COO order) wins.
 *  - mean divides by the number of incoming edges, also when weighted.
 *  - Inputs must be finite; a NaN or Inf input returns ORACLE_ERR_NONFINITE.
 *
 * Sum and mean accumulate in fp64 (the message w * x_j of two fp32 numbers
 * is exact in fp64). Alongside every sum the oracle returns S = sum of
 * |message| per output element, the scale of the fp32 rounding error that
 * any reordering of the same sum may carry.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#define ORACLE_OK 0
#define ORACLE_ERR_ARG (-1)
#define ORACLE_ERR_INDEX (-2)
#define ORACLE_ERR_NONFINITE (-3)

/* message kinds phi (Eq. 1) */
#define ORACLE_MSG_SRC 0       /* x_j, times w_{j,i} when a weight is given */
#define ORACLE_MSG_DIFF 1      /* x_j - x_i (EdgeConv-style) */
#define ORACLE_MSG_EDGE_ADD 2  /* x_j + e_{j,i} (F-dimensional edge features) */
#define ORACLE_MSG_EDGE_RELU 3 /* max(x_j + e_{j,i}, 0) */
#define ORACLE_MSG_EDGE_MUL 4  /* x_j * e_{j,i}, elementwise */

/* aggregations (the permutation-invariant operator of Eq. 1) */
#define ORACLE_SUM 0
#define ORACLE_MEAN 1
#define ORACLE_MAX 2

int oracle_abi_version(void) { return 1; }

static int check_index_range(const int64_t *idx, int64_t count, int64_t bound) {
    for (int64_t k = 0; k < count; ++k)
        if (idx[k] < 0 || idx[k] >= bound) return ORACLE_ERR_INDEX;
    return ORACLE_OK;
}

/* In-degree: deg[i] = number of edges whose target is i (Eq. 1's |N(i)|,
 * counted with multiplicity). */
int oracle_degree(const int64_t *edge_index, int64_t E, int64_t N, int64_t *deg) {
    if (E < 0 || N < 0 || (E > 0 && !edge_index) || (N > 0 && !deg)) return ORACLE_ERR_ARG;
    const int64_t *dst = edge_index + E;
    if (check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    for (int64_t i = 0; i < N; ++i) deg[i] = 0;
    for (int64_t k = 0; k < E; ++k) deg[dst[k]] += 1;
    return ORACLE_OK;
}

/* Compressed-row (CSR) form of the COO edge list, rows = targets
 * (Appendix A: the row-ordered, "coalesced" layout that sparse-matrix
 * multiplication needs). Counting sort, stable by construction: inside a
 * row the edges keep ascending original edge id.
 *   rowptr [N+1], col [E] = source of each CSR slot, perm [E] = edge id. */
int oracle_coo_to_csr(const int64_t *edge_index, int64_t E, int64_t N,
                      int64_t *rowptr, int64_t *col, int64_t *perm) {
    if (E < 0 || N < 0 || !rowptr || (E > 0 && (!edge_index || !col || !perm))) return ORACLE_ERR_ARG;
    const int64_t *src = edge_index;
    const int64_t *dst = edge_index + E;
    if (check_index_range(src, E, N) || check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    for (int64_t i = 0; i <= N; ++i) rowptr[i] = 0;
    for (int64_t k = 0; k < E; ++k) rowptr[dst[k] + 1] += 1;
    for (int64_t i = 0; i < N; ++i) rowptr[i + 1] += rowptr[i];
    int64_t *next = (int64_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int64_t));
    if (!next) return ORACLE_ERR_ARG;
    for (int64_t i = 0; i < N; ++i) next[i] = rowptr[i];
    for (int64_t k = 0; k < E; ++k) {
        int64_t p = next[dst[k]]++;
        col[p] = src[k];
        perm[p] = k;
    }
    free(next);
    return ORACLE_OK;
}

/* GCN normalisation (the GCN operator of Section 2, as used by the configs):
 * on an edge list that already holds the self-loops,
 *   d_i    = sum of w_k over edges k with target i   (w = 1 when absent),
 *   dinv_i = 1 / sqrt(d_i), or 0 when d_i = 0,
 *   norm_k = dinv_j * w_k * dinv_i          for edge k = (j -> i),
 * all in fp64. */
int oracle_gcn_norm(const int64_t *edge_index, const double *w, int64_t E, int64_t N, double *norm) {
    if (E < 0 || N < 0 || (E > 0 && (!edge_index || !norm))) return ORACLE_ERR_ARG;
    const int64_t *src = edge_index;
    const int64_t *dst = edge_index + E;
    if (check_index_range(src, E, N) || check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    double *d = (double *)calloc((size_t)(N > 0 ? N : 1), sizeof(double));
    if (!d) return ORACLE_ERR_ARG;
    for (int64_t k = 0; k < E; ++k) d[dst[k]] += w ? w[k] : 1.0;
    for (int64_t i = 0; i < N; ++i) d[i] = d[i] > 0.0 ? 1.0 / sqrt(d[i]) : 0.0;
    for (int64_t k = 0; k < E; ++k) norm[k] = d[src[k]] * (w ? w[k] : 1.0) * d[dst[k]];
    free(d);
    return ORACLE_OK;
}

/* Shared by propagate and pooling: reduce messages m_k (k = 0..E-1, in
 * order) into rows tgt[k]. The message of element (k, f) is built by
 * the caller-supplied source row, weight, (for DIFF) target row and (for
 * the EDGE kinds) edge feature row ea[k]. */
static int reduce_edges(const float *x, int64_t N_src, int64_t F,
                        const int64_t *src, const int64_t *tgt, int64_t E, int64_t N_out,
                        const float *w, const float *ea, int msg, int aggr,
                        double *out, int64_t *argmax, double *sabs, int64_t sentinel) {
    int64_t *cnt = (int64_t *)calloc((size_t)(N_out > 0 ? N_out : 1), sizeof(int64_t));
    float *best = (float *)malloc((size_t)((N_out * F) > 0 ? N_out * F : 1) * sizeof(float));
    if (!cnt || !best) { free(cnt); free(best); return ORACLE_ERR_ARG; }
    for (int64_t t = 0; t < N_out * F; ++t) {
        out[t] = 0.0;
        if (sabs) sabs[t] = 0.0;
        if (argmax) argmax[t] = sentinel;
        best[t] = 0.0f;
    }
    for (int64_t k = 0; k < E; ++k) {
        const int64_t j = src[k], i = tgt[k];
        cnt[i] += 1;
        for (int64_t f = 0; f < F; ++f) {
            const float xj = x[j * F + f];
            const int64_t o = i * F + f;
            if (aggr == ORACLE_MAX) {
                float m;
                if (msg == ORACLE_MSG_DIFF) m = xj - x[i * F + f];
                else if (msg == ORACLE_MSG_EDGE_ADD) m = xj + ea[k * F + f];
                else if (msg == ORACLE_MSG_EDGE_RELU) m = xj + ea[k * F + f] > 0.0f ? xj + ea[k * F + f] : 0.0f;
                else if (msg == ORACLE_MSG_EDGE_MUL) m = xj * ea[k * F + f];
                else if (w) m = w[k] * xj;
                else m = xj;
                if (m == 0.0f) m = 0.0f; /* -0.0 -> +0.0 */
                if (argmax[o] == sentinel || m > best[o]) {
                    best[o] = m;
                    argmax[o] = k;
                }
            } else {
                double m;
                if (msg == ORACLE_MSG_DIFF) m = (double)xj - (double)x[i * F + f];
                else if (msg == ORACLE_MSG_EDGE_ADD) m = (double)xj + (double)ea[k * F + f];
                else if (msg == ORACLE_MSG_EDGE_RELU) m = fmax((double)xj + (double)ea[k * F + f], 0.0);
                else if (msg == ORACLE_MSG_EDGE_MUL) m = (double)xj * (double)ea[k * F + f];
                else if (w) m = (double)w[k] * (double)xj;
                else m = (double)xj;
                out[o] += m;
                if (sabs) sabs[o] += fabs(m);
            }
        }
    }
    for (int64_t i = 0; i < N_out; ++i) {
        for (int64_t f = 0; f < F; ++f) {
            const int64_t o = i * F + f;
            if (aggr == ORACLE_MAX) {
                out[o] = cnt[i] > 0 ? (double)best[o] : 0.0;
            } else if (aggr == ORACLE_MEAN && cnt[i] > 0) {
                out[o] = out[o] / (double)cnt[i];
                if (sabs) sabs[o] = sabs[o] / (double)cnt[i];
            }
        }
    }
    free(cnt);
    free(best);
    return ORACLE_OK;
}

static int all_finite(const float *a, int64_t n) {
    for (int64_t t = 0; t < n; ++t)
        if (!isfinite(a[t])) return 0;
    return 1;
}

/* Propagate, Eq. (1) with gamma = identity:
 *   out_i = AGG_{k : I[1,k] = i} phi_k,
 *   phi_k = x_j (SRC), w_k * x_j (SRC with weight), x_j - x_i (DIFF), or,
 *   with F-dimensional edge features e_k = ea[k] (the e_{j,i} of Eq. 1):
 *   x_j + e_k (EDGE_ADD), max(x_j + e_k, 0) (EDGE_RELU), x_j * e_k (EDGE_MUL),
 * for every feature column. out is fp64 [N,F]; argmax (int64 [N,F], max
 * only, else may be NULL) holds the winning edge id; sabs (nullable) holds
 * sum |phi| (divided by the degree for mean). Max compares the messages
 * formed in fp32 (one fp32 add or multiply). */
int oracle_propagate(const float *x, int64_t N, int64_t F,
                     const int64_t *edge_index, int64_t E, const float *w, const float *ea,
                     int msg, int aggr, double *out, int64_t *argmax, double *sabs) {
    if (N < 0 || F < 0 || E < 0) return ORACLE_ERR_ARG;
    if (msg < ORACLE_MSG_SRC || msg > ORACLE_MSG_EDGE_MUL) return ORACLE_ERR_ARG;
    if (aggr != ORACLE_SUM && aggr != ORACLE_MEAN && aggr != ORACLE_MAX) return ORACLE_ERR_ARG;
    const int edge_msg = msg >= ORACLE_MSG_EDGE_ADD;
    if (w && msg != ORACLE_MSG_SRC) return ORACLE_ERR_ARG;
    if (edge_msg != (ea != NULL) && E * F > 0) return ORACLE_ERR_ARG;
    if (aggr == ORACLE_MAX && N * F > 0 && !argmax) return ORACLE_ERR_ARG;
    if (N * F > 0 && (!x || !out)) return ORACLE_ERR_ARG;
    if (E > 0 && !edge_index) return ORACLE_ERR_ARG;
    const int64_t *src = edge_index;
    const int64_t *dst = edge_index + E;
    if (check_index_range(src, E, N) || check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    if (!all_finite(x, N * F) || (w && !all_finite(w, E)) || (ea && !all_finite(ea, E * F))) return ORACLE_ERR_NONFINITE;
    return reduce_edges(x, N, F, src, dst, E, N, w, ea, msg, aggr, out, argmax, sabs, E);
}

/* Global pooling (Section 2, "Global Pooling" and "Mini-batch Handling"):
 * out_g = AGG_{n : batch[n] = g} x_n, for B graphs. The assignment vector
 * batch must be non-decreasing. argmax holds the winning node id, N if the
 * graph is empty. */
int oracle_global_pool(const float *x, int64_t N, int64_t F, const int64_t *batch, int64_t B,
                       int aggr, double *out, int64_t *argmax, double *sabs) {
    if (N < 0 || F < 0 || B < 0) return ORACLE_ERR_ARG;
    if (aggr != ORACLE_SUM && aggr != ORACLE_MEAN && aggr != ORACLE_MAX) return ORACLE_ERR_ARG;
    if (aggr == ORACLE_MAX && B * F > 0 && !argmax) return ORACLE_ERR_ARG;
    if (N > 0 && !batch) return ORACLE_ERR_ARG;
    if (B * F > 0 && !out) return ORACLE_ERR_ARG;
    if (check_index_range(batch, N, B)) return ORACLE_ERR_INDEX;
    for (int64_t n = 1; n < N; ++n)
        if (batch[n] < batch[n - 1]) return ORACLE_ERR_ARG;
    if (!all_finite(x, N * F)) return ORACLE_ERR_NONFINITE;
    int64_t *node = (int64_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int64_t));
    if (!node) return ORACLE_ERR_ARG;
    for (int64_t n = 0; n < N; ++n) node[n] = n;
    int rc = reduce_edges(x, N, F, node, batch, N, B, NULL, NULL, ORACLE_MSG_SRC, aggr, out, argmax, sabs, N);
    free(node);
    return rc;
}

/* Gradient of oracle_propagate (Eq. (1), gamma = identity) for a given
 * upstream gradient g = dL/d out [N,F]:
 *   sum / mean: every edge k = (j -> i) passes s_i * g_i back, s_i = 1 (sum) or
 *     1/deg_i (mean):  grad_x[j] += w_k s_i g_i,  grad_w[k] += s_i <g_i, x_j>;
 *     for DIFF (phi = x_j - x_i):  grad_x[j] += s_i g_i,  grad_x[i] -= s_i g_i.
 *   max: only the winning edge k = argmax[i,f] of each output element receives
 *     it:  grad_x[j,f] += w_k g_{i,f},  grad_w[k] += g_{i,f} x_{j,f};
 *     DIFF: grad_x[j,f] += g_{i,f}, grad_x[i,f] -= g_{i,f}. Empty rows pass nothing.
 * argmax is the forward's (sentinel E for empty rows). grad_x fp64 [N,F];
 * grad_w fp64 [E] (nullable; needs a weight and msg SRC); sabs_x / sabs_w
 * (nullable) hold the sum of |terms| of each output. */
int oracle_propagate_backward(const float *x, int64_t N, int64_t F, const int64_t *edge_index, int64_t E,
                              const float *w, int msg, int aggr, const float *grad_out, const int64_t *argmax,
                              double *grad_x, double *grad_w, double *sabs_x, double *sabs_w) {
    if (N < 0 || F < 0 || E < 0) return ORACLE_ERR_ARG;
    if (msg != ORACLE_MSG_SRC && msg != ORACLE_MSG_DIFF) return ORACLE_ERR_ARG;
    if (aggr != ORACLE_SUM && aggr != ORACLE_MEAN && aggr != ORACLE_MAX) return ORACLE_ERR_ARG;
    if (msg == ORACLE_MSG_DIFF && w) return ORACLE_ERR_ARG;
    if (grad_w && (!w || msg != ORACLE_MSG_SRC)) return ORACLE_ERR_ARG;
    if (N * F > 0 && (!x || !grad_out || !grad_x)) return ORACLE_ERR_ARG;
    if (aggr == ORACLE_MAX && N * F > 0 && !argmax) return ORACLE_ERR_ARG;
    if (E > 0 && !edge_index) return ORACLE_ERR_ARG;
    const int64_t *src = edge_index;
    const int64_t *dst = edge_index + E;
    if (check_index_range(src, E, N) || check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    if (!all_finite(x, N * F) || !all_finite(grad_out, N * F) || (w && !all_finite(w, E))) return ORACLE_ERR_NONFINITE;
    for (int64_t t = 0; t < N * F; ++t) {
        grad_x[t] = 0.0;
        if (sabs_x) sabs_x[t] = 0.0;
    }
    for (int64_t k = 0; k < E && grad_w; ++k) {
        grad_w[k] = 0.0;
        if (sabs_w) sabs_w[k] = 0.0;
    }
    if (aggr == ORACLE_MAX) {
        for (int64_t i = 0; i < N; ++i) {
            for (int64_t f = 0; f < F; ++f) {
                const int64_t k = argmax[i * F + f];
                if (k == E) continue; /* empty row */
                if (k < 0 || k > E || dst[k] != i) return ORACLE_ERR_INDEX;
                const int64_t j = src[k];
                const double g = grad_out[i * F + f];
                if (msg == ORACLE_MSG_DIFF) {
                    grad_x[j * F + f] += g;
                    grad_x[i * F + f] -= g;
                    if (sabs_x) {
                        sabs_x[j * F + f] += fabs(g);
                        sabs_x[i * F + f] += fabs(g);
                    }
                } else {
                    const double wk = w ? (double)w[k] : 1.0;
                    grad_x[j * F + f] += wk * g;
                    if (sabs_x) sabs_x[j * F + f] += fabs(wk * g);
                    if (grad_w) {
                        grad_w[k] += g * (double)x[j * F + f];
                        if (sabs_w) sabs_w[k] += fabs(g * (double)x[j * F + f]);
                    }
                }
            }
        }
        return ORACLE_OK;
    }
    int64_t *deg = (int64_t *)calloc((size_t)(N > 0 ? N : 1), sizeof(int64_t));
    if (!deg) return ORACLE_ERR_ARG;
    for (int64_t k = 0; k < E; ++k) deg[dst[k]] += 1;
    for (int64_t k = 0; k < E; ++k) {
        const int64_t j = src[k], i = dst[k];
        const double sc = aggr == ORACLE_MEAN ? 1.0 / (double)deg[i] : 1.0;
        const double wk = w ? (double)w[k] : 1.0;
        for (int64_t f = 0; f < F; ++f) {
            const double g = sc * (double)grad_out[i * F + f];
            if (msg == ORACLE_MSG_DIFF) {
                grad_x[j * F + f] += g;
                grad_x[i * F + f] -= g;
                if (sabs_x) {
                    sabs_x[j * F + f] += fabs(g);
                    sabs_x[i * F + f] += fabs(g);
                }
            } else {
                grad_x[j * F + f] += wk * g;
                if (sabs_x) sabs_x[j * F + f] += fabs(wk * g);
                if (grad_w) {
                    grad_w[k] += g * (double)x[j * F + f];
                    if (sabs_w) sabs_w[k] += fabs(g * (double)x[j * F + f]);
                }
            }
        }
    }
    free(deg);
    return ORACLE_OK;
}

/* Gradient of oracle_propagate with the edge-feature messages (Eq. (1) with
 * F-dimensional e_{j,i}; phi = x_j + e, max(x_j + e, 0) or x_j * e,
 * elementwise) for g = dL/d out [N,F]. Each edge k = (j -> i) receives
 * d_k = s_i g_i (sum: s_i = 1, mean: s_i = 1/deg_i), or, for max, g_{i,f}
 * in the columns f where k is the forward's argmax[i,f] and 0 elsewhere;
 * then by the chain rule through phi:
 *   x_j + e:          grad_x[j] += d_k,             grad_e[k] = d_k;
 *   max(x_j + e, 0):  both times [x_j + e_k > 0] (the sign of the exact sum;
 *                     a message that is exactly 0 passes nothing);
 *   x_j * e:          grad_x[j] += d_k * e_k,       grad_e[k] = d_k * x_j.
 * grad_x fp64 [N,F], grad_e fp64 [E,F] in edge order (either may be NULL,
 * not both); sabs_x / sabs_e (nullable) hold the sum of |terms|. */
int oracle_propagate_edge_backward(const float *x, int64_t N, int64_t F, const int64_t *edge_index, int64_t E,
                                   const float *ea, int msg, int aggr, const float *grad_out,
                                   const int64_t *argmax, double *grad_x, double *grad_e, double *sabs_x,
                                   double *sabs_e) {
    if (N < 0 || F < 0 || E < 0) return ORACLE_ERR_ARG;
    if (msg != ORACLE_MSG_EDGE_ADD && msg != ORACLE_MSG_EDGE_RELU && msg != ORACLE_MSG_EDGE_MUL) return ORACLE_ERR_ARG;
    if (aggr != ORACLE_SUM && aggr != ORACLE_MEAN && aggr != ORACLE_MAX) return ORACLE_ERR_ARG;
    if (!grad_x && !grad_e) return ORACLE_ERR_ARG;
    if (N * F > 0 && (!x || !grad_out)) return ORACLE_ERR_ARG;
    if (E * F > 0 && !ea) return ORACLE_ERR_ARG;
    if (aggr == ORACLE_MAX && N * F > 0 && !argmax) return ORACLE_ERR_ARG;
    if (E > 0 && !edge_index) return ORACLE_ERR_ARG;
    const int64_t *src = edge_index;
    const int64_t *dst = edge_index + E;
    if (check_index_range(src, E, N) || check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    if (!all_finite(x, N * F) || !all_finite(grad_out, N * F) || !all_finite(ea, E * F)) return ORACLE_ERR_NONFINITE;
    for (int64_t t = 0; grad_x && t < N * F; ++t) {
        grad_x[t] = 0.0;
        if (sabs_x) sabs_x[t] = 0.0;
    }
    for (int64_t t = 0; grad_e && t < E * F; ++t) {
        grad_e[t] = 0.0;
        if (sabs_e) sabs_e[t] = 0.0;
    }
    int64_t *deg = (int64_t *)calloc((size_t)(N > 0 ? N : 1), sizeof(int64_t));
    if (!deg) return ORACLE_ERR_ARG;
    for (int64_t k = 0; k < E; ++k) deg[dst[k]] += 1;
    for (int64_t k = 0; k < E; ++k) {
        const int64_t j = src[k], i = dst[k];
        for (int64_t f = 0; f < F; ++f) {
            double d;
            if (aggr == ORACLE_MAX) {
                const int64_t a = argmax[i * F + f];
                if (a < 0 || a > E) { free(deg); return ORACLE_ERR_INDEX; }
                d = a == k ? (double)grad_out[i * F + f] : 0.0;
            } else {
                d = (double)grad_out[i * F + f];
                if (aggr == ORACLE_MEAN) d /= (double)deg[i];
            }
            const double xj = x[j * F + f], e = ea[k * F + f];
            double dx, de;
            if (msg == ORACLE_MSG_EDGE_ADD) {
                dx = d;
                de = d;
            } else if (msg == ORACLE_MSG_EDGE_RELU) {
                const double on = xj + e > 0.0 ? 1.0 : 0.0;
                dx = d * on;
                de = d * on;
            } else {
                dx = d * e;
                de = d * xj;
            }
            if (grad_x) {
                grad_x[j * F + f] += dx;
                if (sabs_x) sabs_x[j * F + f] += fabs(dx);
            }
            if (grad_e) {
                grad_e[k * F + f] = de;
                if (sabs_e) sabs_e[k * F + f] = fabs(de);
            }
        }
    }
    free(deg);
    return ORACLE_OK;
}

/* ---------------------------------------------------------------------------
 * Attention over incoming edges (Section 2 names GAT among the operators
 * expressed by Eq. (1); Section 3, runtime paragraph, credits GAT's speed to
 * a dedicated sparse softmax). With H attention heads every edge k carries
 * H scores s[k,h] (row-major [E,H]).
 * ------------------------------------------------------------------------- */

/* GAT edge score for edge k = (j -> i) and head h:
 *   e[k,h] = LeakyReLU(a_src[j,h] + a_dst[i,h]),  LeakyReLU(v) = v if v >= 0,
 * slope * v otherwise. a_src / a_dst are the per-node halves of GAT's
 * attention vector applied to the transformed features, fp32 [N,H]. The
 * sum of two fp32 numbers and its product with an fp32 slope are exact in
 * fp64. e is fp64 [E,H]. */
int oracle_gat_scores(const float *a_src, const float *a_dst, int64_t N, int64_t H,
                      const int64_t *edge_index, int64_t E, float slope, double *e) {
    if (N < 0 || H < 0 || E < 0) return ORACLE_ERR_ARG;
    if (E * H > 0 && (!a_src || !a_dst || !edge_index || !e)) return ORACLE_ERR_ARG;
    const int64_t *src = edge_index;
    const int64_t *dst = edge_index + E;
    if (check_index_range(src, E, N) || check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    if (!all_finite(a_src, N * H) || !all_finite(a_dst, N * H) || !isfinite(slope)) return ORACLE_ERR_NONFINITE;
    for (int64_t k = 0; k < E; ++k)
        for (int64_t h = 0; h < H; ++h) {
            const double v = (double)a_src[src[k] * H + h] + (double)a_dst[dst[k] * H + h];
            e[k * H + h] = v >= 0.0 ? v : (double)slope * v;
        }
    return ORACLE_OK;
}

/* Softmax over the incoming edges of every target, per head:
 *   alpha[k,h] = exp(s[k,h] - m[i,h]) / sum_{k' : I[1,k'] = i} exp(s[k',h] - m[i,h]),
 *   m[i,h] = max_{k' : I[1,k'] = i} s[k',h],  i = I[1,k].
 * Subtracting the segment maximum leaves the value unchanged and keeps
 * every exponential in (0, 1]. Targets without incoming edges own no
 * entries. s fp64 [E,H]; alpha fp64 [E,H]. */
int oracle_segment_softmax(const double *s, int64_t E, int64_t H, const int64_t *edge_index, int64_t N,
                           double *alpha) {
    if (N < 0 || H < 0 || E < 0) return ORACLE_ERR_ARG;
    if (E * H > 0 && (!s || !edge_index || !alpha)) return ORACLE_ERR_ARG;
    const int64_t *dst = edge_index + E;
    if (check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    for (int64_t t = 0; t < E * H; ++t)
        if (!isfinite(s[t])) return ORACLE_ERR_NONFINITE;
    double *m = (double *)malloc((size_t)(N * H > 0 ? N * H : 1) * sizeof(double));
    double *den = (double *)malloc((size_t)(N * H > 0 ? N * H : 1) * sizeof(double));
    if (!m || !den) {
        free(m);
        free(den);
        return ORACLE_ERR_ARG;
    }
    for (int64_t t = 0; t < N * H; ++t) {
        m[t] = -INFINITY;
        den[t] = 0.0;
    }
    for (int64_t k = 0; k < E; ++k)
        for (int64_t h = 0; h < H; ++h)
            if (s[k * H + h] > m[dst[k] * H + h]) m[dst[k] * H + h] = s[k * H + h];
    for (int64_t k = 0; k < E; ++k)
        for (int64_t h = 0; h < H; ++h) den[dst[k] * H + h] += exp(s[k * H + h] - m[dst[k] * H + h]);
    for (int64_t k = 0; k < E; ++k)
        for (int64_t h = 0; h < H; ++h)
            alpha[k * H + h] = exp(s[k * H + h] - m[dst[k] * H + h]) / den[dst[k] * H + h];
    free(m);
    free(den);
    return ORACLE_OK;
}

/* Gradient of the segment softmax for an upstream gradient g = dL/d alpha:
 *   grad_s[k,h] = alpha[k,h] * (g[k,h] - t[i,h]),  t[i,h] = sum_{k' in seg(i)} alpha[k',h] g[k',h].
 * alpha and g fp32 [E,H] (alpha as the forward stored it); grad_s fp64;
 * sabs (nullable) = |alpha g| + |alpha| sum_{k'} |alpha' g'|, the scale of
 * the rounding error of any evaluation order. */
int oracle_segment_softmax_backward(const float *alpha, const float *g, int64_t E, int64_t H,
                                    const int64_t *edge_index, int64_t N, double *grad_s, double *sabs) {
    if (N < 0 || H < 0 || E < 0) return ORACLE_ERR_ARG;
    if (E * H > 0 && (!alpha || !g || !edge_index || !grad_s)) return ORACLE_ERR_ARG;
    const int64_t *dst = edge_index + E;
    if (check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    if (!all_finite(alpha, E * H) || !all_finite(g, E * H)) return ORACLE_ERR_NONFINITE;
    double *t = (double *)calloc((size_t)(N * H > 0 ? N * H : 1), sizeof(double));
    double *ta = (double *)calloc((size_t)(N * H > 0 ? N * H : 1), sizeof(double));
    if (!t || !ta) {
        free(t);
        free(ta);
        return ORACLE_ERR_ARG;
    }
    for (int64_t k = 0; k < E; ++k)
        for (int64_t h = 0; h < H; ++h) {
            const double ag = (double)alpha[k * H + h] * (double)g[k * H + h];
            t[dst[k] * H + h] += ag;
            ta[dst[k] * H + h] += fabs(ag);
        }
    for (int64_t k = 0; k < E; ++k)
        for (int64_t h = 0; h < H; ++h) {
            const double a = alpha[k * H + h];
            grad_s[k * H + h] = a * ((double)g[k * H + h] - t[dst[k] * H + h]);
            if (sabs) sabs[k * H + h] = fabs(a * (double)g[k * H + h]) + fabs(a) * ta[dst[k] * H + h];
        }
    free(t);
    free(ta);
    return ORACLE_OK;
}

/* Attention-weighted aggregation with H heads (GAT's message alpha_{j,i} x_j
 * under sum aggregation, Eq. (1), heads concatenated): x is [N, H*C] with
 * head h owning columns h*C .. h*C+C-1, and
 *   out[i, h*C + c] = sum_{k : I[1,k] = i} alpha[k,h] * x[I[0,k], h*C + c].
 * alpha fp32 [E,H]; out fp64 [N, H*C]; sabs (nullable) = sum |term|. */
int oracle_propagate_heads(const float *x, int64_t N, int64_t H, int64_t C, const int64_t *edge_index, int64_t E,
                           const float *alpha, double *out, double *sabs) {
    if (N < 0 || H < 0 || C < 0 || E < 0) return ORACLE_ERR_ARG;
    const int64_t F = H * C;
    if (N * F > 0 && (!x || !out)) return ORACLE_ERR_ARG;
    if (E * H > 0 && (!alpha || !edge_index)) return ORACLE_ERR_ARG;
    const int64_t *src = edge_index;
    const int64_t *dst = edge_index + E;
    if (check_index_range(src, E, N) || check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    if (!all_finite(x, N * F) || !all_finite(alpha, E * H)) return ORACLE_ERR_NONFINITE;
    for (int64_t t = 0; t < N * F; ++t) {
        out[t] = 0.0;
        if (sabs) sabs[t] = 0.0;
    }
    for (int64_t k = 0; k < E; ++k)
        for (int64_t h = 0; h < H; ++h) {
            const double a = alpha[k * H + h];
            for (int64_t c = 0; c < C; ++c) {
                const double term = a * (double)x[src[k] * F + h * C + c];
                out[dst[k] * F + h * C + c] += term;
                if (sabs) sabs[dst[k] * F + h * C + c] += fabs(term);
            }
        }
    return ORACLE_OK;
}

/* Gradient of oracle_propagate_heads for g = dL/d out [N, H*C]:
 *   grad_x[j, h*C + c] += alpha[k,h] g[i, h*C + c],
 *   grad_alpha[k,h]     = sum_c g[i, h*C + c] x[j, h*C + c],   k = (j -> i).
 * grad_x fp64 [N, H*C], grad_alpha fp64 [E,H] (nullable), sabs_* nullable. */
int oracle_propagate_heads_backward(const float *x, int64_t N, int64_t H, int64_t C, const int64_t *edge_index,
                                    int64_t E, const float *alpha, const float *g, double *grad_x,
                                    double *grad_alpha, double *sabs_x, double *sabs_a) {
    if (N < 0 || H < 0 || C < 0 || E < 0) return ORACLE_ERR_ARG;
    const int64_t F = H * C;
    if (N * F > 0 && (!x || !g || !grad_x)) return ORACLE_ERR_ARG;
    if (E * H > 0 && (!alpha || !edge_index)) return ORACLE_ERR_ARG;
    const int64_t *src = edge_index;
    const int64_t *dst = edge_index + E;
    if (check_index_range(src, E, N) || check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    if (!all_finite(x, N * F) || !all_finite(g, N * F) || !all_finite(alpha, E * H)) return ORACLE_ERR_NONFINITE;
    for (int64_t t = 0; t < N * F; ++t) {
        grad_x[t] = 0.0;
        if (sabs_x) sabs_x[t] = 0.0;
    }
    for (int64_t k = 0; k < E; ++k)
        for (int64_t h = 0; h < H; ++h) {
            const int64_t j = src[k], i = dst[k];
            const double a = alpha[k * H + h];
            double dot = 0.0, dabs = 0.0;
            for (int64_t c = 0; c < C; ++c) {
                const double gi = g[i * F + h * C + c];
                grad_x[j * F + h * C + c] += a * gi;
                if (sabs_x) sabs_x[j * F + h * C + c] += fabs(a * gi);
                dot += gi * (double)x[j * F + h * C + c];
                dabs += fabs(gi * (double)x[j * F + h * C + c]);
            }
            if (grad_alpha) grad_alpha[k * H + h] = dot;
            if (sabs_a) sabs_a[k * H + h] = dabs;
        }
    return ORACLE_OK;
}

/* ---------------------------------------------------------------------------
 * Dense feature transform of a GCN layer (Section 2 lists GCN; its layer
 * multiplies the node features by a weight matrix before or after the
 * normalised aggregation): out = X Theta.
 * ------------------------------------------------------------------------- */

/* out[n, o] = sum_k x[n, k] * theta[k, o]; x [N, Fi], theta [Fi, Fo] fp32
 * (values as stored, e.g. bf16 widened exactly), out fp64 [N, Fo]; sabs
 * (nullable) = sum_k |x[n, k] theta[k, o]|. */
int oracle_dense_transform(const float *x, int64_t N, int64_t Fi, const float *theta, int64_t Fo, double *out,
                           double *sabs) {
    if (N < 0 || Fi < 0 || Fo < 0) return ORACLE_ERR_ARG;
    if (N * Fo > 0 && !out) return ORACLE_ERR_ARG;
    if (N * Fi > 0 && !x) return ORACLE_ERR_ARG;
    if (Fi * Fo > 0 && !theta) return ORACLE_ERR_ARG;
    if (!all_finite(x, N * Fi) || !all_finite(theta, Fi * Fo)) return ORACLE_ERR_NONFINITE;
    for (int64_t n = 0; n < N; ++n)
        for (int64_t o = 0; o < Fo; ++o) {
            double acc = 0.0, a = 0.0;
            for (int64_t k = 0; k < Fi; ++k) {
                const double t = (double)x[n * Fi + k] * (double)theta[k * Fo + o];
                acc += t;
                a += fabs(t);
            }
            out[n * Fo + o] = acc;
            if (sabs) sabs[n * Fo + o] = a;
        }
    return ORACLE_OK;
}

/* Gradient of oracle_gat_scores for g = dL/d e [E,H] (fp32):
 *   v = a_src[j,h] + a_dst[i,h],  de/dv = 1 if v >= 0 else slope,
 *   grad_src[j,h] += g[k,h] de/dv,  grad_dst[i,h] += g[k,h] de/dv   for k = (j -> i).
 * The branch is taken on the exact sum (its sign equals that of the
 * correctly rounded fp32 sum). grad_src, grad_dst fp64 [N,H]; sabs_* (nullable)
 * sum |terms|. */
int oracle_gat_scores_backward(const float *a_src, const float *a_dst, int64_t N, int64_t H,
                               const int64_t *edge_index, int64_t E, float slope, const float *g,
                               double *grad_src, double *grad_dst, double *sabs_src, double *sabs_dst) {
    if (N < 0 || H < 0 || E < 0) return ORACLE_ERR_ARG;
    if (N * H > 0 && (!a_src || !a_dst || !grad_src || !grad_dst)) return ORACLE_ERR_ARG;
    if (E * H > 0 && (!edge_index || !g)) return ORACLE_ERR_ARG;
    const int64_t *src = edge_index;
    const int64_t *dst = edge_index + E;
    if (check_index_range(src, E, N) || check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;
    if (!all_finite(a_src, N * H) || !all_finite(a_dst, N * H) || !all_finite(g, E * H) || !isfinite(slope))
        return ORACLE_ERR_NONFINITE;
    for (int64_t t = 0; t < N * H; ++t) {
        grad_src[t] = 0.0;
        grad_dst[t] = 0.0;
        if (sabs_src) sabs_src[t] = 0.0;
        if (sabs_dst) sabs_dst[t] = 0.0;
    }
    for (int64_t k = 0; k < E; ++k)
        for (int64_t h = 0; h < H; ++h) {
            const double v = (double)a_src[src[k] * H + h] + (double)a_dst[dst[k] * H + h];
            const double gv = (double)g[k * H + h] * (v >= 0.0 ? 1.0 : (double)slope);
            grad_src[src[k] * H + h] += gv;
            grad_dst[dst[k] * H + h] += gv;
            if (sabs_src) sabs_src[src[k] * H + h] += fabs(gv);
            if (sabs_dst) sabs_dst[dst[k] * H + h] += fabs(gv);
        }
    return ORACLE_OK;
}
