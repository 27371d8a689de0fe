/*
 * Sanitizer driver for the oracle (test infrastructure): built together with
 * oracle/oracle.c under AddressSanitizer and UndefinedBehaviorSanitizer by
 * tests/test_sanitize.py. It calls every oracle entry point on small seeded
 * graphs (duplicates, self-loops, isolated and empty rows, degenerate sizes)
 * with exactly sized heap buffers, so that any read or write outside them,
 * any use of uninitialised or freed memory and any undefined arithmetic is
 * reported, and checks the invariants each result must satisfy. Exit 0 when
 * every check holds.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_degree(const int64_t *, int64_t, int64_t, int64_t *);
int oracle_coo_to_csr(const int64_t *, int64_t, int64_t, int64_t *, int64_t *, int64_t *);
int oracle_gcn_norm(const int64_t *, const double *, int64_t, int64_t, double *);
int oracle_propagate(const float *, int64_t, int64_t, const int64_t *, int64_t, const float *, const float *, int, int,
                     double *, int64_t *, double *);
int oracle_global_pool(const float *, int64_t, int64_t, const int64_t *, int64_t, int, double *, int64_t *, double *);
int oracle_propagate_backward(const float *, int64_t, int64_t, const int64_t *, int64_t, const float *, int, int,
                              const float *, const int64_t *, double *, double *, double *, double *);
int oracle_propagate_edge_backward(const float *, int64_t, int64_t, const int64_t *, int64_t, const float *, int, int,
                                   const float *, const int64_t *, double *, double *, double *, double *);
int oracle_gat_scores(const float *, const float *, int64_t, int64_t, const int64_t *, int64_t, float, double *);
int oracle_segment_softmax(const double *, int64_t, int64_t, const int64_t *, int64_t, double *);
int oracle_segment_softmax_backward(const float *, const float *, int64_t, int64_t, const int64_t *, int64_t, double *,
                                    double *);
int oracle_propagate_heads(const float *, int64_t, int64_t, int64_t, const int64_t *, int64_t, const float *, double *,
                           double *);
int oracle_propagate_heads_backward(const float *, int64_t, int64_t, int64_t, const int64_t *, int64_t, const float *,
                                    const float *, double *, double *, double *, double *);
int oracle_dense_transform(const float *, int64_t, int64_t, const float *, int64_t, double *, double *);
int oracle_gat_scores_backward(const float *, const float *, int64_t, int64_t, const int64_t *, int64_t, float,
                               const float *, double *, double *, double *, double *);

static int failures = 0;
#define CHECK(cond, ...)                                  \
    do {                                                  \
        if (!(cond)) {                                    \
            fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
            fprintf(stderr, __VA_ARGS__);                 \
            fprintf(stderr, "\n");                        \
            ++failures;                                   \
        }                                                 \
    } while (0)

static uint64_t rng_state;
static uint64_t next_u64(void) { /* splitmix64 */
    uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}
static int64_t below(int64_t n) { return n > 0 ? (int64_t)(next_u64() % (uint64_t)n) : 0; }
static float unit(void) { return (float)((double)(next_u64() >> 11) / 9007199254740992.0 * 2.0 - 1.0); }

/* exactly sized buffers: zero-size requests still get a unique pointer */
static void *xmalloc(size_t n) {
    void *p = malloc(n ? n : 1);
    if (!p) abort();
    return p;
}

static void run_graph(int64_t N, int64_t E, int64_t F, int64_t H) {
    int64_t *ei = xmalloc(sizeof(int64_t) * 2 * E);
    for (int64_t k = 0; k < E; ++k) {
        ei[k] = below(N);
        ei[E + k] = (k % 7 == 3 && k > 0) ? ei[E + k - 1] : below(N); /* duplicates and repeated targets */
    }
    float *x = xmalloc(sizeof(float) * N * F), *w = xmalloc(sizeof(float) * E), *g = xmalloc(sizeof(float) * N * F);
    float *ea = xmalloc(sizeof(float) * E * F);
    for (int64_t i = 0; i < N * F; ++i) x[i] = unit(), g[i] = unit();
    for (int64_t k = 0; k < E; ++k) w[k] = unit();
    for (int64_t i = 0; i < E * F; ++i) ea[i] = unit();

    /* degree and CSR */
    int64_t *deg = xmalloc(sizeof(int64_t) * N);
    CHECK(oracle_degree(ei, E, N, deg) == 0, "degree");
    int64_t total = 0;
    for (int64_t i = 0; i < N; ++i) total += deg[i];
    CHECK(total == E, "sum of degrees %lld != E %lld", (long long)total, (long long)E);
    int64_t *rp = xmalloc(sizeof(int64_t) * (N + 1)), *col = xmalloc(sizeof(int64_t) * E), *perm = xmalloc(sizeof(int64_t) * E);
    CHECK(oracle_coo_to_csr(ei, E, N, rp, col, perm) == 0, "coo_to_csr");
    CHECK(rp[0] == 0 && rp[N] == E, "rowptr ends");
    char *seen = xmalloc((size_t)E);
    memset(seen, 0, (size_t)E);
    for (int64_t i = 0; i < N; ++i) {
        CHECK(rp[i + 1] - rp[i] == deg[i], "row %lld length", (long long)i);
        for (int64_t p = rp[i]; p < rp[i + 1]; ++p) {
            CHECK(perm[p] >= 0 && perm[p] < E && !seen[perm[p]], "perm");
            if (perm[p] >= 0 && perm[p] < E) seen[perm[p]] = 1;
            CHECK(ei[E + perm[p]] == i && ei[perm[p]] == col[p], "slot %lld", (long long)p);
            CHECK(p == rp[i] || perm[p] > perm[p - 1], "stable order");
        }
    }

    /* gcn_norm, unweighted and weighted (positive weights keep every degree > 0) */
    double *norm = xmalloc(sizeof(double) * E), *wd = xmalloc(sizeof(double) * E);
    for (int64_t k = 0; k < E; ++k) wd[k] = fabs((double)w[k]) + 0.5;
    CHECK(oracle_gcn_norm(ei, NULL, E, N, norm) == 0, "gcn_norm");
    for (int64_t k = 0; k < E; ++k)
        CHECK(fabs(norm[k] - 1.0 / sqrt((double)deg[ei[k]] * (double)deg[ei[E + k]])) <= 1e-12 || deg[ei[k]] == 0,
              "gcn_norm value");
    CHECK(oracle_gcn_norm(ei, wd, E, N, norm) == 0, "gcn_norm weighted");

    /* propagate: every message and aggregation; sum = mean * deg; max >= every message */
    double *out = xmalloc(sizeof(double) * N * F), *out2 = xmalloc(sizeof(double) * N * F);
    double *sabs = xmalloc(sizeof(double) * N * F);
    int64_t *arg = xmalloc(sizeof(int64_t) * N * F);
    for (int msg = 0; msg <= 4; ++msg) {
        const float *wm = msg == 0 ? w : NULL;
        const float *em = msg >= 2 ? ea : NULL;
        CHECK(oracle_propagate(x, N, F, ei, E, wm, em, msg, 0, out, NULL, sabs) == 0, "propagate sum msg %d", msg);
        CHECK(oracle_propagate(x, N, F, ei, E, wm, em, msg, 1, out2, NULL, sabs) == 0, "propagate mean msg %d", msg);
        for (int64_t i = 0; i < N; ++i)
            for (int64_t f = 0; f < F; ++f)
                CHECK(fabs(out2[i * F + f] * (double)deg[i] - out[i * F + f]) <= 1e-9 * (1.0 + fabs(out[i * F + f])),
                      "sum = mean * deg");
        CHECK(oracle_propagate(x, N, F, ei, E, wm, em, msg, 2, out, arg, sabs) == 0, "propagate max msg %d", msg);
        for (int64_t i = 0; i < N * F; ++i) CHECK(arg[i] >= 0 && arg[i] <= E, "argmax range");
        for (int64_t i = 0; i < N; ++i)
            for (int64_t f = 0; f < F; ++f)
                CHECK((deg[i] == 0) == (arg[i * F + f] == E), "empty row <=> sentinel");
    }

    /* propagate backward for every aggregation, and the edge-message backward */
    double *gx = xmalloc(sizeof(double) * N * F), *gw = xmalloc(sizeof(double) * E), *sx = xmalloc(sizeof(double) * N * F),
           *sw = xmalloc(sizeof(double) * E), *ge = xmalloc(sizeof(double) * E * F), *se = xmalloc(sizeof(double) * E * F);
    CHECK(oracle_propagate(x, N, F, ei, E, w, NULL, 0, 2, out, arg, sabs) == 0, "max for backward");
    for (int aggr = 0; aggr <= 2; ++aggr) {
        CHECK(oracle_propagate_backward(x, N, F, ei, E, w, 0, aggr, g, aggr == 2 ? arg : NULL, gx, gw, sx, sw) == 0,
              "propagate_backward aggr %d", aggr);
        CHECK(oracle_propagate_backward(x, N, F, ei, E, NULL, 1, aggr, g, NULL, gx, NULL, sx, NULL) == 0 || aggr == 2,
              "propagate_backward diff aggr %d", aggr);
    }
    for (int msg = 2; msg <= 4; ++msg) {
        CHECK(oracle_propagate(x, N, F, ei, E, NULL, ea, msg, 2, out, arg, sabs) == 0, "edge max");
        for (int aggr = 0; aggr <= 2; ++aggr)
            CHECK(oracle_propagate_edge_backward(x, N, F, ei, E, ea, msg, aggr, g, aggr == 2 ? arg : NULL, gx, ge, sx,
                                                 se) == 0,
                  "edge backward msg %d aggr %d", msg, aggr);
    }

    /* global pooling over a sorted batch vector with an empty graph */
    const int64_t B = N > 2 ? 3 : 1;
    int64_t *batch = xmalloc(sizeof(int64_t) * N);
    for (int64_t i = 0; i < N; ++i) batch[i] = (B == 3 && i >= N / 2) ? 2 : 0; /* graph 1 empty */
    double *pool = xmalloc(sizeof(double) * B * F), *psabs = xmalloc(sizeof(double) * B * F);
    int64_t *parg = xmalloc(sizeof(int64_t) * B * F);
    for (int aggr = 0; aggr <= 2; ++aggr)
        CHECK(oracle_global_pool(x, N, F, batch, B, aggr, pool, aggr == 2 ? parg : NULL, psabs) == 0, "pool %d", aggr);
    if (B == 3)
        for (int64_t f = 0; f < F; ++f) CHECK(pool[F + f] == 0.0 && parg[F + f] == N, "empty graph pools to 0 / N");

    /* attention: scores, softmax (rows sum to 1), its backward, heads and their gradients */
    if (F % H == 0) {
        const int64_t C = F / H;
        float *as = xmalloc(sizeof(float) * N * H), *ad = xmalloc(sizeof(float) * N * H);
        for (int64_t i = 0; i < N * H; ++i) as[i] = unit(), ad[i] = unit();
        double *sc = xmalloc(sizeof(double) * E * H), *al = xmalloc(sizeof(double) * E * H);
        CHECK(oracle_gat_scores(as, ad, N, H, ei, E, 0.2f, sc) == 0, "gat_scores");
        CHECK(oracle_segment_softmax(sc, E, H, ei, N, al) == 0, "segment_softmax");
        double *rs = xmalloc(sizeof(double) * N * H);
        for (int64_t i = 0; i < N * H; ++i) rs[i] = 0.0;
        for (int64_t k = 0; k < E; ++k)
            for (int64_t h = 0; h < H; ++h) rs[ei[E + k] * H + h] += al[k * H + h];
        for (int64_t i = 0; i < N; ++i)
            for (int64_t h = 0; h < H; ++h) CHECK(deg[i] == 0 || fabs(rs[i * H + h] - 1.0) < 1e-12, "softmax sums to 1");
        float *alf = xmalloc(sizeof(float) * E * H), *ge2 = xmalloc(sizeof(float) * E * H);
        for (int64_t i = 0; i < E * H; ++i) alf[i] = (float)al[i], ge2[i] = unit();
        double *gs = xmalloc(sizeof(double) * E * H), *ss = xmalloc(sizeof(double) * E * H);
        CHECK(oracle_segment_softmax_backward(alf, ge2, E, H, ei, N, gs, ss) == 0, "softmax backward");
        CHECK(oracle_propagate_heads(x, N, H, C, ei, E, alf, out, sabs) == 0, "propagate_heads");
        double *ga = xmalloc(sizeof(double) * E * H), *sa = xmalloc(sizeof(double) * E * H);
        CHECK(oracle_propagate_heads_backward(x, N, H, C, ei, E, alf, g, gx, ga, sx, sa) == 0, "heads backward");
        double *g1 = xmalloc(sizeof(double) * N * H), *g2 = xmalloc(sizeof(double) * N * H),
               *s1 = xmalloc(sizeof(double) * N * H), *s2 = xmalloc(sizeof(double) * N * H);
        CHECK(oracle_gat_scores_backward(as, ad, N, H, ei, E, 0.2f, ge2, g1, g2, s1, s2) == 0, "scores backward");
        free(as), free(ad), free(sc), free(al), free(rs), free(alf), free(ge2), free(gs), free(ss), free(ga), free(sa);
        free(g1), free(g2), free(s1), free(s2);
    }

    /* dense transform against a plain triple loop */
    const int64_t Fo = 5;
    float *th = xmalloc(sizeof(float) * F * Fo);
    for (int64_t i = 0; i < F * Fo; ++i) th[i] = unit();
    double *dt = xmalloc(sizeof(double) * N * Fo), *ds = xmalloc(sizeof(double) * N * Fo);
    CHECK(oracle_dense_transform(x, N, F, th, Fo, dt, ds) == 0, "dense_transform");
    for (int64_t i = 0; i < N; ++i)
        for (int64_t o = 0; o < Fo; ++o) {
            double r = 0.0;
            for (int64_t f = 0; f < F; ++f) r += (double)x[i * F + f] * (double)th[f * Fo + o];
            CHECK(fabs(dt[i * Fo + o] - r) <= 1e-12 * (1.0 + ds[i * Fo + o]), "dense value");
        }

    free(ei), free(x), free(w), free(g), free(ea), free(deg), free(rp), free(col), free(perm), free(seen), free(norm);
    free(wd), free(out), free(out2), free(sabs), free(arg), free(gx), free(gw), free(sx), free(sw), free(ge), free(se);
    free(batch), free(pool), free(psabs), free(parg), free(th), free(dt), free(ds);
}

int main(void) {
    rng_state = 12345;
    /* (N, E, F, H): a single node, graphs without edges, duplicates and
     * isolated rows, odd widths, several heads */
    const int64_t shapes[][4] = {{1, 0, 1, 1}, {1, 3, 2, 1}, {5, 0, 4, 2}, {7, 40, 3, 1},
                                 {50, 600, 16, 4}, {64, 2000, 8, 8}, {300, 100, 6, 3}};
    for (size_t s = 0; s < sizeof(shapes) / sizeof(shapes[0]); ++s)
        run_graph(shapes[s][0], shapes[s][1], shapes[s][2], shapes[s][3]);

    /* argument errors are returned, not faulted on */
    int64_t ei[2] = {0, 0};
    int64_t d = 0;
    CHECK(oracle_degree(ei, -1, 1, &d) != 0, "negative E");
    CHECK(oracle_degree(NULL, 1, 1, &d) != 0, "NULL edge_index");
    int64_t bad[2] = {0, 5};
    CHECK(oracle_degree(bad, 1, 2, &d) != 0, "target out of range");
    float nan_x[1] = {NAN};
    double o1[1], s1[1];
    CHECK(oracle_propagate(nan_x, 1, 1, ei, 1, NULL, NULL, 0, 0, o1, NULL, s1) != 0, "non-finite input");
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("oracle under ASan/UBSan: every entry point, every check passed\n");
    return 0;
}
