/*
 * Drives every function of the oracle (oracle/oracle.c) over small seeded
 * inputs and the degenerate cases (no edges, one node, empty rows and
 * graphs, several heads, rectangular graphs, ties), with every buffer
 * allocated at exactly the size the function's contract states, so that an
 * AddressSanitizer / UndefinedBehaviorSanitizer build reports any access
 * outside it. Test infrastructure: built and run by tests/test_sanitize.py.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int orc_check_edges(int64_t, const int64_t *, const int64_t *, int64_t, int64_t);
void orc_csr_by_target(int64_t, int64_t, const int64_t *, const int64_t *, int64_t *, int64_t *,
                       int64_t *);
int64_t orc_gcn_norm(int64_t, int64_t, const int64_t *, const int64_t *, const float *, int,
                     int64_t *, int64_t *, float *, float *);
int orc_aggregate(int64_t, const int64_t *, const int64_t *, const float *, int64_t, const float *,
                  int64_t, int64_t, int64_t, int, double *, float *, int64_t *, double *);
int orc_aggregate_rows(int64_t, const int64_t *, const int64_t *, const float *, int64_t,
                       const float *, int64_t, int64_t, int64_t, int, const int64_t *, int64_t,
                       double *, float *, int64_t *, double *);
int orc_propagate(int64_t, const int64_t *, const int64_t *, const float *, const float *, int64_t,
                  int64_t, int64_t, int64_t, double, const float *, double *, double *);
int orc_aggregate_backward(int64_t, const int64_t *, const int64_t *, const float *, int64_t,
                           const float *, int64_t, int64_t, int64_t, int64_t, int, const float *,
                           const int64_t *, double *, double *);
int orc_segment_softmax_backward(int64_t, int64_t, const float *, const float *, const int64_t *,
                                 int64_t, double *);
int orc_segment_softmax(int64_t, int64_t, const float *, const int64_t *, int64_t, double *,
                        float *);
int orc_segment_pool(int64_t, int64_t, int64_t, const float *, const int64_t *, int64_t, int,
                     double *, float *, int64_t *, double *);
int orc_segment_pool_backward(int64_t, int64_t, const int64_t *, int64_t, int, const float *,
                              const int64_t *, double *);
int orc_gat_scores(int64_t, const int64_t *, const int64_t *, const float *, int64_t, int64_t,
                   int64_t, const float *, const float *, float, double *, double *);
int orc_gat_layer(int64_t, const int64_t *, const int64_t *, const float *, int64_t, int64_t,
                  int64_t, const float *, const float *, float, double *, double *, double *);
int orc_dot_scores(int64_t, const int64_t *, const int64_t *, const float *, const float *, int64_t,
                   int64_t, int64_t, int64_t, double, double *);
int orc_dot_layer(int64_t, const int64_t *, const int64_t *, const float *, const float *,
                  const float *, int64_t, int64_t, int64_t, int64_t, double, double *, double *,
                  double *);
void orc_batch_offsets(int64_t, const int64_t *, int64_t *);
void orc_batch_graphs(int64_t, const int64_t *, const int64_t *, const int64_t *, int64_t *,
                      int64_t *, int64_t *);

static uint64_t rng_state = 88172645463325252ull;
static uint64_t next_u64(void)
{
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 7;
    rng_state ^= rng_state << 17;
    return rng_state;
}
static int64_t below(int64_t n) { return n > 0 ? (int64_t)(next_u64() % (uint64_t)n) : 0; }
static float normal(void)
{
    double u = ((double)(next_u64() >> 11) + 0.5) / 9007199254740992.0;
    double v = ((double)(next_u64() >> 11) + 0.5) / 9007199254740992.0;
    return (float)(sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v));
}
/* exactly n elements (at least one byte allocated so that malloc(0) is not NULL) */
static void *alloc(size_t n, size_t size) { return malloc(n * size > 0 ? n * size : 1); }
static float *floats(int64_t n)
{
    float *p = alloc((size_t)n, sizeof(float));
    for (int64_t i = 0; i < n; ++i)
        p[i] = normal();
    return p;
}

static int failures = 0;
#define CHECK(cond)                                                        \
    do {                                                                   \
        if (!(cond)) {                                                     \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
            ++failures;                                                    \
        }                                                                  \
    } while (0)

static void graph_case(int64_t N, int64_t N_src, int64_t E, int64_t H, int64_t D, int hub)
{
    const int64_t F = H * D, ldx = F + 3;
    int64_t *src = alloc((size_t)E, sizeof(int64_t)), *tgt = alloc((size_t)E, sizeof(int64_t));
    for (int64_t e = 0; e < E; ++e) {
        src[e] = below(N_src);
        tgt[e] = (hub && e % 3 == 0) ? 0 : below(N);
    }
    CHECK(orc_check_edges(E, src, tgt, N_src, N) == 0);
    int64_t *rowptr = alloc((size_t)N + 1, sizeof(int64_t));
    int64_t *col = alloc((size_t)E, sizeof(int64_t)), *perm = alloc((size_t)E, sizeof(int64_t));
    orc_csr_by_target(E, N, src, tgt, rowptr, col, perm);
    CHECK(rowptr[N] == E);
    float *w = floats(E * H), *x = floats(N_src * ldx), *dy = floats(N * F);
    for (int64_t r = 0; r < 3; ++r) {
        double *o64 = alloc((size_t)(N * F), sizeof(double)), *sc = alloc((size_t)(N * F), sizeof(double));
        float *of = alloc((size_t)(N * F), sizeof(float));
        int64_t *arg = alloc((size_t)(N * F), sizeof(int64_t));
        CHECK(orc_aggregate(E, src, tgt, w, H, x, ldx, F, N, (int)r, o64, of, arg, sc) == 0);
        int64_t n_rows = N / 2 + 1;
        int64_t *slot = alloc((size_t)N, sizeof(int64_t));
        for (int64_t t = 0; t < N; ++t)
            slot[t] = t < n_rows ? t : -1;
        CHECK(orc_aggregate_rows(E, src, tgt, w, H, x, ldx, F, N, (int)r, slot, n_rows, o64, of,
                                 arg, sc) == 0);
        double *dx = alloc((size_t)(N_src * F), sizeof(double)), *dw = alloc((size_t)(E * H), sizeof(double));
        CHECK(orc_aggregate_backward(E, src, tgt, w, H, x, ldx, F, N_src, N, (int)r, dy,
                                     r == 2 ? arg : NULL, dx, dw) == 0);
        free(o64), free(sc), free(of), free(arg), free(slot), free(dx), free(dw);
    }
    /* attention over the edge list */
    float *s = floats(E * H), *al = alloc((size_t)(E * H), sizeof(float));
    double *a64 = alloc((size_t)(E * H), sizeof(double)), *ds = alloc((size_t)(E * H), sizeof(double));
    CHECK(orc_segment_softmax(E, H, s, tgt, N, a64, al) == 0);
    CHECK(orc_segment_softmax_backward(E, H, al, s, tgt, N, ds) == 0);
    if (N == N_src) {
        float *h = floats(N * F), *as = floats(H * D), *ad = floats(H * D);
        double *g64 = alloc((size_t)(E * H), sizeof(double)), *gs = alloc((size_t)(E * H), sizeof(double));
        CHECK(orc_gat_scores(E, src, tgt, h, N, H, D, as, ad, 0.2f, g64, gs) == 0);
        double *l64 = alloc((size_t)(N * F), sizeof(double)), *ls = alloc((size_t)(N * F), sizeof(double));
        CHECK(orc_gat_layer(E, src, tgt, h, N, H, D, as, ad, 0.2f, l64, a64, ls) == 0);
        /* normalisation with and without loops, then propagation */
        for (int loops = 0; loops < 2; ++loops) {
            const int64_t Ep = E + (loops ? N : 0);
            int64_t *os = alloc((size_t)Ep, sizeof(int64_t)), *ot = alloc((size_t)Ep, sizeof(int64_t));
            float *ow = alloc((size_t)Ep, sizeof(float)), *deg = alloc((size_t)N, sizeof(float));
            CHECK(orc_gcn_norm(E, N, src, tgt, loops ? NULL : w, loops, os, ot, ow, deg) == Ep);
            double *p64 = alloc((size_t)(N * F), sizeof(double)), *ps = alloc((size_t)(N * F), sizeof(double));
            CHECK(orc_propagate(Ep, os, ot, ow, x, ldx, N, F, 3, 0.1, h, p64, ps) == 0);
            free(os), free(ot), free(ow), free(deg), free(p64), free(ps);
        }
        free(h), free(as), free(ad), free(g64), free(gs), free(l64), free(ls);
    }
    float *q = floats(N * F), *k = floats(N_src * F), *v = floats(N_src * F);
    double *s64 = alloc((size_t)(E * H), sizeof(double)), *d64 = alloc((size_t)(N * F), sizeof(double));
    double *dS = alloc((size_t)(N * F), sizeof(double));
    CHECK(orc_dot_scores(E, src, tgt, q, k, N, N_src, H, D, 0.25, s64) == 0);
    CHECK(orc_dot_layer(E, src, tgt, q, k, v, N, N_src, H, D, 0.25, d64, a64, dS) == 0);
    free(q), free(k), free(v), free(s64), free(d64), free(dS);
    free(s), free(al), free(a64), free(ds);
    free(src), free(tgt), free(rowptr), free(col), free(perm), free(w), free(x), free(dy);
}

static void pool_case(int64_t G, int64_t F)
{
    int64_t *sizes = alloc((size_t)G, sizeof(int64_t)), *counts = alloc((size_t)G, sizeof(int64_t));
    int64_t Nb = 0, E = 0;
    for (int64_t g = 0; g < G; ++g) {
        sizes[g] = g % 4 == 1 ? 0 : 1 + below(9); /* some empty graphs */
        counts[g] = sizes[g] ? below(2 * sizes[g] + 1) : 0;
        Nb += sizes[g];
        E += counts[g];
    }
    int64_t *off = alloc((size_t)G + 1, sizeof(int64_t));
    orc_batch_offsets(G, sizes, off);
    CHECK(off[G] == Nb);
    int64_t *local = alloc((size_t)(2 * E), sizeof(int64_t));
    for (int64_t g = 0, e = 0; g < G; ++g)
        for (int64_t j = 0; j < counts[g]; ++j, ++e) {
            local[e] = below(sizes[g]);
            local[E + e] = below(sizes[g]);
        }
    /* stacked local lists: graph 0's (src row, then tgt row), then graph 1's, ... */
    int64_t *stacked = alloc((size_t)(2 * E), sizeof(int64_t));
    for (int64_t g = 0, e = 0, o = 0; g < G; ++g) {
        for (int64_t j = 0; j < counts[g]; ++j)
            stacked[o + j] = local[e + j];
        for (int64_t j = 0; j < counts[g]; ++j)
            stacked[o + counts[g] + j] = local[E + e + j];
        o += 2 * counts[g];
        e += counts[g];
    }
    int64_t *bs = alloc((size_t)E, sizeof(int64_t)), *bt = alloc((size_t)E, sizeof(int64_t));
    int64_t *gi = alloc((size_t)Nb, sizeof(int64_t));
    orc_batch_graphs(G, sizes, counts, stacked, bs, bt, gi);
    float *x = floats(Nb * F), *dy = floats(G * F);
    for (int r = 0; r < 3; ++r) {
        double *o64 = alloc((size_t)(G * F), sizeof(double)), *sc = alloc((size_t)(G * F), sizeof(double));
        float *of = alloc((size_t)(G * F), sizeof(float));
        int64_t *arg = alloc((size_t)(G * F), sizeof(int64_t));
        double *dx = alloc((size_t)(Nb * F), sizeof(double));
        CHECK(orc_segment_pool(Nb, F, F, x, gi, G, r, o64, of, arg, sc) == 0);
        CHECK(orc_segment_pool_backward(Nb, F, gi, G, r, dy, r == 2 ? arg : NULL, dx) == 0);
        free(o64), free(sc), free(of), free(arg), free(dx);
    }
    free(sizes), free(counts), free(off), free(local), free(stacked), free(bs), free(bt), free(gi);
    free(x), free(dy);
}

int main(void)
{
    graph_case(1, 1, 0, 1, 1, 0);      /* one node, no edges */
    graph_case(1, 1, 7, 1, 3, 0);      /* one node, loops only */
    graph_case(50, 50, 0, 2, 4, 0);    /* no edges: every row empty */
    graph_case(40, 40, 300, 1, 5, 1);  /* a hub row */
    graph_case(60, 25, 500, 3, 2, 0);  /* rectangular, three heads */
    graph_case(200, 200, 3000, 4, 4, 1);
    pool_case(1, 3);
    pool_case(17, 8);
    pool_case(200, 5);
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("oracle driver ok\n");
    return 0;
}
