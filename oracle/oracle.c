/*
 * Oracle for the graph map-reduce hot path of tf_geometric (arXiv 2101.11552):
 * message aggregation (gather along edges, scale, reduce by target) and graph
 * pooling (reduce node vectors by graph).
 *
 * TEST INFRASTRUCTURE ONLY. This file is a plain, slow, obviously correct CPU
 * implementation used by the tests, by the smoke check and by the CPU-baseline
 * leg of the benchmark to judge the HIP library. The library never includes,
 * links or calls it, and it shares no code with the library.
 *
 * Conventions (the paper's Graph object, Sec. 2.1.1):
 *   - A graph is (x, edge_index, edge_weight). edge_index is COO of shape
 *     [2, E] (row 0 = source, row 1 = target); a positive A_ij is an edge from
 *     v_i to v_j. Messages flow source -> target and are reduced by target
 *     node index (the reduce key of Sec. 2.1.2).
 *   - Indices are int64 here; features and weights are float32; every sum is
 *     accumulated in double and rounded once at the end, so the oracle's
 *     error is far below the tolerance applied to the library.
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -fPIC -shared (see build.py).
 * With these flags every float expression below is evaluated in IEEE binary32
 * with one rounding per operation (x86-64 SSE, no contraction into FMA).
 *
 * Parity pins: every function is pinned in the CPU tests against values fixed
 * by the paper or by mathematics (dense brute force, closed forms, library
 * routines, invariants, the paper's worked BatchGraph example; the gradients
 * by central differences of the forward functions and the transpose
 * identity); see the test module for the oracle.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_OK = 0, ORC_ERR_INVALID_ARG = 1, ORC_ERR_INDEX_RANGE = 2, ORC_ERR_UNSORTED = 3 };
enum { ORC_SUM = 0, ORC_MEAN = 1, ORC_MAX = 2 };

/* Every source id in [0, n_src) and every target id in [0, n). */
int orc_check_edges(int64_t E, const int64_t *src, const int64_t *tgt, int64_t n_src, int64_t n)
{
    for (int64_t e = 0; e < E; ++e)
        if (src[e] < 0 || src[e] >= n_src || tgt[e] < 0 || tgt[e] >= n)
            return ORC_ERR_INDEX_RANGE;
    return ORC_OK;
}

/*
 * CSR by target (the reduce key of Sec. 2.1.2 is the target node index): a
 * stable counting sort of the edge list by target. rowptr[t] .. rowptr[t+1]
 * are the positions of the edges entering t (N + 1 entries); within a row the
 * edges keep their input order. perm[k] is the input edge id at position k,
 * col[k] its source id.
 */
void orc_csr_by_target(int64_t E, int64_t N, const int64_t *src, const int64_t *tgt,
                       int64_t *rowptr, int64_t *col, int64_t *perm)
{
    memset(rowptr, 0, (size_t)(N + 1) * sizeof(int64_t));
    for (int64_t e = 0; e < E; ++e)
        rowptr[tgt[e] + 1] += 1;
    for (int64_t t = 0; t < N; ++t)
        rowptr[t + 1] += rowptr[t];
    int64_t *cursor = (int64_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int64_t));
    memcpy(cursor, rowptr, (size_t)N * sizeof(int64_t));
    for (int64_t e = 0; e < E; ++e) {
        int64_t k = cursor[tgt[e]]++;
        perm[k] = e;
        col[k] = src[e];
    }
    free(cursor);
}

/*
 * GCN normalisation (GCN, cited by the paper in Sec. 2.2; cached per graph
 * structure in Sec. 3): A_hat = D^-1/2 (A + I) D^-1/2 written edge by edge.
 *   1. self-loops: edges (i, i) with weight 1 for i = 0..N-1 are appended
 *      after the E input edges (when add_loops), so E' = E + N;
 *   2. deg[t] = sum of the weights of the edges entering t (double, then
 *      rounded to float32);
 *   3. dinv[t] = 1 / sqrt(deg[t]) for deg[t] > 0, else 0 (float32: IEEE
 *      square root, then IEEE division);
 *   4. w_hat[e] = (dinv[src[e]] * w[e]) * dinv[tgt[e]] in float32.
 * w == NULL means unit weights. out_* hold E' entries; out_deg N entries.
 * Returns E'.
 */
int64_t orc_gcn_norm(int64_t E, int64_t N, const int64_t *src, const int64_t *tgt,
                     const float *w, int add_loops, int64_t *out_src, int64_t *out_tgt,
                     float *out_w, float *out_deg)
{
    int64_t Ep = E + (add_loops ? N : 0);
    float *wp = (float *)malloc((size_t)(Ep > 0 ? Ep : 1) * sizeof(float));
    for (int64_t e = 0; e < E; ++e) {
        out_src[e] = src[e];
        out_tgt[e] = tgt[e];
        wp[e] = w ? w[e] : 1.0f;
    }
    if (add_loops)
        for (int64_t i = 0; i < N; ++i) {
            out_src[E + i] = i;
            out_tgt[E + i] = i;
            wp[E + i] = 1.0f;
        }
    double *deg = (double *)calloc((size_t)(N > 0 ? N : 1), sizeof(double));
    float *dinv = (float *)malloc((size_t)(N > 0 ? N : 1) * sizeof(float));
    for (int64_t e = 0; e < Ep; ++e)
        deg[out_tgt[e]] += (double)wp[e];
    for (int64_t t = 0; t < N; ++t) {
        float d = (float)deg[t];
        if (out_deg)
            out_deg[t] = d;
        dinv[t] = d > 0.0f ? 1.0f / sqrtf(d) : 0.0f;
    }
    for (int64_t e = 0; e < Ep; ++e) {
        float a = dinv[out_src[e]] * wp[e];
        out_w[e] = a * dinv[out_tgt[e]];
    }
    free(wp);
    free(deg);
    free(dinv);
    return Ep;
}

/*
 * Message aggregation (Sec. 1, Fig. 1; reducer of Sec. 2.1.2):
 *   message m_e[c] = w_e[head(c)] * x[src_e, c], head(c) = c / (F / H)
 *   (w == NULL: unit weights; H = 1: one weight per edge)
 *   sum : out[t, c] = sum over edges e with tgt_e = t of m_e[c]
 *   mean: the sum divided by the number of edges entering t (0 if none)
 *   max : out[t, c] = max over those edges of fl32(w * x), the first edge in
 *         input order winning ties (+0 and -0 compare equal); arg[t, c] is the
 *         winning edge id; a target without edges gets value 0 and arg -1.
 * Sum and mean are written to out64 in double; max to outf / arg. scale[t, c]
 * receives the sum of |m_e[c]| (divided by the count for mean): the size of
 * the terms, which bounds the rounding error of any float32 summation order.
 * Rows not listed in `rows` (when rows != NULL) are not computed: row_slot[t]
 * maps a target to its output row (or -1) and outputs have n_rows rows.
 */
static int aggregate_impl(int64_t E, const int64_t *src, const int64_t *tgt, const float *w,
                          int64_t H, const float *x, int64_t ldx, int64_t F, int64_t N,
                          int reduce, const int64_t *row_slot, int64_t n_rows, double *out64,
                          float *outf, int64_t *arg, double *scale)
{
    if (H < 1 || F % H != 0)
        return ORC_ERR_INVALID_ARG;
    int64_t per_head = F / H;
    int64_t *cnt = (int64_t *)calloc((size_t)(n_rows > 0 ? n_rows : 1), sizeof(int64_t));
    char *seen = (char *)calloc((size_t)(n_rows > 0 ? n_rows : 1), 1);
    for (int64_t r = 0; r < n_rows * F; ++r) {
        if (out64) out64[r] = 0.0;
        if (outf) outf[r] = 0.0f;
        if (arg) arg[r] = -1;
        if (scale) scale[r] = 0.0;
    }
    for (int64_t e = 0; e < E; ++e) {
        int64_t t = tgt[e];
        int64_t r = row_slot ? row_slot[t] : t;
        if (r < 0)
            continue;
        cnt[r] += 1;
        const float *xs = x + src[e] * ldx;
        for (int64_t c = 0; c < F; ++c) {
            float wv = w ? w[e * H + c / per_head] : 1.0f;
            if (reduce == ORC_MAX) {
                float m = wv * xs[c];
                if (!seen[r] || m > outf[r * F + c]) {
                    outf[r * F + c] = m;
                    arg[r * F + c] = e;
                }
            } else {
                double m = (double)wv * (double)xs[c]; /* exact in double */
                out64[r * F + c] += m;
                if (scale) scale[r * F + c] += fabs(m);
            }
        }
        seen[r] = 1;
    }
    if (reduce == ORC_MEAN)
        for (int64_t r = 0; r < n_rows; ++r)
            for (int64_t c = 0; c < F; ++c) {
                out64[r * F + c] = cnt[r] ? out64[r * F + c] / (double)cnt[r] : 0.0;
                if (scale) scale[r * F + c] = cnt[r] ? scale[r * F + c] / (double)cnt[r] : 0.0;
            }
    free(cnt);
    free(seen);
    (void)N;
    return ORC_OK;
}

int orc_aggregate(int64_t E, const int64_t *src, const int64_t *tgt, const float *w, int64_t H,
                  const float *x, int64_t ldx, int64_t F, int64_t N, int reduce, double *out64,
                  float *outf, int64_t *arg, double *scale)
{
    return aggregate_impl(E, src, tgt, w, H, x, ldx, F, N, reduce, NULL, N, out64, outf, arg,
                          scale);
}

/* The same, for a sample of target rows only (row_slot[t] = output row or -1). */
int orc_aggregate_rows(int64_t E, const int64_t *src, const int64_t *tgt, const float *w,
                       int64_t H, const float *x, int64_t ldx, int64_t F, int64_t N, int reduce,
                       const int64_t *row_slot, int64_t n_rows, double *out64, float *outf,
                       int64_t *arg, double *scale)
{
    return aggregate_impl(E, src, tgt, w, H, x, ldx, F, N, reduce, row_slot, n_rows, out64, outf,
                          arg, scale);
}

/*
 * K-step propagation (SGC and APPNP, Sec. 2.2): Z_0 = x and
 *   Z_{k+1} = (1 - alpha) * A Z_k + alpha * h,   (A Z)[t] = sum over edges e -> t of w_e Z[src_e]
 * for k < K; out64 = Z_K, all in double (h may be NULL when alpha == 0).
 * scale receives the same recurrence on absolute values (|w|, |x|, |h|,
 * |1 - alpha|, |alpha|): the size of the terms behind every output.
 */
int orc_propagate(int64_t E, const int64_t *src, const int64_t *tgt, const float *w,
                  const float *x, int64_t ldx, int64_t N, int64_t F, int64_t K, double alpha,
                  const float *h, double *out64, double *scale)
{
    if (alpha != 0.0 && h == NULL)
        return ORC_ERR_INVALID_ARG;
    for (int64_t e = 0; e < E; ++e)
        if (src[e] < 0 || src[e] >= N || tgt[e] < 0 || tgt[e] >= N)
            return ORC_ERR_INDEX_RANGE;
    size_t n = (size_t)(N * F > 0 ? N * F : 1);
    double *z = (double *)malloc(n * sizeof(double)), *s = (double *)malloc(n * sizeof(double));
    double *y = (double *)malloc(n * sizeof(double)), *sy = (double *)malloc(n * sizeof(double));
    for (int64_t i = 0; i < N; ++i)
        for (int64_t c = 0; c < F; ++c) {
            z[i * F + c] = (double)x[i * ldx + c];
            s[i * F + c] = fabs((double)x[i * ldx + c]);
        }
    for (int64_t k = 0; k < K; ++k) {
        memset(y, 0, n * sizeof(double));
        memset(sy, 0, n * sizeof(double));
        for (int64_t e = 0; e < E; ++e) {
            double we = w ? (double)w[e] : 1.0;
            for (int64_t c = 0; c < F; ++c) {
                y[tgt[e] * F + c] += we * z[src[e] * F + c];
                sy[tgt[e] * F + c] += fabs(we) * s[src[e] * F + c];
            }
        }
        for (int64_t i = 0; i < N * F; ++i) {
            double hv = h ? (double)h[i] : 0.0;
            z[i] = (1.0 - alpha) * y[i] + alpha * hv;
            s[i] = fabs(1.0 - alpha) * sy[i] + fabs(alpha) * fabs(hv);
        }
    }
    memcpy(out64, z, (size_t)(N * F) * sizeof(double));
    if (scale)
        memcpy(scale, s, (size_t)(N * F) * sizeof(double));
    free(z); free(s); free(y); free(sy);
    return ORC_OK;
}

/*
 * Gradients of orc_aggregate for a loss L with dL/d out = dy ([N, F]):
 *   sum : dx[s, c] += w_e[head(c)] dy[t, c]            for every edge e = (s -> t)
 *         dw[e, k] += dy[t, c] x[s, c]                 over the columns c of head k
 *   mean: the same terms divided by the number of edges entering t
 *   max : only the terms of edge e at columns c where e is the argmax of (t, c)
 *         (arg: [N, F] edge ids from the forward max, -1 for empty targets)
 * dx64 [N_src, F] and dw64 [E, H] (either may be NULL) in double.
 */
int orc_aggregate_backward(int64_t E, const int64_t *src, const int64_t *tgt, const float *w,
                           int64_t H, const float *x, int64_t ldx, int64_t F, int64_t N_src,
                           int64_t N, int reduce, const float *dy, const int64_t *arg,
                           double *dx64, double *dw64)
{
    if (H < 1 || F % H != 0 || (reduce == ORC_MAX && arg == NULL))
        return ORC_ERR_INVALID_ARG;
    int64_t per_head = F / H;
    int64_t *cnt = (int64_t *)calloc((size_t)(N > 0 ? N : 1), sizeof(int64_t));
    for (int64_t e = 0; e < E; ++e)
        cnt[tgt[e]] += 1;
    if (dx64)
        memset(dx64, 0, (size_t)(N_src * F) * sizeof(double));
    if (dw64)
        memset(dw64, 0, (size_t)(E * H) * sizeof(double));
    for (int64_t e = 0; e < E; ++e) {
        int64_t s = src[e], t = tgt[e];
        for (int64_t c = 0; c < F; ++c) {
            if (reduce == ORC_MAX && arg[t * F + c] != e)
                continue;
            double g = (double)dy[t * F + c];
            if (reduce == ORC_MEAN)
                g /= (double)cnt[t];
            int64_t k = c / per_head;
            double wv = w ? (double)w[e * H + k] : 1.0;
            if (dx64)
                dx64[s * F + c] += wv * g;
            if (dw64)
                dw64[e * H + k] += g * (double)x[s * ldx + c];
        }
    }
    free(cnt);
    return ORC_OK;
}

/*
 * Gradient of orc_segment_softmax: with alpha = softmax(s) per (segment, head)
 * and dL/d alpha = da, dL/d s[e, h] = alpha[e, h] (da[e, h] - sum over the
 * segment of alpha * da). alpha, da: [E, H] float32; ds64 in double.
 */
int orc_segment_softmax_backward(int64_t E, int64_t H, const float *alpha, const float *da,
                                 const int64_t *seg, int64_t N, double *ds64)
{
    for (int64_t e = 0; e < E; ++e)
        if (seg[e] < 0 || seg[e] >= N)
            return ORC_ERR_INDEX_RANGE;
    double *dot = (double *)calloc((size_t)(N * H > 0 ? N * H : 1), sizeof(double));
    for (int64_t e = 0; e < E; ++e)
        for (int64_t h = 0; h < H; ++h)
            dot[seg[e] * H + h] += (double)alpha[e * H + h] * (double)da[e * H + h];
    for (int64_t e = 0; e < E; ++e)
        for (int64_t h = 0; h < H; ++h)
            ds64[e * H + h] = (double)alpha[e * H + h] *
                              ((double)da[e * H + h] - dot[seg[e] * H + h]);
    free(dot);
    return ORC_OK;
}

/*
 * Segment softmax, the map -> reduce -> map workflow of Fig. 5(a), Sec. 2.1.2:
 * for every segment t (the edges with seg[e] = t) and head h,
 *   alpha[e, h] = exp(s[e, h] - m) / sum over the segment of exp(s - m)
 * where m is the segment's maximum score (subtracting it leaves the result
 * unchanged and keeps exp finite). Scores are float32 [E, H]; the exponentials
 * and the sum are taken in double. Output in the input edge order.
 */
int orc_segment_softmax(int64_t E, int64_t H, const float *s, const int64_t *seg, int64_t N,
                        double *out64, float *outf)
{
    for (int64_t e = 0; e < E; ++e)
        if (seg[e] < 0 || seg[e] >= N)
            return ORC_ERR_INDEX_RANGE;
    float *m = (float *)malloc((size_t)(N * H > 0 ? N * H : 1) * sizeof(float));
    char *has = (char *)calloc((size_t)(N > 0 ? N : 1), 1);
    double *den = (double *)calloc((size_t)(N * H > 0 ? N * H : 1), sizeof(double));
    for (int64_t e = 0; e < E; ++e) {
        int64_t t = seg[e];
        for (int64_t h = 0; h < H; ++h)
            if (!has[t] || s[e * H + h] > m[t * H + h])
                m[t * H + h] = s[e * H + h];
        has[t] = 1;
    }
    for (int64_t e = 0; e < E; ++e)
        for (int64_t h = 0; h < H; ++h)
            den[seg[e] * H + h] += exp((double)s[e * H + h] - (double)m[seg[e] * H + h]);
    for (int64_t e = 0; e < E; ++e)
        for (int64_t h = 0; h < H; ++h) {
            int64_t i = seg[e] * H + h;
            double a = exp((double)s[e * H + h] - (double)m[i]) / den[i];
            if (out64) out64[e * H + h] = a;
            if (outf) outf[e * H + h] = (float)a;
        }
    free(m);
    free(has);
    free(den);
    return ORC_OK;
}

/*
 * Graph pooling by node_graph_index (Sec. 1 Fig. 2(a); BatchGraph, Sec. 2.1.1):
 * node n contributes x[n, :] to graph gi[n]. gi must be non-decreasing (the
 * sorted segment ids that BatchGraph produces) and inside [0, G).
 *   sum / mean (divided by the node count) in double; max in float32 with the
 *   lowest node id winning ties, arg = node id; a graph with no nodes gets 0
 *   and arg -1. scale as in orc_aggregate.
 */
int orc_segment_pool(int64_t Nb, int64_t F, int64_t ldx, const float *x, const int64_t *gi,
                     int64_t G, int reduce, double *out64, float *outf, int64_t *arg,
                     double *scale)
{
    for (int64_t n = 0; n < Nb; ++n) {
        if (gi[n] < 0 || gi[n] >= G)
            return ORC_ERR_INDEX_RANGE;
        if (n > 0 && gi[n] < gi[n - 1])
            return ORC_ERR_UNSORTED;
    }
    int64_t *cnt = (int64_t *)calloc((size_t)(G > 0 ? G : 1), sizeof(int64_t));
    for (int64_t r = 0; r < G * F; ++r) {
        if (out64) out64[r] = 0.0;
        if (outf) outf[r] = 0.0f;
        if (arg) arg[r] = -1;
        if (scale) scale[r] = 0.0;
    }
    for (int64_t n = 0; n < Nb; ++n) {
        int64_t g = gi[n];
        for (int64_t c = 0; c < F; ++c) {
            float v = x[n * ldx + c];
            if (reduce == ORC_MAX) {
                if (cnt[g] == 0 || v > outf[g * F + c]) {
                    outf[g * F + c] = v;
                    arg[g * F + c] = n;
                }
            } else {
                out64[g * F + c] += (double)v;
                if (scale) scale[g * F + c] += fabs((double)v);
            }
        }
        cnt[g] += 1;
    }
    if (reduce == ORC_MEAN)
        for (int64_t g = 0; g < G; ++g)
            for (int64_t c = 0; c < F; ++c) {
                out64[g * F + c] = cnt[g] ? out64[g * F + c] / (double)cnt[g] : 0.0;
                if (scale) scale[g * F + c] = cnt[g] ? scale[g * F + c] / (double)cnt[g] : 0.0;
            }
    free(cnt);
    return ORC_OK;
}

/*
 * Gradient of orc_segment_pool for dL/d out = dy ([G, F]): node n of graph g
 * receives dy[g, c] (sum), dy[g, c] / (nodes of g) (mean), or dy[g, c] only
 * where it was the argmax of (g, c) (max; arg as the forward returned it).
 * dx64: [Nb, F] in double.
 */
int orc_segment_pool_backward(int64_t Nb, int64_t F, const int64_t *gi, int64_t G, int reduce,
                              const float *dy, const int64_t *arg, double *dx64)
{
    for (int64_t n = 0; n < Nb; ++n) {
        if (gi[n] < 0 || gi[n] >= G)
            return ORC_ERR_INDEX_RANGE;
        if (n > 0 && gi[n] < gi[n - 1])
            return ORC_ERR_UNSORTED;
    }
    if (reduce == ORC_MAX && arg == NULL)
        return ORC_ERR_INVALID_ARG;
    int64_t *cnt = (int64_t *)calloc((size_t)(G > 0 ? G : 1), sizeof(int64_t));
    for (int64_t n = 0; n < Nb; ++n)
        cnt[gi[n]] += 1;
    for (int64_t n = 0; n < Nb; ++n) {
        int64_t g = gi[n];
        for (int64_t c = 0; c < F; ++c) {
            double v = (double)dy[g * F + c];
            if (reduce == ORC_MEAN)
                v /= (double)cnt[g];
            if (reduce == ORC_MAX && arg[g * F + c] != n)
                v = 0.0;
            dx64[n * F + c] = v;
        }
    }
    free(cnt);
    return ORC_OK;
}

/*
 * GAT attention scores, the first map of Fig. 5(a): with heads laid out as
 * h[n, k*D + d] (head k, dim d),
 *   a_s[n, k] = sum_d a_src[k, d] h[n, k, d],  a_d[n, k] = sum_d a_dst[k, d] h[n, k, d]
 *   s[e, k]   = LeakyReLU(a_s[src_e, k] + a_d[tgt_e, k]) with negative slope
 * all in double from the float32 inputs. scale[e, k] receives the size of the
 * terms: (sum |a_src h_src| + sum |a_dst h_dst|), times |slope| when s < 0.
 */
int orc_gat_scores(int64_t E, const int64_t *src, const int64_t *tgt, const float *h, int64_t N,
                   int64_t H, int64_t D, const float *a_src, const float *a_dst, float slope,
                   double *out64, double *scale)
{
    double *as = (double *)calloc((size_t)(N * H > 0 ? N * H : 1), sizeof(double));
    double *ad = (double *)calloc((size_t)(N * H > 0 ? N * H : 1), sizeof(double));
    double *as_abs = (double *)calloc((size_t)(N * H > 0 ? N * H : 1), sizeof(double));
    double *ad_abs = (double *)calloc((size_t)(N * H > 0 ? N * H : 1), sizeof(double));
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < H; ++k)
            for (int64_t d = 0; d < D; ++d) {
                double hv = (double)h[n * H * D + k * D + d];
                as[n * H + k] += (double)a_src[k * D + d] * hv;
                ad[n * H + k] += (double)a_dst[k * D + d] * hv;
                as_abs[n * H + k] += fabs((double)a_src[k * D + d] * hv);
                ad_abs[n * H + k] += fabs((double)a_dst[k * D + d] * hv);
            }
    for (int64_t e = 0; e < E; ++e) {
        if (src[e] < 0 || src[e] >= N || tgt[e] < 0 || tgt[e] >= N) {
            free(as); free(ad); free(as_abs); free(ad_abs);
            return ORC_ERR_INDEX_RANGE;
        }
        for (int64_t k = 0; k < H; ++k) {
            double z = as[src[e] * H + k] + ad[tgt[e] * H + k];
            double sz = as_abs[src[e] * H + k] + ad_abs[tgt[e] * H + k];
            int neg = z < 0.0;
            out64[e * H + k] = neg ? (double)slope * z : z;
            if (scale) scale[e * H + k] = neg ? fabs((double)slope) * sz : sz;
        }
    }
    free(as); free(ad); free(as_abs); free(ad_abs);
    return ORC_OK;
}

/*
 * A GAT attention layer after the projection: the map -> reduce -> map
 * workflow of Fig. 5(a) followed by the weighted message aggregation.
 *   1. scores s[e, k] as orc_gat_scores, rounded to float32 (the map's output);
 *   2. alpha[e, k] = softmax of s over the edges entering tgt_e (per head);
 *   3. out[t, k*D + d] = sum over the edges e entering t of alpha[e, k] h[src_e, k*D + d].
 * Steps 2 and 3 in double. alpha64 ([E, H], may be NULL) receives alpha;
 * scale[t, c] the sum of |alpha h| (the size of the terms).
 */
int orc_gat_layer(int64_t E, const int64_t *src, const int64_t *tgt, const float *h, int64_t N,
                  int64_t H, int64_t D, const float *a_src, const float *a_dst, float slope,
                  double *out64, double *alpha64, double *scale)
{
    int64_t F = H * D;
    double *s64 = (double *)malloc((size_t)(E * H > 0 ? E * H : 1) * sizeof(double));
    float *s32 = (float *)malloc((size_t)(E * H > 0 ? E * H : 1) * sizeof(float));
    double *al = (double *)malloc((size_t)(E * H > 0 ? E * H : 1) * sizeof(double));
    int rc = orc_gat_scores(E, src, tgt, h, N, H, D, a_src, a_dst, slope, s64, NULL);
    if (rc == ORC_OK) {
        for (int64_t i = 0; i < E * H; ++i)
            s32[i] = (float)s64[i];
        rc = orc_segment_softmax(E, H, s32, tgt, N, al, NULL);
    }
    if (rc == ORC_OK) {
        memset(out64, 0, (size_t)(N * F) * sizeof(double));
        if (scale)
            memset(scale, 0, (size_t)(N * F) * sizeof(double));
        for (int64_t e = 0; e < E; ++e)
            for (int64_t c = 0; c < F; ++c) {
                double m = al[e * H + c / D] * (double)h[src[e] * F + c];
                out64[tgt[e] * F + c] += m;
                if (scale)
                    scale[tgt[e] * F + c] += fabs(m);
            }
        if (alpha64)
            memcpy(alpha64, al, (size_t)(E * H) * sizeof(double));
    }
    free(s64);
    free(s32);
    free(al);
    return rc;
}

/*
 * Transformer-style attention (the GAT variant of the paper's library, Sec.
 * 4.2), scaled dot-product scores per edge and head:
 *   s[e, k] = scale * sum_d q[tgt_e, k*D + d] * key[src_e, k*D + d]
 * q: [N, H*D] (targets), key: [N_src, H*D] (sources); s64: [E, H] in double.
 */
int orc_dot_scores(int64_t E, const int64_t *src, const int64_t *tgt, const float *q,
                   const float *key, int64_t N, int64_t N_src, int64_t H, int64_t D,
                   double scale, double *s64)
{
    if (orc_check_edges(E, src, tgt, N_src, N) != ORC_OK)
        return ORC_ERR_INDEX_RANGE;
    int64_t F = H * D;
    for (int64_t e = 0; e < E; ++e)
        for (int64_t k = 0; k < H; ++k) {
            double acc = 0.0;
            for (int64_t d = 0; d < D; ++d)
                acc += (double)q[tgt[e] * F + k * D + d] * (double)key[src[e] * F + k * D + d];
            s64[e * H + k] = scale * acc;
        }
    return ORC_OK;
}

/*
 * The whole layer: scores as above (rounded to float32, as a float32 kernel
 * would hold them), the segment softmax per target and head, and
 * out[t, k*D + d] = sum over the edges e entering t of alpha[e, k] v[src_e, k*D + d].
 * v: [N_src, H*D]. out64 / scale: [N, H*D]; alpha64: [E, H] or NULL.
 */
int orc_dot_layer(int64_t E, const int64_t *src, const int64_t *tgt, const float *q,
                  const float *key, const float *v, int64_t N, int64_t N_src, int64_t H,
                  int64_t D, double scale, double *out64, double *alpha64, double *S)
{
    int64_t F = H * D;
    size_t n = (size_t)(E * H > 0 ? E * H : 1);
    double *s64 = (double *)malloc(n * sizeof(double));
    float *s32 = (float *)malloc(n * sizeof(float));
    double *al = (double *)malloc(n * sizeof(double));
    int rc = orc_dot_scores(E, src, tgt, q, key, N, N_src, H, D, scale, s64);
    if (rc == ORC_OK) {
        for (int64_t i = 0; i < E * H; ++i)
            s32[i] = (float)s64[i];
        rc = orc_segment_softmax(E, H, s32, tgt, N, al, NULL);
    }
    if (rc == ORC_OK) {
        memset(out64, 0, (size_t)(N * F) * sizeof(double));
        if (S)
            memset(S, 0, (size_t)(N * F) * sizeof(double));
        for (int64_t e = 0; e < E; ++e)
            for (int64_t c = 0; c < F; ++c) {
                double m = al[e * H + c / D] * (double)v[src[e] * F + c];
                out64[tgt[e] * F + c] += m;
                if (S)
                    S[tgt[e] * F + c] += fabs(m);
            }
        if (alpha64)
            memcpy(alpha64, al, (size_t)(E * H) * sizeof(double));
    }
    free(s64);
    free(s32);
    free(al);
    return rc;
}

/*
 * BatchGraph reindexing (Sec. 2.1.1, Fig. 4): node j of graph i becomes
 * j + offset[i], where offset[i] is the number of nodes in graphs 0..i-1.
 * offsets has G + 1 entries (the last one is the total node count).
 */
void orc_batch_offsets(int64_t G, const int64_t *sizes, int64_t *offsets)
{
    offsets[0] = 0;
    for (int64_t i = 0; i < G; ++i)
        offsets[i + 1] = offsets[i] + sizes[i];
}

/*
 * Combine G graphs into one BatchGraph: every local edge (u, v) of graph i
 * becomes (u + offset[i], v + offset[i]); edge lists are stacked in graph
 * order; graph_index[n] = i for the nodes of graph i. edge_counts[i] is the
 * number of edges of graph i, local_edges holds them consecutively as
 * [src..., tgt...] pairs per graph (2 * edge_counts[i] values each).
 */
void orc_batch_graphs(int64_t G, const int64_t *sizes, const int64_t *edge_counts,
                      const int64_t *local_edges, int64_t *out_src, int64_t *out_tgt,
                      int64_t *graph_index)
{
    int64_t off = 0, e_out = 0, pos = 0;
    for (int64_t i = 0; i < G; ++i) {
        const int64_t *ls = local_edges + pos;
        const int64_t *lt = local_edges + pos + edge_counts[i];
        for (int64_t e = 0; e < edge_counts[i]; ++e) {
            out_src[e_out] = ls[e] + off;
            out_tgt[e_out] = lt[e] + off;
            ++e_out;
        }
        for (int64_t j = 0; j < sizes[i]; ++j)
            graph_index[off + j] = i;
        pos += 2 * edge_counts[i];
        off += sizes[i];
    }
}
