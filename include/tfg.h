/*
 * tfg.h — C ABI of the MI355X (gfx950) graph map-reduce hot path.
 *
 * The operations are the two aggregation types of tf_geometric (arXiv
 * 2101.11552, Sec. 1): message aggregation — gather source-node features
 * along the edges, scale them by edge weights, reduce them into the target
 * node — and graph pooling — reduce the node vectors of each graph of a
 * BatchGraph into one vector per graph. Around them sit the GCN normalisation
 * the paper caches per graph (Sec. 3) and the map -> reduce -> map softmax
 * workflow for attention scores (Sec. 2.1.2, Fig. 5). Built on them: fused
 * attention layers (the additive GAT score and the Transformer-style scaled
 * dot product of Sec. 4.2), multi-step propagation (SGC, APPNP; Sec. 2.2),
 * BatchGraph construction (Sec. 2.1.1, 2.1.3), and the gradients of the
 * aggregation, the softmax and the pooling for training through graphs built
 * inside a model.
 *
 * Conventions shared by every call
 * --------------------------------
 * Graphs are the paper's Graph object (Sec. 2.1.1): node features x, and the
 * adjacency matrix in COO form: edge_index of shape [2, E], row-major, row 0
 * the source ids and row 1 the target ids (edge e goes from edge_index[e] to
 * edge_index[E + e]); edge_weight [E] (or [E, H], one weight per head).
 * Messages flow source -> target and are reduced by the target id, the reduce
 * key of the paper's reducer (Sec. 2.1.2).
 *
 * Index arrays are int32 (TFG_I32) or int64 (TFG_I64). Node counts, edge
 * counts (including appended self-loops), E * H and feature counts must stay
 * below 2^31 - 2^20 = 2,146,435,072 (else TFG_ERR_TOO_LARGE): positions are
 * 32-bit inside the kernels, with a margin for the strides that step through
 * them. Floating-point data is
 * float32, row-major; a feature matrix has a leading dimension ldx >= F (in
 * elements). Outputs are dense row-major with leading dimension F.
 *
 * Memory: every pointer except `tfg_graph*` handles is DEVICE memory owned by
 * the caller. The library never allocates device memory: callers query the
 * workspace size (tfg_*_ws_bytes) and pass a buffer of at least that many
 * bytes (256-byte aligned). Inputs are only read; outputs must not overlap
 * inputs. Host allocations: the small tfg_graph struct, and 32 bytes of
 * pinned host memory per calling thread (allocated on its first synchronising
 * call, kept until the process ends) into which counters are read back.
 *
 * Streams: every call enqueues its kernels on `stream` (a hipStream_t; NULL is
 * the null stream) and returns without waiting, except where a call is
 * documented to synchronise. Buffers must stay valid until the stream work is
 * done.
 *
 * Errors: calls return a tfg_status. Argument errors (null pointers, negative
 * sizes, bad enums, a workspace that is too small) are detected on the host
 * before anything is enqueued. Index errors (an id outside its range) and an
 * unsorted graph index are detected on the device: kernels clamp such ids so
 * they never access memory out of bounds, record the error in a device flag,
 * and calls that synchronise report it. tfg_last_error() gives a message for
 * the last failing call of the calling thread.
 *
 * Determinism: for fixed inputs, every output is bitwise reproducible from run
 * to run (no floating-point atomics anywhere).
 */
#ifndef TFG_H
#define TFG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TFG_ABI_VERSION 1

typedef enum {
    TFG_OK = 0,
    TFG_ERR_INVALID_ARG = 1, /* null pointer, negative size, bad enum, F % H != 0, mismatch with a graph */
    TFG_ERR_INDEX_RANGE = 2, /* an edge id outside [0, N_src) / [0, N), a graph id outside [0, G) */
    TFG_ERR_UNSORTED = 3,    /* graph_index is not non-decreasing */
    TFG_ERR_TOO_LARGE = 4,   /* a count is not below 2^31 - 2^20 (32-bit internal positions) */
    TFG_ERR_WORKSPACE = 5,   /* buffer smaller than the size the matching query returned, or not 256-byte aligned */
    TFG_ERR_HIP = 6          /* the HIP runtime reported an error; see tfg_last_error() */
} tfg_status;

typedef enum { TFG_SUM = 0, TFG_MEAN = 1, TFG_MAX = 2 } tfg_reduce;
typedef enum { TFG_I32 = 0, TFG_I64 = 1 } tfg_index_type;
/* Order of a per-edge array: the caller's COO edge order, the graph order of
 * a graph handle (edges grouped by target; see tfg_graph_create), or, where a
 * call takes a transposed graph too, that graph's order (edges grouped by
 * source; see tfg_graph_create_transposed). */
typedef enum { TFG_COO = 0, TFG_CSR = 1, TFG_CSR_T = 2 } tfg_edge_order;

typedef void *tfg_stream_t; /* hipStream_t */

/* Opaque graph handle: the CSR-by-target form of one edge list plus the
 * launch plan for it (host struct; its device arrays live in a caller-owned
 * buffer). */
typedef struct tfg_graph tfg_graph;

const char *tfg_status_string(int status);
/* Message for the last failing call on this thread ("" if none). */
const char *tfg_last_error(void);
int tfg_abi_version(void);

/* ------------------------------------------------------------------------ */
/* Graph handle: COO -> CSR by target.                                       */
/* ------------------------------------------------------------------------ */
/*
 * The paper keeps graphs in COO form and reduces over unsorted keys (Sec.
 * 2.1.1, 2.1.2); on the GPU the reduction is done over a CSR-by-target copy,
 * built once per graph structure and reused, in the spirit of the paper's
 * graph-level cache (Sec. 3).
 *
 * Graph order. The handle orders the E' edges (the E input edges, then the N
 * appended self-loops when add_self_loops != 0; loop i has edge id E + i) by
 * the key (target, source part), keeping the input order among equal keys,
 * where source part = source / ceil(N_src / P) for P source parts. This is
 * the unique stable order for that key. With P = 1 it is the CSR by target
 * with the input order inside each target; with P > 1 the edges of each
 * target are further grouped by source range, which lets the aggregation
 * visit the whole graph one source range at a time so that the gathered
 * feature rows stay in the L2 caches. Every per-edge array passed in
 * TFG_CSR order follows this order.
 *
 * src_parts: P, or 0 to let the library choose (P > 1 only when the source
 *   table is large and rows are long: N_src * 512 bytes >= 32 MiB and
 *   E' / N >= 16 * P; at most 16 parts).
 *
 * tfg_graph_bytes: sizes of the persistent buffer (`buf`, kept until
 *   destroy) and of the scratch buffer (`scratch`, needed only during create).
 *
 * tfg_graph_create: validates every id (source in [0, N_src), target in
 *   [0, N)), builds rowptr [N+1], col [E'] (source id per position) and perm
 *   [E'] (input edge id per position) in graph order, and plans the
 *   aggregation launches. Synchronises `stream` once; returns
 *   TFG_ERR_INDEX_RANGE (and no handle) if an id is out of range. `buf` must
 *   stay valid and unmodified until tfg_graph_destroy; `scratch` may be reused
 *   as soon as the call returns.
 *
 * tfg_graph_csr: copies rowptr / col / perm (any may be NULL) into caller
 *   buffers of N+1 / E' / E' int32, enqueued on `stream`.
 * tfg_graph_segments: copies the N*P + 1 segment starts (segment t*P + p =
 *   the edges of target t in source part p) into `segptr`.
 * tfg_graph_info: host-side sizes of the handle (any pointer may be NULL).
 * tfg_check: synchronises `stream` and returns TFG_ERR_INDEX_RANGE if any
 *   device-side check on this graph failed, else TFG_OK.
 * tfg_graph_destroy: frees the host struct (not `buf`).
 *
 * A handle belongs to the device that was current when it was created; every
 * call that reads it fails with TFG_ERR_INVALID_ARG on another device.
 */
int tfg_graph_bytes(int64_t E, int64_t N_src, int64_t N, int add_self_loops, int src_parts,
                    size_t *buf_bytes, size_t *scratch_bytes);
int tfg_graph_create(const void *edge_index, int index_type, int64_t E, int64_t N_src, int64_t N,
                     int add_self_loops, int src_parts, void *buf, size_t buf_bytes,
                     void *scratch, size_t scratch_bytes, tfg_stream_t stream, tfg_graph **out);
/*
 * tfg_graph_create_transposed: the graph of the reversed edge list (every
 *   input edge s -> t becomes t -> s): N_src rows (the sources), col holds
 *   targets, perm the input edge ids (loops: E + i, as above). It carries the
 *   backward aggregation, whose gradient flows from targets to sources. Size
 *   its buffers with tfg_graph_bytes(E, N, N_src, ...) (the two node counts
 *   swapped). Same checks and synchronisation as tfg_graph_create.
 */
int tfg_graph_create_transposed(const void *edge_index, int index_type, int64_t E, int64_t N_src,
                                int64_t N, int add_self_loops, int src_parts, void *buf,
                                size_t buf_bytes, void *scratch, size_t scratch_bytes,
                                tfg_stream_t stream, tfg_graph **out);
int tfg_graph_csr(const tfg_graph *g, int32_t *rowptr, int32_t *col, int32_t *perm,
                  tfg_stream_t stream);
/*
 * tfg_edge_reorder: moves a per-edge array [E', H] from the order of `from`
 *   to the order of `to` (NULL = the caller's COO order, else a graph handle;
 *   both handles, or the handle and the COO array, must describe the same E'
 *   edges, e.g. a graph and its transpose). Gathers through the target order's
 *   perm; leaving a graph order scatters through the source order's perm
 *   (with one value per edge on graphs of 2^20 edges or more, through buckets
 *   of destinations in `ws`); graph -> graph goes through COO order in `ws`.
 *   Query the workspace with tfg_edge_reorder_ws_bytes. Per-edge values that depend only on the
 *   graph structure (normalised weights) are reordered once and cached, like
 *   the graph itself. out must not overlap in.
 */
size_t tfg_edge_reorder_ws_bytes(const tfg_graph *from, const tfg_graph *to, int64_t H);
int tfg_edge_reorder(const tfg_graph *from, const tfg_graph *to, const float *in, int64_t H,
                     float *out, void *ws, size_t ws_bytes, tfg_stream_t stream);
int tfg_graph_segments(const tfg_graph *g, int32_t *segptr, tfg_stream_t stream);
int tfg_graph_info(const tfg_graph *g, int64_t *E_total, int64_t *N, int64_t *N_src,
                   int64_t *src_parts, int64_t *n_chunks, int64_t *n_rows_split,
                   int64_t *n_part_items);
int tfg_check(const tfg_graph *g, tfg_stream_t stream);
int tfg_graph_destroy(tfg_graph *g);

/* ------------------------------------------------------------------------ */
/* GCN normalisation                                                         */
/* ------------------------------------------------------------------------ */
/*
 * The GCN propagation matrix A_hat = D^-1/2 (A + I) D^-1/2 (GCN, Sec. 2.2),
 * edge by edge, cached per graph structure (Sec. 3):
 *   - with add_self_loops, a loop (i, i) of weight 1 is appended after the E
 *     input edges for every node i (E' = E + N); existing loops are kept;
 *   - deg[t]  = sum of the weights of the edges entering t (float32; with
 *     unit weights an exact integer);
 *   - dinv[t] = 1 / sqrt(deg[t]) if deg[t] > 0, else 0 (IEEE sqrt, IEEE divide);
 *   - w_hat[e] = (dinv[src_e] * w_e) * dinv[tgt_e] (float32, left to right).
 * edge_weight: [E] float32 or NULL (all ones). N_src = N (square A).
 * Outputs (each may be NULL):
 *   out_edge_index      [2, E'] int32, COO: the input edges, then the loops;
 *   out_edge_weight     [E'] w_hat in that COO order;
 *   out_edge_weight_csr [E'] w_hat in the graph order of `g` (needs g);
 *   out_deg             [N].
 * g: NULL, or a graph created from the same edge_index with the same N and
 *   add_self_loops. With g == NULL a transient graph is built inside `ws`
 *   (the call then synchronises and reports index errors).
 */
size_t tfg_gcn_norm_ws_bytes(int64_t E, int64_t N, int add_self_loops, const tfg_graph *g);
int tfg_gcn_norm(const void *edge_index, int index_type, int64_t E, const float *edge_weight,
                 int64_t N, int add_self_loops, const tfg_graph *g, int32_t *out_edge_index,
                 float *out_edge_weight, float *out_edge_weight_csr, float *out_deg, void *ws,
                 size_t ws_bytes, tfg_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Message aggregation                                                       */
/* ------------------------------------------------------------------------ */
/*
 * Message aggregation (Sec. 1, Fig. 1) with a reduce-by-target reducer (Sec.
 * 2.1.2). For every edge e and feature column c the message is
 *   m_e[c] = w_e[head(c)] * x[src_e, c],   head(c) = c / (F / H),
 * (w_e = 1 when edge_weight is NULL) and for every target t:
 *   TFG_SUM : out[t, c] = sum of m_e[c] over the edges entering t
 *   TFG_MEAN: that sum divided by the number of edges entering t
 *   TFG_MAX : out[t, c] = max of fl32(w * x) over those edges; argmax[t, c] is
 *             the id of the winning edge in edge_index (the first one in input
 *             order on ties; +0 and -0 tie)
 * A target without edges gets 0 (and argmax -1).
 *
 * edge_index: [2, E] (E = all edges, including loops a previous
 *   tfg_gcn_norm appended); may be NULL when g is given. edge_weight: NULL,
 *   [E] (H = 1) or [E, H], in `weight_order` (TFG_CSR: the graph order of g,
 *   requires g). x: [N_src, F] with leading dimension ldx. out: [N, F].
 *   argmax: [N, F] int32, TFG_MAX only (may be NULL).
 * Sums are float32 in a fixed order: each lane keeps short partial chains
 *   that are combined pairwise, so the error stays within a few hundred units
 *   of float32 rounding of the sum of |m_e[c]|, however long the row.
 * g: NULL, or a graph of this edge_index (its E' equal to E, same N and
 *   N_src); NULL builds a transient graph in `ws` (the call then synchronises).
 *   With P > 1 source parts and a large x the call visits the graph one
 *   source part at a time, writing partial rows to `ws` and combining them
 *   in part order.
 */
size_t tfg_aggregate_ws_bytes(int64_t E, int64_t N_src, int64_t N, int64_t F, int reduce,
                              const tfg_graph *g);
int tfg_aggregate(const void *edge_index, int index_type, int64_t E, const float *edge_weight,
                  int64_t H, int weight_order, const float *x, int64_t N_src, int64_t F,
                  int64_t ldx, int64_t N, int reduce, const tfg_graph *g, float *out,
                  int32_t *argmax, void *ws, size_t ws_bytes, tfg_stream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * aggregation as tfg_aggregate on a cached graph, with the same kernels and
 * bit-identical results, but no workspace argument. The partial rows that
 * tfg_aggregate keeps in `ws` go to a static device array of the library,
 * TFG_NOALLOC_SCRATCH_BYTES bytes on every GPU it runs on, held until the
 * process ends. The call allocates nothing and does not synchronise.
 * g is required (the functional form would need a transient graph); the other
 * arguments are those of tfg_aggregate. A graph and width whose partial rows
 * (the workspace tfg_aggregate_ws_bytes reports, for that handle) exceed the
 * limit give TFG_ERR_WORKSPACE before any launch.
 * Calls that overlap on one GPU (two streams, two threads) share the one
 * array and race: order them on one stream, or use tfg_aggregate.
 */
#define TFG_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int tfg_aggregate_noalloc(const void *edge_index, int index_type, int64_t E,
                          const float *edge_weight, int64_t H, int weight_order, const float *x,
                          int64_t N_src, int64_t F, int64_t ldx, int64_t N, int reduce,
                          const tfg_graph *g, float *out, int32_t *argmax, tfg_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Backward aggregation                                                      */
/* ------------------------------------------------------------------------ */
/*
 * Gradients of tfg_aggregate, for training through graphs built inside the
 * model: graph construction (Sec. 2.1.1) and batching (Sec. 2.1.3) are
 * differentiable, so gradients reach the features and the edge weights. Given dy = dL/d out ([N, F],
 * contiguous), for every edge e = (s -> t) and column c of head k:
 *   TFG_SUM : dx[s, c] += w_e[k] dy[t, c];   dw[e, k] += dy[t, c] x[s, c]
 *   TFG_MEAN: the same with dy[t, c] / (number of edges entering t)
 *   TFG_MAX : only where argmax[t, c] == e (the forward's winning edge).
 * Nothing is accumulated across calls: dx and dw are overwritten.
 * g: the forward graph (tfg_graph_create). gt: NULL, or its transpose
 *   (tfg_graph_create_transposed of the same edge list); required for dx.
 * edge_weight: NULL (all ones) or [E', H] in weight_order (TFG_CSR: the graph
 *   order of g; TFG_CSR_T: the graph order of gt, which the dx gather reads
 *   sequentially, see tfg_edge_reorder). x: [N_src, F] (leading dimension
 *   ldx), needed for dw.
 * argmax: [N, F] int32 from the forward TFG_MAX call (required for TFG_MAX).
 * dx: NULL or [N_src, F] (a source without edges gets 0).
 * dw: NULL or [E', H] in dw_order (TFG_COO: the caller's edge order, loops
 *   after the input edges; TFG_CSR: the graph order of g).
 * Sums are float32 in a fixed order, as in tfg_aggregate: dx goes through the
 * same kernel over gt; each dw entry is one dot product over the columns of
 * its head. Enqueued on `stream`, no synchronisation.
 */
size_t tfg_aggregate_backward_ws_bytes(const tfg_graph *g, const tfg_graph *gt, int64_t F,
                                       int64_t H, int reduce, int weight_order,
                                       int has_edge_weight);
int tfg_aggregate_backward(const tfg_graph *g, const tfg_graph *gt, const float *edge_weight,
                           int64_t H, int weight_order, const float *x, int64_t ldx,
                           const float *dy, int64_t F, int reduce, const int32_t *argmax,
                           float *dx, float *dw, int dw_order, void *ws, size_t ws_bytes,
                           tfg_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Multi-step propagation                                                    */
/* ------------------------------------------------------------------------ */
/*
 * K propagation steps over a square graph (SGC and APPNP, Sec. 2.2):
 *   Z_0 = x,  Z_{k+1} = (1 - alpha) * A Z_k + alpha * h  (k < K),  out = Z_K
 * where (A Z)[t] = sum over the edges e entering t of w_e * Z[src_e] (the sum
 * aggregation of tfg_aggregate). SGC: alpha = 0 (h unused, may be NULL);
 * APPNP: 0 < alpha <= 1 with h = the initial predictions (often x).
 * g: a graph with N_src == N; edge_weight: NULL (all ones) or [E'] in
 * weight_order (TFG_CSR: the graph order, e.g. tfg_gcn_norm's CSR output).
 * x: [N, F] (leading dimension ldx); h: [N, F] (leading dimension ldh);
 * out: [N, F]. out must not overlap x or h. Every step is one aggregation
 * launch whose epilogue applies the update; K = 0 copies x.
 */
size_t tfg_propagate_ws_bytes(const tfg_graph *g, int64_t F, int64_t K);
int tfg_propagate(const tfg_graph *g, const float *edge_weight, int weight_order, const float *x,
                  int64_t F, int64_t ldx, int64_t K, float alpha, const float *h, int64_t ldh,
                  float *out, void *ws, size_t ws_bytes, tfg_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Attention: edge scores and segment softmax                               */
/* ------------------------------------------------------------------------ */
/*
 * The first map of the paper's GAT workflow (Sec. 2.1.2, Fig. 5a): per node
 * and head k, a_s[n, k] = sum_d a_src[k, d] h[n, k*D + d] and a_d likewise
 * with a_dst; per edge, s[e, k] = LeakyReLU(a_s[src_e, k] + a_d[tgt_e, k])
 * with negative slope `slope`. h: [N, H*D]; a_src, a_dst: [H, D];
 * out_scores: [E, H] in the caller's edge order.
 */
size_t tfg_gat_edge_scores_ws_bytes(int64_t N, int64_t H);
int tfg_gat_edge_scores(const void *edge_index, int index_type, int64_t E, const float *h,
                        int64_t N, int64_t H, int64_t D, const float *a_src, const float *a_dst,
                        float slope, float *out_scores, void *ws, size_t ws_bytes,
                        tfg_stream_t stream);

/*
 * Segment softmax: the reduce and the last map of the same workflow (Sec.
 * 2.1.2, Fig. 5): for every segment t (the edges with seg[e] = t) and head h,
 *   out[e, h] = exp(s[e, h] - m) / sum over the segment of exp(s - m)
 * with m the segment's maximum (a shift that leaves the result unchanged).
 * scores: [E, H]; seg: [E] target ids in [0, N) (normally edge_index + E);
 * out: [E, H] in the caller's edge order; out_csr: NULL or [E, H] in the graph
 * order of g (feeds tfg_aggregate with TFG_CSR weights). g: NULL or a graph
 * whose targets are seg (built from the edge list seg belongs to). The
 * maximum and the denominator (double) come out of one online sweep per row;
 * long rows are cut into chunks whose statistics are combined in chunk order
 * (workspace: per-chunk statistics, plus the transient graph when g is NULL).
 */
size_t tfg_segment_softmax_ws_bytes(int64_t E, int64_t H, int64_t N, const tfg_graph *g);
int tfg_segment_softmax(const float *scores, int64_t E, int64_t H, const void *seg,
                        int index_type, int64_t N, const tfg_graph *g, float *out,
                        float *out_csr, void *ws, size_t ws_bytes, tfg_stream_t stream);

/*
 * Gradient of tfg_segment_softmax: for alpha = the segment softmax of the
 * scores and dalpha = dL/d alpha (both [E, H] in the caller's edge order),
 *   dscores[e, h] = alpha[e, h] * (dalpha[e, h] - sum over the segment of
 *                   alpha * dalpha at head h)
 * with the segment sum in double. seg / g as in tfg_segment_softmax.
 */
size_t tfg_segment_softmax_backward_ws_bytes(int64_t E, int64_t H, int64_t N,
                                             const tfg_graph *g);
int tfg_segment_softmax_backward(const float *alpha, const float *dalpha, int64_t E, int64_t H,
                                 const void *seg, int index_type, int64_t N, const tfg_graph *g,
                                 float *dscores, void *ws, size_t ws_bytes, tfg_stream_t stream);

/*
 * The same workflow over a graph handle with the per-edge arrays in `order`:
 * TFG_COO (edge ids of g: the input edges, then the loops) or TFG_CSR (the
 * graph order of g, position k of tfg_graph_csr, the order in which
 * tfg_aggregate reads TFG_CSR weights). In the graph order every target's
 * edges are one contiguous run, so the softmax reads its scores and writes
 * its alpha without the permutation: a GAT layer can keep its scores, alpha
 * and weights in that order from end to end (Sec. 2.1.2, Fig. 5a; the graph
 * is the per-graph cache of Sec. 3).
 * tfg_gat_graph_scores: the additive scores of tfg_gat_edge_scores for the
 *   E' edges of g (sources and targets one node set of N nodes: g forward,
 *   N_src == N); out_scores [E', H] in `order`; h [N, H*D]; a_src, a_dst
 *   [H, D]; ws: tfg_gat_graph_scores_ws_bytes(g, H) bytes (the node
 *   projections). Bit-identical to tfg_gat_edge_scores on the same edges.
 * tfg_segment_softmax_graph: scores and out [E', H], both in `order`, the
 *   segments the targets of g; bit-identical to tfg_segment_softmax with g
 *   (TFG_CSR: to its out_csr). ws: tfg_segment_softmax_graph_ws_bytes(g, H).
 * tfg_segment_softmax_graph_backward: its gradient as
 *   tfg_segment_softmax_backward, alpha, dalpha and dscores [E', H] in
 *   `order`; g forward; the same workspace size.
 * Errors: TFG_ERR_INVALID_ARG (NULL g or pointers, bad H / D / order, a
 * graph of the wrong kind), TFG_ERR_WORKSPACE.
 */
size_t tfg_gat_graph_scores_ws_bytes(const tfg_graph *g, int64_t H);
int tfg_gat_graph_scores(const tfg_graph *g, const float *h, int64_t H, int64_t D,
                         const float *a_src, const float *a_dst, float slope, float *out_scores,
                         int order, void *ws, size_t ws_bytes, tfg_stream_t stream);
size_t tfg_segment_softmax_graph_ws_bytes(const tfg_graph *g, int64_t H);
int tfg_segment_softmax_graph(const tfg_graph *g, const float *scores, int64_t H, int order,
                              float *out, void *ws, size_t ws_bytes, tfg_stream_t stream);
int tfg_segment_softmax_graph_backward(const tfg_graph *g, const float *alpha,
                                       const float *dalpha, int64_t H, int order,
                                       float *dscores, void *ws, size_t ws_bytes,
                                       tfg_stream_t stream);

/*
 * Fused attention aggregation: the whole GAT workflow of Fig. 5(a) plus the
 * weighted message aggregation in one pass over the graph, without writing
 * the [E, H] scores or coefficients:
 *   s[e, k]     = LeakyReLU(a_src[k] . h[src_e, k] + a_dst[k] . h[tgt_e, k], slope)
 *   alpha[e, k] = softmax of s[., k] over the edges entering tgt_e
 *   out[t, k*D + d] = sum over the edges e entering t of alpha[e, k] h[src_e, k*D + d]
 * Equal (up to rounding) to tfg_gat_edge_scores -> tfg_segment_softmax ->
 * tfg_aggregate with per-head weights. g: a square graph (N_src == N);
 * h: [N, H*D]; a_src, a_dst: [H, D]; H <= 64; out: [N, H*D] (a target
 * without edges gets 0). alpha_out: NULL, or [E', H] to also receive alpha in
 * the caller's edge order (edge ids as in the graph, loops included).
 * Each row is swept once: the maximum and the denominator (double) are kept
 * online, rescaled whenever the maximum grows, so the result differs from the
 * three-step chain only by rounding; rows longer than the graph's chunk are
 * cut into chunks whose partial results are combined in chunk order.
 * ws: tfg_gat_aggregate_ws_bytes(g, H, D) bytes.
 */
size_t tfg_gat_aggregate_ws_bytes(const tfg_graph *g, int64_t H, int64_t D);
int tfg_gat_aggregate(const tfg_graph *g, const float *h, int64_t H, int64_t D,
                      const float *a_src, const float *a_dst, float slope, float *out,
                      float *alpha_out, void *ws, size_t ws_bytes, tfg_stream_t stream);

/*
 * Transformer-style attention, the GAT variant the paper's library uses (Sec.
 * 4.2): per edge e = (s -> t) and head k, the scaled dot product
 *   s[e, k] = scale * sum_d q[t, k*D + d] * key[s, k*D + d]
 * (scale usually 1/sqrt(D)), the softmax of s[., k] over the edges entering
 * each target, and out[t, k*D + d] = sum over those edges of alpha[e, k] *
 * v[s, k*D + d]. q: [N, H*D] (one row per target), key, v: [N_src, H*D] (per
 * source); all contiguous. The query, key and value projections are dense
 * layers outside this library.
 * tfg_edge_dot_scores: the scores alone, [E', H] in `order` (TFG_COO: edge
 *   ids of g, loops after the input edges; TFG_CSR: the graph order); they
 *   feed tfg_segment_softmax and tfg_aggregate (the unfused chain). Any D.
 * tfg_gat_dot_aggregate: the whole layer in one sweep per row, as
 *   tfg_gat_aggregate (online maximum and denominator, chunks of long rows
 *   merged in order); D a power of two, at most 64; H <= 64. alpha_out: NULL
 *   or [E', H] in edge-id order. ws: tfg_gat_dot_aggregate_ws_bytes(g, H, D).
 */
int tfg_edge_dot_scores(const tfg_graph *g, const float *q, const float *key, int64_t H,
                        int64_t D, float scale, float *out_scores, int order,
                        tfg_stream_t stream);
size_t tfg_gat_dot_aggregate_ws_bytes(const tfg_graph *g, int64_t H, int64_t D);
int tfg_gat_dot_aggregate(const tfg_graph *g, const float *q, const float *key, const float *v,
                          int64_t H, int64_t D, float scale, float *out, float *alpha_out,
                          void *ws, size_t ws_bytes, tfg_stream_t stream);

/* ------------------------------------------------------------------------ */
/* Graph pooling                                                             */
/* ------------------------------------------------------------------------ */
/*
 * Graph pooling (Sec. 1, Fig. 2a) over a BatchGraph's node_graph_index (Sec.
 * 2.1.1): node n belongs to graph graph_index[n]; ids must be in [0, G) and
 * non-decreasing (BatchGraph numbers the nodes graph by graph).
 *   TFG_SUM / TFG_MEAN (divided by the node count) / TFG_MAX with argmax =
 *   node id (the lowest on ties). A graph without nodes gets 0 (argmax -1).
 * x: [Nb, F] with leading dimension ldx; out: [G, F]; argmax: [G, F] int32 or
 * NULL (TFG_MAX only). validate != 0: synchronise and return
 * TFG_ERR_INDEX_RANGE / TFG_ERR_UNSORTED for bad ids; validate == 0: do not
 * wait (bad ids are clamped: no fault, unspecified values).
 */
size_t tfg_segment_pool_ws_bytes(int64_t Nb, int64_t G);
int tfg_segment_pool(const float *x, int64_t Nb, int64_t F, int64_t ldx, const void *graph_index,
                     int index_type, int64_t G, int reduce, float *out, int32_t *argmax,
                     int validate, void *ws, size_t ws_bytes, tfg_stream_t stream);

/*
 * Gradient of tfg_segment_pool, for training graph-level models through the
 * pooling (Sec. 4.1): given dy = dL/d out ([G, F], contiguous), node n of
 * graph g receives dx[n, c] = dy[g, c] (TFG_SUM), dy[g, c] / (nodes of g)
 * (TFG_MEAN), or dy[g, c] if argmax[g, c] == n and 0 otherwise (TFG_MAX;
 * argmax as the forward call returned it). dx: [Nb, F] with leading
 * dimension ldx, overwritten. graph_index, validate and ws as in
 * tfg_segment_pool (same workspace size).
 */
int tfg_segment_pool_backward(const float *dy, int64_t G, int64_t F, const void *graph_index,
                              int index_type, int64_t Nb, int reduce, const int32_t *argmax,
                              float *dx, int64_t ldx, int validate, void *ws, size_t ws_bytes,
                              tfg_stream_t stream);

/* ------------------------------------------------------------------------ */
/* BatchGraph construction                                                   */
/* ------------------------------------------------------------------------ */
/*
 * Combines G graphs into one BatchGraph (Sec. 2.1.1, Fig. 4): node j of graph
 * i gets the id j + (number of nodes in graphs 0..i-1), every local edge is
 * shifted by its graph's offset, and node_graph_index[n] is the graph of node
 * n (non-decreasing). Node features need no change: they are the per-graph
 * rows stacked in graph order.
 * node_counts, edge_counts: [G] (index_type); local_edge_index: [2, E] with
 * the edges of graph 0, then graph 1, ... (row 0 sources, row 1 targets, ids
 * local to their graph); E = sum of edge_counts, Nb = sum of node_counts (both
 * from tfg_batch_graphs_totals when the caller does not know them).
 * Outputs: out_edge_index [2, E] and out_graph_index [Nb] (index_type);
 * out_node_offsets / out_edge_offsets: NULL or [G + 1] int32.
 * validate != 0: synchronise and return TFG_ERR_INDEX_RANGE if a count is
 * negative, a local id is outside its graph, or E / Nb differ from the sums.
 */
/*
 * The sizes of a BatchGraph before it is built (Sec. 2.1.1): *Nb = sum of
 * node_counts and *E = sum of edge_counts ([G], index_type, device memory),
 * summed on the device in 64 bits. ws: tfg_batch_graphs_ws_bytes(G) bytes,
 * 256-byte aligned. Synchronises the stream once to read the totals back.
 * Errors: TFG_ERR_INVALID_ARG (bad G or index type, NULL pointer),
 * TFG_ERR_INDEX_RANGE (a negative count), TFG_ERR_WORKSPACE.
 */
int tfg_batch_graphs_totals(int64_t G, const void *node_counts, const void *edge_counts,
                            int index_type, void *ws, size_t ws_bytes, tfg_stream_t stream,
                            int64_t *Nb, int64_t *E);

size_t tfg_batch_graphs_ws_bytes(int64_t G);
int tfg_batch_graphs(int64_t G, const void *node_counts, const void *edge_counts,
                     const void *local_edge_index, int index_type, int64_t E, int64_t Nb,
                     void *out_edge_index, void *out_graph_index, int32_t *out_node_offsets,
                     int32_t *out_edge_offsets, int validate, void *ws, size_t ws_bytes,
                     tfg_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* TFG_H */
