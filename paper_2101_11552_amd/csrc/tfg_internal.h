// Internal declarations of the HIP library behind include/tfg.h (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstddef>
#include <cstdint>
#include <string>

#include "../../include/tfg.h"

namespace tfg {

constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kBlock = 256;        // threads per block for most kernels (4 waves)
// Kernels whose wavefronts each take their own work items run one wavefront
// per block, so that a CU starts the next item as soon as any wavefront ends.
constexpr int kItemBlock = 64;
constexpr int kDefaultChunk = 128; // max edges per work item of the row plan
constexpr int kMaxChunk = 1 << 16;  // largest chunk the tuning knob may set
constexpr int kShortRow = 8;       // rows of at most this many edges are "short"

// Device error flag bits (graph->err and the pooling workspace flag).
constexpr int kErrIndex = 1;
constexpr int kErrUnsorted = 2;

// One aggregation work item, processed by one wavefront: the positions
// [kbeg, kend) (graph order) of target `row`. slot < 0: the item covers the
// whole row and writes the output row; slot >= 0: the item writes partial
// result `slot` and a fix-up pass combines the row's partials in order.
struct WorkItem {
  int row, kbeg, kend, slot;
};
// A row reduced from partials: slots slot0 .. slot0 + nchunks - 1, in order.
struct SplitRow {
  int row, slot0, nchunks, deg;
};

constexpr int kMaxParts = 16;

// Host view of a graph; the arrays live in the caller's persistent buffer.
//
// Edge order ("graph order"): edges sorted by the key (target, source part),
// input order kept among equal keys, where source part = source / part_rows.
// With parts == 1 this is the stable CSR by target. With parts > 1 the edges
// of each row are grouped by source range, which lets the aggregation visit
// the whole graph one source range at a time (the gathered rows of one range
// stay in the L2 caches while it is processed).
struct Graph {
  int64_t E_in = 0;    // input edges
  int64_t E = 0;       // total edges (input + appended loops)
  int64_t N = 0;       // targets
  int64_t N_src = 0;   // sources
  int loops = 0;
  int transposed = 0;  // built from the reversed edge list (rows are sources)
  int chunk = kDefaultChunk;
  int parts = 1;            // source parts P
  int64_t part_rows = 1;    // sources per part
  int* rowptr = nullptr;    // [N+1]
  int* segptr = nullptr;    // [N*P+1]: start of (row, part); == rowptr when P == 1
  int* col = nullptr;       // [E] source id per position
  int* perm = nullptr;      // [E] input edge id per position
  int* key = nullptr;       // [E] sort key per position: target * parts + source part
  // row plan: one item per row (long rows cut into chunks + fix-up)
  WorkItem* heavy = nullptr;  // chunks of split rows; heavy[i] writes partial i
  WorkItem* light = nullptr;  // whole rows
  SplitRow* split = nullptr;
  int n_heavy = 0, n_light = 0, n_split = 0;
  // the light rows again, by length: short (0..kShortRow edges, row ids,
  // several per wavefront) and the rest (whole-row items, one per wavefront)
  WorkItem* short_rows = nullptr;  // (row, kbeg, kend, -1): one load gives a row's extent
  WorkItem* long_rows = nullptr;
  int n_short = 0, n_long = 0;
  // part plan (P > 1): one item per (part, row) segment chunk, part-major
  // order; every item writes a partial, prows[t] reduces row t's partials
  WorkItem* pexec = nullptr;
  SplitRow* prows = nullptr;
  int n_pexec = 0;
  // device: [0] heavy, [1] light, [2] split, [3] error flags, [4] part items,
  // [5] short rows, [6] other light rows
  int* counters = nullptr;
  int device = 0;
};

// Sizes of the persistent part of a graph.
struct GraphLayout {
  size_t rowptr, segptr, col, perm, key, heavy, light, split, pexec, prows, short_rows, long_rows,
      counters, total;
  int64_t cap_heavy, cap_light, cap_split, cap_pexec;
};
GraphLayout graph_layout(int64_t E, int64_t N, int parts, int chunk);
size_t graph_scratch_bytes(int64_t E, int64_t N, int parts);
int default_chunk();
// Pinned host ints (8) of the calling thread for counter readbacks, or NULL.
int* readback_buffer();
// Number of source parts for a graph: `requested` if >= 1 (capped), else a
// choice from the sizes (P > 1 only when the gathered table is much larger
// than the L2 caches and rows are long enough to be split by source range).
int choose_parts(int64_t E, int64_t N, int64_t N_src, int requested);

// Thread-local error message.
void set_error(const std::string& msg);
int fail(int status, const std::string& msg);
int hip_fail(hipError_t e, const char* what);

#define TFG_HIP(call)                                   \
  do {                                                  \
    hipError_t e_ = (call);                             \
    if (e_ != hipSuccess) return hip_fail(e_, #call);   \
  } while (0)
#define TFG_LAUNCHED(what)                              \
  do {                                                  \
    hipError_t e_ = hipGetLastError();                  \
    if (e_ != hipSuccess) return hip_fail(e_, what);    \
  } while (0)

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// ---- launchers (each returns a tfg_status) --------------------------------
// csr.hip
// src may be NULL (a target-only list: col is then all zero).
int build_graph(Graph& g, const void* src, const void* tgt, int index_type, void* scratch,
                size_t scratch_bytes, hipStream_t s);
// tile_sums: exclusive_scan_sums(n) ints of scratch
int exclusive_scan(const int* in, int* out, int64_t n, int* tile_sums, hipStream_t s);
int64_t exclusive_scan_sums(int64_t n);
// norm.hip
int launch_gcn_norm(const Graph& g, const void* edge_index, int index_type,
                    const float* edge_weight, int32_t* out_edge_index, float* out_w,
                    float* out_w_csr, float* out_deg, float* dinv_ws, hipStream_t s);
// aggregate.hip
// With h != NULL (or scale != 1) every output row becomes scale * sum +
// alpha * h[row] (sum reduction only): one propagation step. With mask != NULL
// ([rows of x, F] int32, sum only) element c of x[col_k] counts only where
// mask[col_k, c] == perm[k].
int launch_aggregate(const Graph& g, const float* w, int H, int w_order, const float* x,
                     int64_t F, int64_t ldx, int reduce, float* out, int32_t* argmax,
                     void* ws, hipStream_t s, float scale = 1.0f, float alpha = 0.0f,
                     const float* h = nullptr, int64_t ldh = 0, const int32_t* mask = nullptr);
size_t aggregate_partial_bytes(int64_t n_partials, int64_t F, int reduce);
// Device address, on the current device, of the library's static scratch
// (TFG_NOALLOC_SCRATCH_BYTES bytes); looked up once per device.
int noalloc_scratch(void** ptr);
// Whether an aggregation over g with F features uses the part plan.
bool use_part_plan(const Graph& g, int64_t F);
// softmax.hip
int launch_gat_scores(const void* edge_index, int index_type, int64_t E, const float* h,
                      int64_t N, int H, int D, const float* a_src, const float* a_dst,
                      float slope, float* out, float* proj_ws, int* err, hipStream_t s);
// Per-chunk softmax statistics of the long rows: [n_chunks, H] float maxima
// and double sums (the workspace of the softmax launches).
size_t row_stats_bytes(int64_t n_chunks, int64_t H);
// graph_order: scores and out in the graph order of g (position k), out_csr unused.
int launch_segment_softmax(const Graph& g, const float* scores, int H, float* out,
                           float* out_csr, void* ws, hipStream_t s, bool graph_order = false);
// The additive scores over a graph handle (projections into proj_ws, [2, N, H]),
// written in the graph order or (by_perm) at the caller's edge ids.
int launch_gat_graph_scores(const Graph& g, const float* h, int H, int D, const float* a_src,
                            const float* a_dst, float slope, float* out, int by_perm,
                            float* proj_ws, hipStream_t s);
// pool.hip
int launch_segment_pool(const float* x, int64_t Nb, int64_t F, int64_t ldx,
                        const void* graph_index, int index_type, int64_t G, int reduce,
                        float* out, int32_t* argmax, int* goff_ws, int* err, hipStream_t s);

int launch_segment_pool_backward(const float* dy, int64_t G, int64_t F, const void* graph_index,
                                 int index_type, int64_t Nb, int reduce, const int32_t* argmax,
                                 float* dx, int64_t ldx, int* goff, int* err, hipStream_t s);

// softmax.hip: a_s = a_src . h and a_d = a_dst . h per (node, head)
int launch_node_projections(const float* h, int64_t N, int H, int D, const float* a_src,
                            const float* a_dst, float* as, float* ad, hipStream_t s);
// backward.hip: gradients of launch_aggregate (dx over gt, the transposed
// graph; dw over g) and of launch_segment_softmax.
size_t aggregate_backward_ws_bytes(const Graph& g, const Graph* gt, int64_t F, int64_t H,
                                   int reduce, int w_order, bool has_w);
int launch_aggregate_backward(const Graph& g, const Graph* gt, const float* w, int H, int w_order,
                              const float* x, int64_t ldx, const float* dy, int64_t F,
                              int reduce, const int32_t* argmax, float* dx, float* dw,
                              int dw_order, void* ws, hipStream_t s);
// out[k] = in[perm_to[k]] (COO -> graph), out[perm_from[k]] = in[k] (graph ->
// COO), or both through tmp ([E, H] floats); either perm may be NULL.
// out[perm[k], h] = in[k, h], bucketed on large graphs when ws holds
// perm_scatter_ws_bytes(E, H) (0: the plain scatter, no scratch)
size_t perm_scatter_ws_bytes(int64_t E, int H);
int launch_perm_scatter(const int* perm, int64_t E, int H, const float* in, float* out, void* ws,
                        size_t ws_bytes, hipStream_t s);
size_t edge_reorder_ws_bytes(int64_t E, int H, bool from, bool to);
int launch_edge_reorder(const int* perm_from, const int* perm_to, int64_t E, int H,
                        const float* in, float* out, void* ws, size_t ws_bytes, hipStream_t s);
int launch_segment_softmax_backward(const Graph& g, const float* alpha, const float* dalpha,
                                    int H, float* ds, void* ws, hipStream_t s,
                                    bool graph_order = false);
// gat.hip
size_t gat_aggregate_ws_bytes(const Graph& g, int64_t H, int64_t D);
// Scaled dot-product variant: D a power of two, at most 64.
bool dot_attention_shape_ok(int64_t D);
int launch_gat_dot_aggregate(const Graph& g, const float* q, const float* key, const float* v,
                             int H, int D, float scale, float* out, float* alpha_out, void* ws,
                             hipStream_t s);
// backward.hip: out[e, k] = scale * <q[t_e], key[s_e]> over the columns of
// head k, in COO (by_perm) or graph order.
int launch_edge_dot(const Graph& g, const float* q, const float* key, int64_t ldk, int64_t F,
                    int H, float scale, float* out, int by_perm, hipStream_t s);
int max_fused_heads();
int launch_gat_aggregate(const Graph& g, const float* h, int H, int D, const float* a_src,
                         const float* a_dst, float slope, float* out, float* alpha_out, void* ws,
                         hipStream_t s);
// batch.hip
size_t batch_ws_bytes(int64_t G);
// Node and edge totals of the counts and a negative-count flag: five ints
// (node total low, high; edge total low, high; flag) at `out`.
int launch_batch_totals(int64_t G, const void* node_counts, const void* edge_counts,
                        int index_type, int* out, hipStream_t s);
// out_node_off / out_edge_off: NULL or [G + 1] copies of the offsets.
int launch_batch_graphs(int64_t G, const void* node_counts, const void* edge_counts,
                        const void* local_edge_index, int index_type, int64_t E, int64_t Nb,
                        void* out_edge_index, void* out_graph_index, int* node_off, int* edge_off,
                        int* out_node_off, int* out_edge_off, int* sums, int* err,
                        hipStream_t s);

}  // namespace tfg
