// extern "C" entry points of include/tfg.h: argument checks, workspace
// carving and graph handles around the kernels in the .hip sources.
#include <algorithm>
#include <cstring>
#include <new>
#include <string>

#include "tfg_internal.h"

struct tfg_graph {
  tfg::Graph g;
};

namespace tfg {

namespace {
thread_local std::string g_last_error;
// Counts (nodes, edges with their appended loops, E * H, features, graphs)
// stay below 2^31 - 2^20: kernels keep positions in 32-bit ints and step
// through them in strides of up to a work item (at most 2^16 positions), so
// the margin keeps every position plus a stride representable.
constexpr int64_t kMaxCount = (int64_t(1) << 31) - (int64_t(1) << 20);
}  // namespace

void set_error(const std::string& msg) { g_last_error = msg; }

int fail(int status, const std::string& msg) {
  set_error(msg);
  return status;
}

int hip_fail(hipError_t e, const char* what) {
  set_error(std::string(what) + ": " + hipGetErrorString(e));
  return TFG_ERR_HIP;
}

namespace {

hipStream_t as_stream(tfg_stream_t s) { return reinterpret_cast<hipStream_t>(s); }

bool bad_index_type(int t) { return t != TFG_I32 && t != TFG_I64; }

// Carves a caller buffer into 256-byte aligned pieces.
struct Carver {
  char* base;
  size_t size, off = 0;
  Carver(void* b, size_t n) : base(static_cast<char*>(b)), size(n) {}
  void* take(size_t bytes) {
    void* p = base ? base + off : nullptr;
    off = align_up(off + bytes, 256);
    return p;
  }
};

// A caller workspace: present, 256-byte aligned (kernels read it with wide
// loads) and at least `need` bytes.
int check_ws(const void* ws, size_t bytes, size_t need) {
  if (ws == nullptr || bytes < need) return fail(TFG_ERR_WORKSPACE, "workspace too small");
  if (reinterpret_cast<uintptr_t>(ws) % 256 != 0)
    return fail(TFG_ERR_WORKSPACE, "workspace not 256-byte aligned");
  return TFG_OK;
}

// Reads n (<= 8) ints from device addresses into `to`, through the calling
// thread's pinned buffer when there is one, and synchronises the stream.
int read_back(hipStream_t s, int n, const int* const* from, int* to) {
  int* pin = readback_buffer();
  int* buf = pin ? pin : to;
  for (int i = 0; i < n; ++i)
    TFG_HIP(hipMemcpyAsync(buf + i, from[i], sizeof(int), hipMemcpyDeviceToHost, s));
  TFG_HIP(hipStreamSynchronize(s));
  if (pin)
    for (int i = 0; i < n; ++i) to[i] = pin[i];
  return TFG_OK;
}

size_t graph_total_bytes(int64_t E, int64_t N, int parts) {
  return graph_layout(E, N, parts, default_chunk()).total + graph_scratch_bytes(E, N, parts);
}

int check_counts(int64_t E, int64_t N, int64_t N_src) {
  if (E < 0 || N < 0 || N_src < 0) return fail(TFG_ERR_INVALID_ARG, "negative size");
  if (E >= kMaxCount || N >= kMaxCount || N_src >= kMaxCount)
    return fail(TFG_ERR_TOO_LARGE, "edge or node count not below 2^31 - 2^20");
  return TFG_OK;
}

// Fills g's device pointers from `buf` and builds the CSR form.
int create_graph(Graph& g, const void* src, const void* tgt, int index_type, int64_t E_in,
                 int64_t N_src, int64_t N, int loops, int src_parts, void* buf, size_t buf_bytes,
                 void* scratch, size_t scratch_bytes, hipStream_t s) {
  g.E_in = E_in;
  g.E = E_in + (loops ? N : 0);
  g.N = N;
  g.N_src = N_src;
  g.loops = loops ? 1 : 0;
  g.chunk = default_chunk();
  int rc = check_counts(g.E, N, N_src);
  if (rc) return rc;
  g.parts = choose_parts(g.E, N, N_src, src_parts);
  g.part_rows = std::max<int64_t>((N_src + g.parts - 1) / g.parts, 1);
  GraphLayout L = graph_layout(g.E, N, g.parts, g.chunk);
  if (buf == nullptr || buf_bytes < L.total)
    return fail(TFG_ERR_WORKSPACE, "graph buffer too small");
  if (reinterpret_cast<uintptr_t>(buf) % 256 != 0 || reinterpret_cast<uintptr_t>(scratch) % 256 != 0)
    return fail(TFG_ERR_WORKSPACE, "graph buffer or scratch not 256-byte aligned");
  char* b = static_cast<char*>(buf);
  g.rowptr = reinterpret_cast<int*>(b + L.rowptr);
  g.segptr = g.parts > 1 ? reinterpret_cast<int*>(b + L.segptr) : g.rowptr;
  g.col = reinterpret_cast<int*>(b + L.col);
  g.perm = reinterpret_cast<int*>(b + L.perm);
  g.key = reinterpret_cast<int*>(b + L.key);
  g.heavy = reinterpret_cast<WorkItem*>(b + L.heavy);
  g.light = reinterpret_cast<WorkItem*>(b + L.light);
  g.split = reinterpret_cast<SplitRow*>(b + L.split);
  g.pexec = reinterpret_cast<WorkItem*>(b + L.pexec);
  g.prows = reinterpret_cast<SplitRow*>(b + L.prows);
  g.short_rows = reinterpret_cast<WorkItem*>(b + L.short_rows);
  g.long_rows = reinterpret_cast<WorkItem*>(b + L.long_rows);
  g.counters = reinterpret_cast<int*>(b + L.counters);
  TFG_HIP(hipGetDevice(&g.device));
  return build_graph(g, src, tgt, index_type, scratch, scratch_bytes, s);
}

// A handle's device arrays live on the device that was current when it was
// built; every call that reads them must run there.
int check_device(const Graph& g) {
  int d = 0;
  TFG_HIP(hipGetDevice(&d));
  if (d != g.device) return fail(TFG_ERR_INVALID_ARG, "the graph lives on another device");
  return TFG_OK;
}

int check_device(const tfg_graph* h) { return h ? check_device(h->g) : TFG_OK; }

const void* tgt_row(const void* edge_index, int index_type, int64_t E) {
  if (edge_index == nullptr) return nullptr;
  return index_type == TFG_I64 ? static_cast<const void*>(static_cast<const int64_t*>(edge_index) + E)
                               : static_cast<const void*>(static_cast<const int32_t*>(edge_index) + E);
}

// Either checks that `g` describes an edge list of E edges over N_src x N
// (with or without loops), or builds a transient graph in the carver.
int graph_or_transient(const tfg_graph* handle, Graph& tmp, const Graph*& g, const void* src,
                       const void* tgt, int index_type, int64_t E, int64_t N_src, int64_t N,
                       int loops, Carver& ws, hipStream_t s) {
  if (handle) {
    g = &handle->g;
    if (g->E_in != E || g->N != N || g->N_src != N_src || g->loops != (loops ? 1 : 0))
      return fail(TFG_ERR_INVALID_ARG, "graph handle does not match the edge list sizes");
    if (g->transposed) return fail(TFG_ERR_INVALID_ARG, "a transposed graph cannot serve here");
    return check_device(*g);
  }
  const int64_t Ep = E + (loops ? N : 0);
  const int parts = choose_parts(Ep, N, N_src, 0);
  GraphLayout L = graph_layout(Ep, N, parts, default_chunk());
  size_t sc = graph_scratch_bytes(Ep, N, parts);
  void* buf = ws.take(L.total);
  void* scratch = ws.take(sc);
  if (ws.off > ws.size) return fail(TFG_ERR_WORKSPACE, "workspace too small");
  int rc = create_graph(tmp, src, tgt, index_type, E, N_src, N, loops, 0, buf, L.total, scratch,
                        sc, s);
  g = &tmp;
  return rc;
}

// Partial rows an aggregation needs: those of the plan it will use (for a
// transient graph, the larger capacity of the two plans).
int64_t partials_needed(int64_t E, int64_t N, int64_t N_src, int64_t F, const tfg_graph* g) {
  if (g) return use_part_plan(g->g, F) ? g->g.n_pexec : g->g.n_heavy;
  const int parts = choose_parts(E, N, N_src, 0);
  const GraphLayout L = graph_layout(E, N, parts, default_chunk());
  return std::max(L.cap_heavy, L.cap_pexec);
}

size_t aggregate_ws_needed(int64_t E, int64_t N, int64_t N_src, int64_t F, int reduce,
                           const tfg_graph* g) {
  if (E < 0 || N < 0 || N_src < 0 || F < 0) return 0;
  size_t b = aggregate_partial_bytes(partials_needed(E, N, N_src, F, g), F, reduce);
  if (!g) b += graph_total_bytes(E, N, choose_parts(E, N, N_src, 0));
  return b;
}

}  // namespace
}  // namespace tfg

using namespace tfg;

extern "C" {

const char* tfg_status_string(int status) {
  switch (status) {
    case TFG_OK: return "ok";
    case TFG_ERR_INVALID_ARG: return "invalid argument";
    case TFG_ERR_INDEX_RANGE: return "index out of range";
    case TFG_ERR_UNSORTED: return "graph index not sorted";
    case TFG_ERR_TOO_LARGE: return "size too large";
    case TFG_ERR_WORKSPACE: return "workspace too small";
    case TFG_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* tfg_last_error(void) { return g_last_error.c_str(); }

int tfg_abi_version(void) { return TFG_ABI_VERSION; }

int tfg_graph_bytes(int64_t E, int64_t N_src, int64_t N, int add_self_loops, int src_parts,
                    size_t* buf_bytes, size_t* scratch_bytes) {
  int rc = check_counts(E, N, N_src);
  if (rc) return rc;
  const int64_t Ep = E + (add_self_loops ? N : 0);
  rc = check_counts(Ep, N, N_src);
  if (rc) return rc;
  const int parts = choose_parts(Ep, N, N_src, src_parts);
  if (buf_bytes) *buf_bytes = graph_layout(Ep, N, parts, default_chunk()).total;
  if (scratch_bytes) *scratch_bytes = graph_scratch_bytes(Ep, N, parts);
  return TFG_OK;
}

namespace {

int create_handle(const void* edge_index, int index_type, int64_t E, int64_t N_src, int64_t N,
                  int add_self_loops, int src_parts, void* buf, size_t buf_bytes, void* scratch,
                  size_t scratch_bytes, tfg_stream_t stream, bool transposed, tfg_graph** out) {
  if (out == nullptr) return fail(TFG_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (bad_index_type(index_type)) return fail(TFG_ERR_INVALID_ARG, "bad index type");
  if (E > 0 && edge_index == nullptr) return fail(TFG_ERR_INVALID_ARG, "edge_index is NULL");
  if (add_self_loops && N_src != N)
    return fail(TFG_ERR_INVALID_ARG, "self-loops need N_src == N");
  if (scratch == nullptr) return fail(TFG_ERR_INVALID_ARG, "scratch is NULL");
  tfg_graph* h = new (std::nothrow) tfg_graph;
  if (!h) return fail(TFG_ERR_HIP, "host allocation failed");
  const void* src = edge_index;
  const void* tgt = tgt_row(edge_index, index_type, E);
  int rc = transposed
               ? create_graph(h->g, tgt, src, index_type, E, N, N_src, add_self_loops, src_parts,
                              buf, buf_bytes, scratch, scratch_bytes, as_stream(stream))
               : create_graph(h->g, src, tgt, index_type, E, N_src, N, add_self_loops, src_parts,
                              buf, buf_bytes, scratch, scratch_bytes, as_stream(stream));
  if (rc) {
    delete h;
    return rc;
  }
  h->g.transposed = transposed ? 1 : 0;
  *out = h;
  return TFG_OK;
}

}  // namespace

int tfg_graph_create(const void* edge_index, int index_type, int64_t E, int64_t N_src, int64_t N,
                     int add_self_loops, int src_parts, void* buf, size_t buf_bytes, void* scratch,
                     size_t scratch_bytes, tfg_stream_t stream, tfg_graph** out) {
  return create_handle(edge_index, index_type, E, N_src, N, add_self_loops, src_parts, buf,
                       buf_bytes, scratch, scratch_bytes, stream, false, out);
}

int tfg_graph_create_transposed(const void* edge_index, int index_type, int64_t E, int64_t N_src,
                                int64_t N, int add_self_loops, int src_parts, void* buf,
                                size_t buf_bytes, void* scratch, size_t scratch_bytes,
                                tfg_stream_t stream, tfg_graph** out) {
  return create_handle(edge_index, index_type, E, N_src, N, add_self_loops, src_parts, buf,
                       buf_bytes, scratch, scratch_bytes, stream, true, out);
}

int tfg_graph_csr(const tfg_graph* h, int32_t* rowptr, int32_t* col, int32_t* perm,
                  tfg_stream_t stream) {
  if (!h) return fail(TFG_ERR_INVALID_ARG, "graph is NULL");
  if (int rc = check_device(h)) return rc;
  const Graph& g = h->g;
  hipStream_t s = as_stream(stream);
  if (rowptr)
    TFG_HIP(hipMemcpyAsync(rowptr, g.rowptr, sizeof(int) * (g.N + 1), hipMemcpyDeviceToDevice, s));
  if (col && g.E)
    TFG_HIP(hipMemcpyAsync(col, g.col, sizeof(int) * g.E, hipMemcpyDeviceToDevice, s));
  if (perm && g.E)
    TFG_HIP(hipMemcpyAsync(perm, g.perm, sizeof(int) * g.E, hipMemcpyDeviceToDevice, s));
  return TFG_OK;
}

size_t tfg_edge_reorder_ws_bytes(const tfg_graph* from, const tfg_graph* to, int64_t H) {
  if (H < 1) return 0;
  const int64_t E = from ? from->g.E : (to ? to->g.E : 0);
  return edge_reorder_ws_bytes(E, (int)H, from != nullptr, to != nullptr) + 256;
}

int tfg_edge_reorder(const tfg_graph* from, const tfg_graph* to, const float* in, int64_t H,
                     float* out, void* ws, size_t ws_bytes, tfg_stream_t stream) {
  if (!from && !to) return fail(TFG_ERR_INVALID_ARG, "no graph handle");
  if (from && to && (from->g.E != to->g.E || from->g.E_in != to->g.E_in))
    return fail(TFG_ERR_INVALID_ARG, "the graphs describe different edge lists");
  const int64_t E = from ? from->g.E : to->g.E;
  if (H < 1 || E * H >= kMaxCount) return fail(TFG_ERR_INVALID_ARG, "bad H");
  if (E > 0 && (in == nullptr || out == nullptr)) return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (E > 0 && in == out) return fail(TFG_ERR_INVALID_ARG, "out overlaps in");
  if (int wrc = check_ws(ws, ws_bytes, tfg_edge_reorder_ws_bytes(from, to, H))) return wrc;
  if (int rc = check_device(from)) return rc;
  if (int rc = check_device(to)) return rc;
  return launch_edge_reorder(from ? from->g.perm : nullptr, to ? to->g.perm : nullptr, E, (int)H,
                             in, out, ws, ws_bytes, as_stream(stream));
}

int tfg_graph_info(const tfg_graph* h, int64_t* E_total, int64_t* N, int64_t* N_src,
                   int64_t* src_parts, int64_t* n_chunks, int64_t* n_rows_split,
                   int64_t* n_part_items) {
  if (!h) return fail(TFG_ERR_INVALID_ARG, "graph is NULL");
  if (E_total) *E_total = h->g.E;
  if (N) *N = h->g.N;
  if (N_src) *N_src = h->g.N_src;
  if (src_parts) *src_parts = h->g.parts;
  if (n_chunks) *n_chunks = h->g.n_heavy;
  if (n_rows_split) *n_rows_split = h->g.n_split;
  if (n_part_items) *n_part_items = h->g.n_pexec;
  return TFG_OK;
}

int tfg_graph_segments(const tfg_graph* h, int32_t* segptr, tfg_stream_t stream) {
  if (!h || !segptr) return fail(TFG_ERR_INVALID_ARG, "NULL argument");
  if (int rc = check_device(h)) return rc;
  const Graph& g = h->g;
  TFG_HIP(hipMemcpyAsync(segptr, g.segptr, sizeof(int) * (g.N * g.parts + 1),
                         hipMemcpyDeviceToDevice, as_stream(stream)));
  return TFG_OK;
}

int tfg_check(const tfg_graph* h, tfg_stream_t stream) {
  if (!h) return fail(TFG_ERR_INVALID_ARG, "graph is NULL");
  if (int rc = check_device(h)) return rc;
  int flags = 0;
  const int* from[1] = {h->g.counters + 3};
  if (int rc = read_back(as_stream(stream), 1, from, &flags)) return rc;
  if (flags & kErrIndex) return fail(TFG_ERR_INDEX_RANGE, "an id was out of range");
  return TFG_OK;
}

int tfg_graph_destroy(tfg_graph* h) {
  delete h;
  return TFG_OK;
}

size_t tfg_gcn_norm_ws_bytes(int64_t E, int64_t N, int add_self_loops, const tfg_graph* g) {
  if (E < 0 || N < 0) return 0;
  size_t b = align_up(sizeof(float) * (size_t)std::max<int64_t>(N, 1), 256);
  if (!g) {
    const int64_t Ep = E + (add_self_loops ? N : 0);
    b += graph_total_bytes(Ep, N, choose_parts(Ep, N, N, 0));
  }
  return b;
}

int tfg_gcn_norm(const void* edge_index, int index_type, int64_t E, const float* edge_weight,
                 int64_t N, int add_self_loops, const tfg_graph* g, int32_t* out_edge_index,
                 float* out_edge_weight, float* out_edge_weight_csr, float* out_deg, void* ws,
                 size_t ws_bytes, tfg_stream_t stream) {
  if (bad_index_type(index_type)) return fail(TFG_ERR_INVALID_ARG, "bad index type");
  int rc = check_counts(E + (add_self_loops ? N : 0), N, N);
  if (rc) return rc;
  if (E > 0 && edge_index == nullptr) return fail(TFG_ERR_INVALID_ARG, "edge_index is NULL");
  if (int wrc = check_ws(ws, ws_bytes, tfg_gcn_norm_ws_bytes(E, N, add_self_loops, g))) return wrc;
  if (out_edge_weight_csr && !g)
    return fail(TFG_ERR_INVALID_ARG, "CSR-order output needs a graph handle");
  hipStream_t s = as_stream(stream);
  Carver c(ws, ws_bytes);
  float* dinv = static_cast<float*>(c.take(sizeof(float) * (size_t)std::max<int64_t>(N, 1)));
  Graph tmp;
  const Graph* gp = nullptr;
  rc = graph_or_transient(g, tmp, gp, edge_index, tgt_row(edge_index, index_type, E), index_type,
                          E, N, N, add_self_loops, c, s);
  if (rc) return rc;
  rc = launch_gcn_norm(*gp, edge_index, index_type, edge_weight, out_edge_index, out_edge_weight,
                       out_edge_weight_csr, out_deg, dinv, s);
  if (rc) return rc;
  if (!g) TFG_HIP(hipStreamSynchronize(s));  // the transient graph lives in ws
  return TFG_OK;
}

size_t tfg_aggregate_ws_bytes(int64_t E, int64_t N_src, int64_t N, int64_t F, int reduce,
                              const tfg_graph* g) {
  return aggregate_ws_needed(E, N, N_src, F, reduce, g);
}

}  // extern "C"

namespace tfg {
namespace {

// The host-side argument checks of tfg_aggregate and tfg_aggregate_noalloc.
int check_aggregate_args(const void* edge_index, int index_type, int64_t E,
                         const float* edge_weight, int64_t H, int weight_order, const float* x,
                         int64_t N_src, int64_t F, int64_t ldx, int64_t N, int reduce,
                         const tfg_graph* g, const float* out) {
  if (bad_index_type(index_type)) return fail(TFG_ERR_INVALID_ARG, "bad index type");
  int rc = check_counts(E, N, N_src);
  if (rc) return rc;
  if (reduce != TFG_SUM && reduce != TFG_MEAN && reduce != TFG_MAX)
    return fail(TFG_ERR_INVALID_ARG, "bad reduce");
  if (weight_order != TFG_COO && weight_order != TFG_CSR)
    return fail(TFG_ERR_INVALID_ARG, "bad weight order");
  if (F < 0 || H < 1 || (F > 0 && F % H != 0))
    return fail(TFG_ERR_INVALID_ARG, "F must be >= 0 and a multiple of H >= 1");
  if (F >= kMaxCount || ldx < F) return fail(TFG_ERR_INVALID_ARG, "bad F / ldx");
  if (N_src * std::max<int64_t>(ldx, 1) >= (int64_t(1) << 62)) return fail(TFG_ERR_TOO_LARGE, "x too large");
  if (E > 0 && edge_index == nullptr && !g) return fail(TFG_ERR_INVALID_ARG, "edge_index is NULL");
  if (N > 0 && F > 0 && out == nullptr) return fail(TFG_ERR_INVALID_ARG, "out is NULL");
  if (E > 0 && F > 0 && x == nullptr) return fail(TFG_ERR_INVALID_ARG, "x is NULL");
  if (weight_order == TFG_CSR && edge_weight && !g)
    return fail(TFG_ERR_INVALID_ARG, "CSR-order weights need a graph handle");
  (void)edge_weight;
  return TFG_OK;
}

// A handle built with loops describes the E' = E_in + N edges of this list.
int check_handle_sizes(const Graph& g, int64_t E, int64_t N, int64_t N_src) {
  if (g.E != E || g.N != N || g.N_src != N_src)
    return fail(TFG_ERR_INVALID_ARG, "graph handle does not match the edge list sizes");
  return check_device(g);
}

}  // namespace
}  // namespace tfg

extern "C" {

int tfg_aggregate_noalloc(const void* edge_index, int index_type, int64_t E,
                          const float* edge_weight, int64_t H, int weight_order, const float* x,
                          int64_t N_src, int64_t F, int64_t ldx, int64_t N, int reduce,
                          const tfg_graph* g, float* out, int32_t* argmax, tfg_stream_t stream) {
  int rc = check_aggregate_args(edge_index, index_type, E, edge_weight, H, weight_order, x, N_src,
                                F, ldx, N, reduce, g, out);
  if (rc) return rc;
  if (!g) return fail(TFG_ERR_INVALID_ARG, "the no-allocation aggregation needs a graph handle");
  if (H > 1 && !edge_weight) H = 1;
  const Graph& gr = g->g;
  if ((rc = check_handle_sizes(gr, E, N, N_src))) return rc;
  const size_t need = aggregate_partial_bytes(partials_needed(E, N, N_src, F, g), F, reduce);
  if (need > (size_t)TFG_NOALLOC_SCRATCH_BYTES)
    return fail(TFG_ERR_WORKSPACE, "the partial rows of this graph (" + std::to_string(need) +
                                       " bytes) exceed the static scratch (" +
                                       std::to_string((size_t)TFG_NOALLOC_SCRATCH_BYTES) +
                                       " bytes); use tfg_aggregate with a workspace");
  void* part = nullptr;
  if ((rc = noalloc_scratch(&part))) return rc;
  return launch_aggregate(gr, edge_weight, (int)H, weight_order, x, F, ldx, reduce, out, argmax,
                          part, as_stream(stream));
}

int tfg_aggregate(const void* edge_index, int index_type, int64_t E, const float* edge_weight,
                  int64_t H, int weight_order, const float* x, int64_t N_src, int64_t F,
                  int64_t ldx, int64_t N, int reduce, const tfg_graph* g, float* out,
                  int32_t* argmax, void* ws, size_t ws_bytes, tfg_stream_t stream) {
  int rc = check_aggregate_args(edge_index, index_type, E, edge_weight, H, weight_order, x, N_src,
                                F, ldx, N, reduce, g, out);
  if (rc) return rc;
  if (H > 1 && !edge_weight) H = 1;
  if (int wrc = check_ws(ws, ws_bytes, aggregate_ws_needed(E, N, N_src, F, reduce, g))) return wrc;
  hipStream_t s = as_stream(stream);
  Carver c(ws, ws_bytes);
  Graph tmp;
  const Graph* gp = nullptr;
  void* part = c.take(aggregate_partial_bytes(partials_needed(E, N, N_src, F, g), F, reduce));
  if (g) {
    gp = &g->g;
    if ((rc = check_handle_sizes(*gp, E, N, N_src))) return rc;
  } else {
    rc = graph_or_transient(nullptr, tmp, gp, edge_index, tgt_row(edge_index, index_type, E),
                            index_type, E, N_src, N, 0, c, s);
    if (rc) return rc;
  }
  rc = launch_aggregate(*gp, edge_weight, (int)H, weight_order, x, F, ldx, reduce, out, argmax,
                        part, s);
  if (rc) return rc;
  if (!g) TFG_HIP(hipStreamSynchronize(s));
  return TFG_OK;
}

size_t tfg_gat_edge_scores_ws_bytes(int64_t N, int64_t H) {
  if (N < 0 || H < 0) return 0;
  return align_up(sizeof(float) * (size_t)std::max<int64_t>(2 * N * H, 1), 256) + 256;
}

int tfg_gat_edge_scores(const void* edge_index, int index_type, int64_t E, const float* h,
                        int64_t N, int64_t H, int64_t D, const float* a_src, const float* a_dst,
                        float slope, float* out_scores, void* ws, size_t ws_bytes,
                        tfg_stream_t stream) {
  if (bad_index_type(index_type)) return fail(TFG_ERR_INVALID_ARG, "bad index type");
  int rc = check_counts(E, N, N);
  if (rc) return rc;
  if (H < 1 || D < 1 || H * D >= kMaxCount) return fail(TFG_ERR_INVALID_ARG, "bad H / D");
  if ((E > 0 && (edge_index == nullptr || out_scores == nullptr)) ||
      (N > 0 && (h == nullptr || a_src == nullptr || a_dst == nullptr)))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (E > 0 && N == 0) return fail(TFG_ERR_INDEX_RANGE, "edges on a graph without nodes");
  if (int wrc = check_ws(ws, ws_bytes, tfg_gat_edge_scores_ws_bytes(N, H))) return wrc;
  float* proj = static_cast<float*>(ws);
  int* err = reinterpret_cast<int*>(static_cast<char*>(ws) +
                                    align_up(sizeof(float) * (size_t)std::max<int64_t>(2 * N * H, 1), 256));
  return launch_gat_scores(edge_index, index_type, E, h, N, (int)H, (int)D, a_src, a_dst, slope,
                           out_scores, proj, err, as_stream(stream));
}

size_t tfg_segment_softmax_ws_bytes(int64_t E, int64_t H, int64_t N, const tfg_graph* g) {
  if (E < 0 || N < 0 || H < 1) return 0;
  if (g) return row_stats_bytes(g->g.n_heavy, H) + 256;
  // a transient graph, then the statistics of its chunks (at most the plan's capacity)
  const int parts = choose_parts(E, N, 1, 0);
  const int64_t cap = graph_layout(E, N, parts, default_chunk()).cap_heavy;
  return graph_total_bytes(E, N, parts) + row_stats_bytes(cap, H) + 256;
}

int tfg_segment_softmax(const float* scores, int64_t E, int64_t H, const void* seg, int index_type,
                        int64_t N, const tfg_graph* g, float* out, float* out_csr, void* ws,
                        size_t ws_bytes, tfg_stream_t stream) {
  if (bad_index_type(index_type)) return fail(TFG_ERR_INVALID_ARG, "bad index type");
  int rc = check_counts(E, N, 1);
  if (rc) return rc;
  if (H < 1 || E * H >= (int64_t(1) << 62)) return fail(TFG_ERR_INVALID_ARG, "bad H");
  if (E > 0 && (scores == nullptr || out == nullptr)) return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (E > 0 && seg == nullptr && g == nullptr) return fail(TFG_ERR_INVALID_ARG, "seg is NULL");
  if (out_csr && !g) return fail(TFG_ERR_INVALID_ARG, "CSR-order output needs a graph handle");
  if (int wrc = check_ws(ws, ws_bytes, tfg_segment_softmax_ws_bytes(E, H, N, g))) return wrc;
  hipStream_t s = as_stream(stream);
  Carver c(ws, ws_bytes);
  const Graph* gp = nullptr;
  Graph tmp;
  if (g) {
    gp = &g->g;
    if (gp->E != E || gp->N != N) return fail(TFG_ERR_INVALID_ARG, "graph handle does not match");
    if (int e = check_device(*gp)) return e;
  } else {
    rc = graph_or_transient(nullptr, tmp, gp, nullptr, seg, index_type, E, 1, N, 0, c, s);
    if (rc) return rc;
  }
  void* stats = c.take(row_stats_bytes(gp->n_heavy, H));
  rc = launch_segment_softmax(*gp, scores, (int)H, out, out_csr, stats, s);
  if (rc) return rc;
  if (!g) TFG_HIP(hipStreamSynchronize(s));
  return TFG_OK;
}

namespace {

// Checks that g (forward) and gt (transposed, may be NULL) describe one edge list.
int check_backward_graphs(const tfg_graph* g, const tfg_graph* gt) {
  if (!g) return fail(TFG_ERR_INVALID_ARG, "the forward graph is NULL");
  if (g->g.transposed) return fail(TFG_ERR_INVALID_ARG, "g must be a forward graph");
  if (gt) {
    const Graph& a = g->g;
    const Graph& b = gt->g;
    if (!b.transposed) return fail(TFG_ERR_INVALID_ARG, "gt must be a transposed graph");
    if (a.E_in != b.E_in || a.N != b.N_src || a.N_src != b.N || a.loops != b.loops)
      return fail(TFG_ERR_INVALID_ARG, "gt does not transpose g");
  }
  return TFG_OK;
}

}  // namespace

size_t tfg_aggregate_backward_ws_bytes(const tfg_graph* g, const tfg_graph* gt, int64_t F,
                                       int64_t H, int reduce, int weight_order,
                                       int has_edge_weight) {
  if (!g || F < 0 || H < 1) return 0;
  return aggregate_backward_ws_bytes(g->g, gt ? &gt->g : nullptr, F, H, reduce, weight_order,
                                     has_edge_weight != 0);
}

int tfg_aggregate_backward(const tfg_graph* g, const tfg_graph* gt, const float* edge_weight,
                           int64_t H, int weight_order, const float* x, int64_t ldx,
                           const float* dy, int64_t F, int reduce, const int32_t* argmax,
                           float* dx, float* dw, int dw_order, void* ws, size_t ws_bytes,
                           tfg_stream_t stream) {
  int rc = check_backward_graphs(g, gt);
  if (rc) return rc;
  if (reduce != TFG_SUM && reduce != TFG_MEAN && reduce != TFG_MAX)
    return fail(TFG_ERR_INVALID_ARG, "bad reduce");
  if (weight_order != TFG_COO && weight_order != TFG_CSR && weight_order != TFG_CSR_T)
    return fail(TFG_ERR_INVALID_ARG, "bad weight order");
  if (weight_order == TFG_CSR_T && edge_weight != nullptr && gt == nullptr)
    return fail(TFG_ERR_INVALID_ARG, "TFG_CSR_T weights need gt");
  if (dw_order != TFG_COO && dw_order != TFG_CSR)
    return fail(TFG_ERR_INVALID_ARG, "bad dw order");
  if (F < 0 || H < 1 || (F > 0 && F % H != 0) || F >= kMaxCount || H >= kMaxCount)
    return fail(TFG_ERR_INVALID_ARG, "bad F or H");
  const Graph& fg = g->g;
  if (fg.E * H >= kMaxCount) return fail(TFG_ERR_TOO_LARGE, "E * H not below 2^31 - 2^20");
  if (fg.N > 0 && F > 0 && dy == nullptr) return fail(TFG_ERR_INVALID_ARG, "dy is NULL");
  if (dx != nullptr && gt == nullptr) return fail(TFG_ERR_INVALID_ARG, "dx needs gt");
  if (dw != nullptr && fg.N_src > 0 && F > 0 && x == nullptr)
    return fail(TFG_ERR_INVALID_ARG, "dw needs x");
  if (dw != nullptr && ldx < F) return fail(TFG_ERR_INVALID_ARG, "ldx < F");
  if (reduce == TFG_MAX && argmax == nullptr)
    return fail(TFG_ERR_INVALID_ARG, "the max gradient needs the forward argmax");
  const Graph* tg = gt ? &gt->g : nullptr;
  if (int wrc = check_ws(ws, ws_bytes,
                         aggregate_backward_ws_bytes(fg, tg, F, H, reduce, weight_order,
                                                     edge_weight != nullptr)))
    return wrc;
  if (int e = check_device(g)) return e;
  if (int e = check_device(gt)) return e;
  hipStream_t s = as_stream(stream);
  return launch_aggregate_backward(fg, dx ? tg : nullptr, edge_weight, (int)H, weight_order, x,
                                   ldx, dy, F, reduce, argmax, dx, dw, dw_order, ws, s);
}

size_t tfg_segment_softmax_backward_ws_bytes(int64_t E, int64_t H, int64_t N,
                                             const tfg_graph* g) {
  return tfg_segment_softmax_ws_bytes(E, H, N, g);
}

int tfg_segment_softmax_backward(const float* alpha, const float* dalpha, int64_t E, int64_t H,
                                 const void* seg, int index_type, int64_t N, const tfg_graph* g,
                                 float* dscores, void* ws, size_t ws_bytes, tfg_stream_t stream) {
  if (bad_index_type(index_type)) return fail(TFG_ERR_INVALID_ARG, "bad index type");
  int rc = check_counts(E, N, 1);
  if (rc) return rc;
  if (H < 1 || E * H >= (int64_t(1) << 62)) return fail(TFG_ERR_INVALID_ARG, "bad H");
  if (E > 0 && (alpha == nullptr || dalpha == nullptr || dscores == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (E > 0 && seg == nullptr && g == nullptr) return fail(TFG_ERR_INVALID_ARG, "seg is NULL");
  if (int wrc = check_ws(ws, ws_bytes, tfg_segment_softmax_backward_ws_bytes(E, H, N, g))) return wrc;
  hipStream_t s = as_stream(stream);
  Carver c(ws, ws_bytes);
  const Graph* gp = nullptr;
  Graph tmp;
  if (g) {
    gp = &g->g;
    if (gp->transposed || gp->E != E || gp->N != N)
      return fail(TFG_ERR_INVALID_ARG, "graph handle does not match");
    if (int e = check_device(*gp)) return e;
  } else {
    rc = graph_or_transient(nullptr, tmp, gp, nullptr, seg, index_type, E, 1, N, 0, c, s);
    if (rc) return rc;
  }
  void* stats = c.take(row_stats_bytes(gp->n_heavy, H));
  rc = launch_segment_softmax_backward(*gp, alpha, dalpha, (int)H, dscores, stats, s);
  if (rc) return rc;
  if (!g) TFG_HIP(hipStreamSynchronize(s));
  return TFG_OK;
}

size_t tfg_segment_pool_ws_bytes(int64_t Nb, int64_t G) {
  (void)Nb;
  if (G < 0) return 0;
  return align_up(sizeof(int) * (size_t)(G + 1), 256) + 256;
}

int tfg_segment_pool(const float* x, int64_t Nb, int64_t F, int64_t ldx, const void* graph_index,
                     int index_type, int64_t G, int reduce, float* out, int32_t* argmax,
                     int validate, void* ws, size_t ws_bytes, tfg_stream_t stream) {
  if (bad_index_type(index_type)) return fail(TFG_ERR_INVALID_ARG, "bad index type");
  int rc = check_counts(0, Nb, 0);
  if (rc) return rc;
  if (G < 0 || G >= kMaxCount) return fail(TFG_ERR_INVALID_ARG, "bad G");
  if (F < 0 || F >= kMaxCount || ldx < F) return fail(TFG_ERR_INVALID_ARG, "bad F / ldx");
  if (reduce != TFG_SUM && reduce != TFG_MEAN && reduce != TFG_MAX)
    return fail(TFG_ERR_INVALID_ARG, "bad reduce");
  if ((Nb > 0 && (graph_index == nullptr || (F > 0 && x == nullptr))) ||
      (G > 0 && F > 0 && out == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (int wrc = check_ws(ws, ws_bytes, tfg_segment_pool_ws_bytes(Nb, G))) return wrc;
  hipStream_t s = as_stream(stream);
  int* goff = static_cast<int*>(ws);
  int* err = reinterpret_cast<int*>(static_cast<char*>(ws) + align_up(sizeof(int) * (size_t)(G + 1), 256));
  rc = launch_segment_pool(x, Nb, F, ldx, graph_index, index_type, G, reduce, out, argmax, goff, err, s);
  if (rc) return rc;
  if (validate) {
    int flags = 0;
    const int* from[1] = {err};
    if (int rrc = read_back(s, 1, from, &flags)) return rrc;
    if (flags & kErrIndex) return fail(TFG_ERR_INDEX_RANGE, "graph_index holds an id outside [0, G)");
    if (flags & kErrUnsorted) return fail(TFG_ERR_UNSORTED, "graph_index is not non-decreasing");
  }
  return TFG_OK;
}

int tfg_segment_pool_backward(const float* dy, int64_t G, int64_t F, const void* graph_index,
                              int index_type, int64_t Nb, int reduce, const int32_t* argmax,
                              float* dx, int64_t ldx, int validate, void* ws, size_t ws_bytes,
                              tfg_stream_t stream) {
  if (bad_index_type(index_type)) return fail(TFG_ERR_INVALID_ARG, "bad index type");
  int rc = check_counts(0, Nb, 0);
  if (rc) return rc;
  if (G < 0 || G >= kMaxCount) return fail(TFG_ERR_INVALID_ARG, "bad G");
  if (F < 0 || F >= kMaxCount || ldx < F) return fail(TFG_ERR_INVALID_ARG, "bad F / ldx");
  if (reduce != TFG_SUM && reduce != TFG_MEAN && reduce != TFG_MAX)
    return fail(TFG_ERR_INVALID_ARG, "bad reduce");
  if (Nb > 0 && F > 0 && (graph_index == nullptr || dx == nullptr || (G > 0 && dy == nullptr)))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (reduce == TFG_MAX && Nb > 0 && F > 0 && G > 0 && argmax == nullptr)
    return fail(TFG_ERR_INVALID_ARG, "the max gradient needs the forward argmax");
  if (int wrc = check_ws(ws, ws_bytes, tfg_segment_pool_ws_bytes(Nb, G))) return wrc;
  hipStream_t s = as_stream(stream);
  int* goff = static_cast<int*>(ws);
  int* err = reinterpret_cast<int*>(static_cast<char*>(ws) + align_up(sizeof(int) * (size_t)(G + 1), 256));
  rc = launch_segment_pool_backward(dy, G, F, graph_index, index_type, Nb, reduce, argmax, dx, ldx,
                                    goff, err, s);
  if (rc) return rc;
  if (validate) {
    int flags = 0;
    const int* from[1] = {err};
    if (int rrc = read_back(s, 1, from, &flags)) return rrc;
    if (flags & kErrIndex) return fail(TFG_ERR_INDEX_RANGE, "graph_index holds an id outside [0, G)");
    if (flags & kErrUnsorted) return fail(TFG_ERR_UNSORTED, "graph_index is not non-decreasing");
  }
  return TFG_OK;
}

size_t tfg_batch_graphs_ws_bytes(int64_t G) { return G < 0 ? 0 : batch_ws_bytes(G); }

int tfg_batch_graphs(int64_t G, const void* node_counts, const void* edge_counts,
                     const void* local_edge_index, int index_type, int64_t E, int64_t Nb,
                     void* out_edge_index, void* out_graph_index, int32_t* out_node_offsets,
                     int32_t* out_edge_offsets, int validate, void* ws, size_t ws_bytes,
                     tfg_stream_t stream) {
  if (bad_index_type(index_type)) return fail(TFG_ERR_INVALID_ARG, "bad index type");
  int rc = check_counts(E, Nb, 0);
  if (rc) return rc;
  if (G < 0 || G >= kMaxCount) return fail(TFG_ERR_INVALID_ARG, "bad G");
  if (G == 0 && (E > 0 || Nb > 0)) return fail(TFG_ERR_INVALID_ARG, "edges or nodes without graphs");
  if (G > 0 && (node_counts == nullptr || edge_counts == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL counts");
  if ((E > 0 && (local_edge_index == nullptr || out_edge_index == nullptr)) ||
      (Nb > 0 && out_graph_index == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (int wrc = check_ws(ws, ws_bytes, batch_ws_bytes(G))) return wrc;
  hipStream_t s = as_stream(stream);
  Carver c(ws, ws_bytes);
  int* node_off = static_cast<int*>(c.take(sizeof(int) * (size_t)(G + 1)));
  int* edge_off = static_cast<int*>(c.take(sizeof(int) * (size_t)(G + 1)));
  int* sums = static_cast<int*>(c.take(sizeof(int) * (size_t)std::max<int64_t>((G + 1 + 2047) / 2048, 1)));
  int* err = static_cast<int*>(c.take(sizeof(int)));
  if (G == 0) return TFG_OK;
  rc = launch_batch_graphs(G, node_counts, edge_counts, local_edge_index, index_type, E, Nb,
                           out_edge_index, out_graph_index, node_off, edge_off, out_node_offsets,
                           out_edge_offsets, sums, err, s);
  if (rc) return rc;
  if (validate) {
    int host[3] = {0, 0, 0};
    const int* from[3] = {err, node_off + G, edge_off + G};
    if (int rrc = read_back(s, 3, from, host)) return rrc;
    if (host[0] & kErrIndex) return fail(TFG_ERR_INDEX_RANGE, "a count or local id is out of range");
    if (host[1] != Nb || host[2] != E)
      return fail(TFG_ERR_INDEX_RANGE, "node / edge counts do not add up to Nb / E");
  }
  return TFG_OK;
}

int tfg_batch_graphs_totals(int64_t G, const void* node_counts, const void* edge_counts,
                            int index_type, void* ws, size_t ws_bytes, tfg_stream_t stream,
                            int64_t* Nb, int64_t* E) {
  if (bad_index_type(index_type)) return fail(TFG_ERR_INVALID_ARG, "bad index type");
  if (G < 0 || G >= kMaxCount) return fail(TFG_ERR_INVALID_ARG, "bad G");
  if (Nb == nullptr || E == nullptr) return fail(TFG_ERR_INVALID_ARG, "NULL result pointer");
  if (G > 0 && (node_counts == nullptr || edge_counts == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL counts");
  if (int wrc = check_ws(ws, ws_bytes, batch_ws_bytes(G))) return wrc;
  *Nb = 0;
  *E = 0;
  if (G == 0) return TFG_OK;
  hipStream_t s = as_stream(stream);
  int* out = static_cast<int*>(ws);
  if (int rc = launch_batch_totals(G, node_counts, edge_counts, index_type, out, s)) return rc;
  int host[5];
  const int* from[5] = {out, out + 1, out + 2, out + 3, out + 4};
  if (int rrc = read_back(s, 5, from, host)) return rrc;
  if (host[4] & kErrIndex) return fail(TFG_ERR_INDEX_RANGE, "a node or edge count is negative");
  *Nb = (int64_t)(uint32_t)host[0] | ((int64_t)host[1] << 32);
  *E = (int64_t)(uint32_t)host[2] | ((int64_t)host[3] << 32);
  return TFG_OK;
}

size_t tfg_propagate_ws_bytes(const tfg_graph* g, int64_t F, int64_t K) {
  if (!g || F < 0 || K < 0) return 0;
  const Graph& gr = g->g;
  size_t b = aggregate_partial_bytes(partials_needed(gr.E, gr.N, gr.N_src, F, g), F, TFG_SUM);
  if (K >= 2) b += align_up(sizeof(float) * (size_t)(gr.N * F), 256);
  return b + 256;
}

int tfg_propagate(const tfg_graph* g, const float* edge_weight, int weight_order, const float* x,
                  int64_t F, int64_t ldx, int64_t K, float alpha, const float* h, int64_t ldh,
                  float* out, void* ws, size_t ws_bytes, tfg_stream_t stream) {
  if (!g) return fail(TFG_ERR_INVALID_ARG, "graph is NULL");
  const Graph& gr = g->g;
  if (gr.N != gr.N_src) return fail(TFG_ERR_INVALID_ARG, "propagation needs a square graph");
  if (F < 0 || F >= kMaxCount || ldx < F || K < 0)
    return fail(TFG_ERR_INVALID_ARG, "bad F / ldx / K");
  if (weight_order != TFG_COO && weight_order != TFG_CSR)
    return fail(TFG_ERR_INVALID_ARG, "bad weight order");
  if (!(alpha >= 0.0f && alpha <= 1.0f)) return fail(TFG_ERR_INVALID_ARG, "alpha outside [0, 1]");
  if (alpha != 0.0f && (h == nullptr || ldh < F))
    return fail(TFG_ERR_INVALID_ARG, "alpha > 0 needs h with ldh >= F");
  if (gr.N > 0 && F > 0 && (x == nullptr || out == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (int wrc = check_ws(ws, ws_bytes, tfg_propagate_ws_bytes(g, F, K))) return wrc;
  if (int e = check_device(gr)) return e;
  hipStream_t s = as_stream(stream);
  if (gr.N == 0 || F == 0) return TFG_OK;
  if (K == 0) {
    TFG_HIP(hipMemcpy2DAsync(out, sizeof(float) * F, x, sizeof(float) * ldx, sizeof(float) * F,
                             gr.N, hipMemcpyDeviceToDevice, s));
    return TFG_OK;
  }
  Carver c(ws, ws_bytes);
  void* part = c.take(aggregate_partial_bytes(partials_needed(gr.E, gr.N, gr.N_src, F, g), F,
                                              TFG_SUM));
  float* tmp = K >= 2 ? static_cast<float*>(c.take(sizeof(float) * (size_t)(gr.N * F))) : nullptr;
  const float* hh = alpha != 0.0f ? h : nullptr;
  // step k writes Z_{k+1}; the buffers alternate so that Z_K lands in out
  for (int64_t k = 0; k < K; ++k) {
    const float* in = k == 0 ? x : ((K - k) % 2 == 0 ? out : tmp);
    const int64_t ld_in = k == 0 ? ldx : F;
    float* dst = (K - (k + 1)) % 2 == 0 ? out : tmp;
    int rc = launch_aggregate(gr, edge_weight, 1, weight_order, in, F, ld_in, TFG_SUM, dst,
                              nullptr, part, s, 1.0f - alpha, alpha, hh, ldh);
    if (rc) return rc;
  }
  return TFG_OK;
}

size_t tfg_gat_aggregate_ws_bytes(const tfg_graph* g, int64_t H, int64_t D) {
  if (!g || H < 1 || D < 1) return 0;
  return gat_aggregate_ws_bytes(g->g, H, D);
}

int tfg_gat_aggregate(const tfg_graph* g, const float* h, int64_t H, int64_t D,
                      const float* a_src, const float* a_dst, float slope, float* out,
                      float* alpha_out, void* ws, size_t ws_bytes, tfg_stream_t stream) {
  if (!g) return fail(TFG_ERR_INVALID_ARG, "graph is NULL");
  const Graph& gr = g->g;
  if (gr.N != gr.N_src) return fail(TFG_ERR_INVALID_ARG, "attention needs a square graph");
  if (H < 1 || H > max_fused_heads() || D < 1 || H * D >= kMaxCount)
    return fail(TFG_ERR_INVALID_ARG, "need 1 <= H <= 64 and D >= 1");
  if (gr.N > 0 && (h == nullptr || a_src == nullptr || a_dst == nullptr || out == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (int wrc = check_ws(ws, ws_bytes, gat_aggregate_ws_bytes(gr, H, D))) return wrc;
  if (int e = check_device(gr)) return e;
  return launch_gat_aggregate(gr, h, (int)H, (int)D, a_src, a_dst, slope, out, alpha_out, ws,
                              as_stream(stream));
}

size_t tfg_gat_dot_aggregate_ws_bytes(const tfg_graph* g, int64_t H, int64_t D) {
  return tfg_gat_aggregate_ws_bytes(g, H, D);
}

int tfg_gat_dot_aggregate(const tfg_graph* g, const float* q, const float* key, const float* v,
                          int64_t H, int64_t D, float scale, float* out, float* alpha_out,
                          void* ws, size_t ws_bytes, tfg_stream_t stream) {
  if (!g) return fail(TFG_ERR_INVALID_ARG, "graph is NULL");
  const Graph& gr = g->g;
  if (H < 1 || H > max_fused_heads() || !dot_attention_shape_ok(D))
    return fail(TFG_ERR_INVALID_ARG, "need 1 <= H <= 64 and D a power of two <= 64");
  if (gr.N > 0 && (q == nullptr || out == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (gr.E > 0 && (key == nullptr || v == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (int wrc = check_ws(ws, ws_bytes, gat_aggregate_ws_bytes(gr, H, D))) return wrc;
  if (int e = check_device(gr)) return e;
  return launch_gat_dot_aggregate(gr, q, key, v, (int)H, (int)D, scale, out, alpha_out, ws,
                                  as_stream(stream));
}

int tfg_edge_dot_scores(const tfg_graph* g, const float* q, const float* key, int64_t H,
                        int64_t D, float scale, float* out_scores, int order,
                        tfg_stream_t stream) {
  if (!g) return fail(TFG_ERR_INVALID_ARG, "graph is NULL");
  const Graph& gr = g->g;
  if (H < 1 || D < 1 || H * D >= kMaxCount || gr.E * H >= kMaxCount)
    return fail(TFG_ERR_INVALID_ARG, "bad H or D");
  if (order != TFG_COO && order != TFG_CSR) return fail(TFG_ERR_INVALID_ARG, "bad order");
  if (gr.E > 0 && (q == nullptr || key == nullptr || out_scores == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (int e = check_device(gr)) return e;
  return launch_edge_dot(gr, q, key, H * D, H * D, (int)H, scale, out_scores,
                         order == TFG_COO ? 1 : 0, as_stream(stream));
}

size_t tfg_gat_graph_scores_ws_bytes(const tfg_graph* g, int64_t H) {
  if (!g || H < 1) return 0;
  return tfg_gat_edge_scores_ws_bytes(g->g.N, H);
}

int tfg_gat_graph_scores(const tfg_graph* g, const float* h, int64_t H, int64_t D,
                         const float* a_src, const float* a_dst, float slope, float* out_scores,
                         int order, void* ws, size_t ws_bytes, tfg_stream_t stream) {
  if (!g) return fail(TFG_ERR_INVALID_ARG, "graph is NULL");
  const Graph& gr = g->g;
  if (gr.transposed || gr.N_src != gr.N)
    return fail(TFG_ERR_INVALID_ARG,
                "scores need a forward graph whose sources and targets are one node set");
  if (H < 1 || D < 1 || H * D >= kMaxCount || gr.E * H >= kMaxCount)
    return fail(TFG_ERR_INVALID_ARG, "bad H or D");
  if (order != TFG_COO && order != TFG_CSR) return fail(TFG_ERR_INVALID_ARG, "bad order");
  if ((gr.E > 0 && out_scores == nullptr) ||
      (gr.N > 0 && (h == nullptr || a_src == nullptr || a_dst == nullptr)))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (int wrc = check_ws(ws, ws_bytes, tfg_gat_graph_scores_ws_bytes(g, H))) return wrc;
  if (int e = check_device(gr)) return e;
  return launch_gat_graph_scores(gr, h, (int)H, (int)D, a_src, a_dst, slope, out_scores,
                                 order == TFG_COO ? 1 : 0, static_cast<float*>(ws),
                                 as_stream(stream));
}

size_t tfg_segment_softmax_graph_ws_bytes(const tfg_graph* g, int64_t H) {
  if (!g || H < 1) return 0;
  return row_stats_bytes(g->g.n_heavy, H) + 256;
}

int tfg_segment_softmax_graph(const tfg_graph* g, const float* scores, int64_t H, int order,
                              float* out, void* ws, size_t ws_bytes, tfg_stream_t stream) {
  if (!g) return fail(TFG_ERR_INVALID_ARG, "graph is NULL");
  const Graph& gr = g->g;
  if (H < 1 || gr.E * H >= (int64_t(1) << 62)) return fail(TFG_ERR_INVALID_ARG, "bad H");
  if (order != TFG_COO && order != TFG_CSR) return fail(TFG_ERR_INVALID_ARG, "bad order");
  if (gr.E > 0 && (scores == nullptr || out == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (int wrc = check_ws(ws, ws_bytes, tfg_segment_softmax_graph_ws_bytes(g, H))) return wrc;
  if (int e = check_device(gr)) return e;
  return launch_segment_softmax(gr, scores, (int)H, out, nullptr, ws, as_stream(stream),
                                order == TFG_CSR);
}

int tfg_segment_softmax_graph_backward(const tfg_graph* g, const float* alpha,
                                       const float* dalpha, int64_t H, int order, float* dscores,
                                       void* ws, size_t ws_bytes, tfg_stream_t stream) {
  if (!g) return fail(TFG_ERR_INVALID_ARG, "graph is NULL");
  const Graph& gr = g->g;
  if (gr.transposed) return fail(TFG_ERR_INVALID_ARG, "g must be a forward graph");
  if (H < 1 || gr.E * H >= (int64_t(1) << 62)) return fail(TFG_ERR_INVALID_ARG, "bad H");
  if (order != TFG_COO && order != TFG_CSR) return fail(TFG_ERR_INVALID_ARG, "bad order");
  if (gr.E > 0 && (alpha == nullptr || dalpha == nullptr || dscores == nullptr))
    return fail(TFG_ERR_INVALID_ARG, "NULL pointer");
  if (int wrc = check_ws(ws, ws_bytes, tfg_segment_softmax_graph_ws_bytes(g, H))) return wrc;
  if (int e = check_device(gr)) return e;
  return launch_segment_softmax_backward(gr, alpha, dalpha, (int)H, dscores, ws,
                                         as_stream(stream), order == TFG_CSR);
}

}  // extern "C"

