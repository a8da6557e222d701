// BatchGraph construction on the GPU (gfx950): node and edge offsets from the
// per-graph counts (exclusive scans), every local edge id shifted by its
// graph's node offset, and the node -> graph index. Each edge and node finds
// its graph by binary search over the offsets (G + 1 entries, L2 resident).
#include "tfg_internal.h"

namespace tfg {
namespace {

template <typename IdxT>
__global__ __launch_bounds__(kBlock) void counts_to_int(const IdxT* __restrict__ nodes,
                                                        const IdxT* __restrict__ edges, int64_t G,
                                                        int* __restrict__ node_off,
                                                        int* __restrict__ edge_off,
                                                        int* __restrict__ err) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g > G) return;
  if (g == G) {  // the scans turn this trailing 0 into the totals
    node_off[G] = 0;
    edge_off[G] = 0;
    return;
  }
  const int64_t n = (int64_t)nodes[g], e = (int64_t)edges[g];
  const bool bad = n < 0 || e < 0 || n >= (int64_t(1) << 31) || e >= (int64_t(1) << 31);
  if (bad) atomicOr(err, kErrIndex);
  node_off[g] = bad ? 0 : (int)n;
  edge_off[g] = bad ? 0 : (int)e;
}

// Last graph whose offset is <= v (offsets non-decreasing, off[0] = 0).
__device__ __forceinline__ int graph_of(const int* __restrict__ off, int64_t G, int64_t v) {
  int64_t lo = 0, hi = G;  // invariant: off[lo] <= v, answer in [lo, hi)
  while (hi - lo > 1) {
    const int64_t mid = (lo + hi) >> 1;
    if ((int64_t)off[mid] <= v) lo = mid; else hi = mid;
  }
  return (int)lo;
}

template <typename IdxT>
__global__ __launch_bounds__(kBlock) void reindex_edges(const IdxT* __restrict__ src,
                                                        const IdxT* __restrict__ tgt,
                                                        int64_t E, int64_t G,
                                                        const int* __restrict__ node_off,
                                                        const int* __restrict__ edge_off,
                                                        IdxT* __restrict__ out_src,
                                                        IdxT* __restrict__ out_tgt,
                                                        int* __restrict__ err) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const int g = graph_of(edge_off, G, e);
  const int64_t off = node_off[g], n = (int64_t)node_off[g + 1] - off;
  const int64_t s = (int64_t)src[e], t = (int64_t)tgt[e];
  if (s < 0 || s >= n || t < 0 || t >= n) atomicOr(err, kErrIndex);
  out_src[e] = (IdxT)(s + off);
  out_tgt[e] = (IdxT)(t + off);
}

template <typename IdxT>
__global__ __launch_bounds__(kBlock) void fill_graph_index(int64_t Nb, int64_t G,
                                                           const int* __restrict__ node_off,
                                                           IdxT* __restrict__ gi) {
  const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n < Nb) gi[n] = (IdxT)graph_of(node_off, G, n);
}

__global__ void zero_flag(int* __restrict__ p) { *p = 0; }

}  // namespace

size_t batch_ws_bytes(int64_t G) {
  const int64_t tiles = (G + 1 + 2047) / 2048;
  return 2 * align_up(sizeof(int) * (size_t)(G + 1), 256) +
         align_up(sizeof(int) * (size_t)std::max<int64_t>(tiles, 1), 256) + 256;
}

int launch_batch_graphs(int64_t G, const void* node_counts, const void* edge_counts,
                        const void* local_edge_index, int index_type, int64_t E, int64_t Nb,
                        void* out_edge_index, void* out_graph_index, int* node_off, int* edge_off,
                        int* sums, int* err, hipStream_t s) {
  zero_flag<<<1, 1, 0, s>>>(err);
  const unsigned gb = (unsigned)((G + 1 + kBlock - 1) / kBlock);
  const unsigned eb = (unsigned)((E + kBlock - 1) / kBlock);
  const unsigned nb = (unsigned)((Nb + kBlock - 1) / kBlock);
  if (index_type == TFG_I64) {
    counts_to_int<int64_t><<<gb, kBlock, 0, s>>>(static_cast<const int64_t*>(node_counts),
                                                  static_cast<const int64_t*>(edge_counts), G,
                                                  node_off, edge_off, err);
  } else {
    counts_to_int<int32_t><<<gb, kBlock, 0, s>>>(static_cast<const int32_t*>(node_counts),
                                                  static_cast<const int32_t*>(edge_counts), G,
                                                  node_off, edge_off, err);
  }
  TFG_LAUNCHED("counts_to_int");
  int rc = exclusive_scan(node_off, node_off, G + 1, sums, s);
  if (rc) return rc;
  rc = exclusive_scan(edge_off, edge_off, G + 1, sums, s);
  if (rc) return rc;
  if (index_type == TFG_I64) {
    const int64_t* ei = static_cast<const int64_t*>(local_edge_index);
    int64_t* oi = static_cast<int64_t*>(out_edge_index);
    if (E > 0)
      reindex_edges<int64_t><<<eb, kBlock, 0, s>>>(ei, ei + E, E, G, node_off, edge_off, oi,
                                                     oi + E, err);
    if (Nb > 0)
      fill_graph_index<int64_t><<<nb, kBlock, 0, s>>>(Nb, G, node_off,
                                                       static_cast<int64_t*>(out_graph_index));
  } else {
    const int32_t* ei = static_cast<const int32_t*>(local_edge_index);
    int32_t* oi = static_cast<int32_t*>(out_edge_index);
    if (E > 0)
      reindex_edges<int32_t><<<eb, kBlock, 0, s>>>(ei, ei + E, E, G, node_off, edge_off, oi,
                                                     oi + E, err);
    if (Nb > 0)
      fill_graph_index<int32_t><<<nb, kBlock, 0, s>>>(Nb, G, node_off,
                                                       static_cast<int32_t*>(out_graph_index));
  }
  TFG_LAUNCHED("reindex_edges / fill_graph_index");
  return TFG_OK;
}

}  // namespace tfg
