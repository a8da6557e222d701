// BatchGraph construction on the GPU (gfx950): node and edge offsets from the
// per-graph counts (exclusive scans), every local edge id shifted by its
// graph's node offset, and the node -> graph index. Each edge and node finds
// its graph by binary search over the offsets (G + 1 entries, L2 resident).
// Up to 16,383 graphs the offsets come from one block and the edges and nodes
// from one more launch; larger batches use the device-wide scan.
#include "wave.h"

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

constexpr int kSmallThreads = 1024;
constexpr int kSmallItems = 16;
constexpr int64_t kSmallMax = (int64_t)kSmallThreads * kSmallItems;  // G + 1 entries at most

// Both offset arrays of up to kSmallMax - 1 graphs in one block: thread i
// holds entries [16 i, 16 i + 16), sums them, and a block scan gives its start.
// Also clears the error word (every later check of the launch ORs into it).
template <typename IdxT>
__global__ __launch_bounds__(kSmallThreads) void batch_offsets_small(
    const IdxT* __restrict__ nodes, const IdxT* __restrict__ edges, int64_t G,
    int* __restrict__ node_off, int* __restrict__ edge_off, int* __restrict__ out_node_off,
    int* __restrict__ out_edge_off, int* __restrict__ err) {
  __shared__ int tmp[kSmallThreads / kWave];
  const int64_t base = (int64_t)threadIdx.x * kSmallItems;
  int nv[kSmallItems], ev[kSmallItems];
  int ns = 0, es = 0;
  bool bad = false;
#pragma unroll
  for (int i = 0; i < kSmallItems; ++i) {
    const int64_t g = base + i;
    int64_t n = 0, e = 0;
    if (g < G) {
      n = (int64_t)nodes[g];
      e = (int64_t)edges[g];
    }
    const bool b = n < 0 || e < 0 || n >= (int64_t(1) << 31) || e >= (int64_t(1) << 31);
    bad |= b;
    nv[i] = b ? 0 : (int)n;
    ev[i] = b ? 0 : (int)e;
    ns += nv[i];
    es += ev[i];
  }
  const bool any_bad = __syncthreads_or(bad);
  int nrun = block_excl_scan<kSmallThreads / kWave>(ns, tmp, nullptr);
  int erun = block_excl_scan<kSmallThreads / kWave>(es, tmp, nullptr);
#pragma unroll
  for (int i = 0; i < kSmallItems; ++i) {
    const int64_t g = base + i;
    if (g <= G) {
      node_off[g] = nrun;
      edge_off[g] = erun;
      if (out_node_off) out_node_off[g] = nrun;
      if (out_edge_off) out_edge_off[g] = erun;
    }
    nrun += nv[i];
    erun += ev[i];
  }
  if (threadIdx.x == 0) *err = any_bad ? kErrIndex : 0;
}

// Totals of both count arrays (one block, 64-bit sums): out[0..1] = the node
// total as (low, high) 32-bit halves, out[2..3] the edge total, out[4] the
// error flag (a negative count). The caller reads the five ints back.
constexpr int kTotalThreads = 1024;
template <typename IdxT>
__global__ __launch_bounds__(kTotalThreads) void count_totals(const IdxT* __restrict__ nodes,
                                                              const IdxT* __restrict__ edges,
                                                              int64_t G, int* __restrict__ out) {
  __shared__ long long part[2][kTotalThreads / kWave];
  long long ns = 0, es = 0;
  bool bad = false;
  for (int64_t g = threadIdx.x; g < G; g += kTotalThreads) {
    const long long n = (long long)nodes[g], e = (long long)edges[g];
    bad |= n < 0 || e < 0;
    ns += n;
    es += e;
  }
  const bool any_bad = __syncthreads_or(bad);
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) {
    ns += __shfl_down(ns, off);
    es += __shfl_down(es, off);
  }
  const int wave = threadIdx.x / kWave;
  if (lane_id() == 0) {
    part[0][wave] = ns;
    part[1][wave] = es;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    long long tn = 0, te = 0;
    for (int w = 0; w < kTotalThreads / kWave; ++w) {
      tn += part[0][w];
      te += part[1][w];
    }
    out[0] = (int)(unsigned)(tn & 0xffffffffll);
    out[1] = (int)(tn >> 32);
    out[2] = (int)(unsigned)(te & 0xffffffffll);
    out[3] = (int)(te >> 32);
    out[4] = any_bad ? kErrIndex : 0;
  }
}

// Edges and nodes in one launch: thread i reindexes edge i and labels node i.
template <typename IdxT>
__global__ __launch_bounds__(kBlock) void batch_fill(const IdxT* __restrict__ src,
                                                     const IdxT* __restrict__ tgt, int64_t E,
                                                     int64_t Nb, int64_t G,
                                                     const int* __restrict__ node_off,
                                                     const int* __restrict__ edge_off,
                                                     IdxT* __restrict__ out_src,
                                                     IdxT* __restrict__ out_tgt,
                                                     IdxT* __restrict__ gi,
                                                     int* __restrict__ err) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < E) {
    const int g = graph_of(edge_off, G, i);
    const int64_t off = node_off[g], n = (int64_t)node_off[g + 1] - off;
    const int64_t s = (int64_t)src[i], t = (int64_t)tgt[i];
    if (s < 0 || s >= n || t < 0 || t >= n) atomicOr(err, kErrIndex);
    out_src[i] = (IdxT)(s + off);
    out_tgt[i] = (IdxT)(t + off);
  }
  if (i < Nb) gi[i] = (IdxT)graph_of(node_off, G, i);
}

template <typename IdxT>
int launch_small(int64_t G, const void* node_counts, const void* edge_counts,
                 const void* local_edge_index, int64_t E, int64_t Nb, void* out_edge_index,
                 void* out_graph_index, int* node_off, int* edge_off, int* out_node_off,
                 int* out_edge_off, int* err, hipStream_t s) {
  batch_offsets_small<IdxT><<<1, kSmallThreads, 0, s>>>(
      static_cast<const IdxT*>(node_counts), static_cast<const IdxT*>(edge_counts), G, node_off,
      edge_off, out_node_off, out_edge_off, err);
  TFG_LAUNCHED("batch_offsets_small");
  const int64_t n = std::max(E, Nb);
  if (n > 0) {
    const IdxT* ei = static_cast<const IdxT*>(local_edge_index);
    IdxT* oi = static_cast<IdxT*>(out_edge_index);
    batch_fill<IdxT><<<(unsigned)((n + kBlock - 1) / kBlock), kBlock, 0, s>>>(
        ei, ei + E, E, Nb, G, node_off, edge_off, oi, oi + E, static_cast<IdxT*>(out_graph_index),
        err);
    TFG_LAUNCHED("batch_fill");
  }
  return TFG_OK;
}

}  // namespace

int launch_batch_totals(int64_t G, const void* node_counts, const void* edge_counts,
                        int index_type, int* out, hipStream_t s) {
  if (index_type == TFG_I64)
    count_totals<int64_t><<<1, kTotalThreads, 0, s>>>(static_cast<const int64_t*>(node_counts),
                                                       static_cast<const int64_t*>(edge_counts),
                                                       G, out);
  else
    count_totals<int32_t><<<1, kTotalThreads, 0, s>>>(static_cast<const int32_t*>(node_counts),
                                                       static_cast<const int32_t*>(edge_counts),
                                                       G, out);
  TFG_LAUNCHED("count_totals");
  return TFG_OK;
}

size_t batch_ws_bytes(int64_t G) {
  const int64_t tiles = (G + 1 + 2047) / 2048;
  return 2 * align_up(sizeof(int) * (size_t)(G + 1), 256) +
         align_up(sizeof(int) * (size_t)std::max<int64_t>(tiles, 1), 256) + 256;
}

int launch_batch_graphs(int64_t G, const void* node_counts, const void* edge_counts,
                        const void* local_edge_index, int index_type, int64_t E, int64_t Nb,
                        void* out_edge_index, void* out_graph_index, int* node_off, int* edge_off,
                        int* out_node_off, int* out_edge_off, int* sums, int* err,
                        hipStream_t s) {
  if (G + 1 <= kSmallMax) {
    if (index_type == TFG_I64)
      return launch_small<int64_t>(G, node_counts, edge_counts, local_edge_index, E, Nb,
                                   out_edge_index, out_graph_index, node_off, edge_off,
                                   out_node_off, out_edge_off, err, s);
    return launch_small<int32_t>(G, node_counts, edge_counts, local_edge_index, E, Nb,
                                 out_edge_index, out_graph_index, node_off, edge_off, out_node_off,
                                 out_edge_off, err, s);
  }
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
  if (out_node_off)
    TFG_HIP(hipMemcpyAsync(out_node_off, node_off, sizeof(int) * (G + 1), hipMemcpyDeviceToDevice,
                           s));
  if (out_edge_off)
    TFG_HIP(hipMemcpyAsync(out_edge_off, edge_off, sizeof(int) * (G + 1), hipMemcpyDeviceToDevice,
                           s));
  return TFG_OK;
}

}  // namespace tfg
