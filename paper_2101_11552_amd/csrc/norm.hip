// GCN normalisation on the CSR-by-target graph (gfx950):
//   deg[t]  = sum of the weights entering t (loops included when appended)
//   dinv[t] = deg > 0 ? 1 / sqrt(deg) : 0         (IEEE sqrt, IEEE divide)
//   w'[e]   = (dinv[src] * w[e]) * dinv[tgt]       (float32, left to right)
// written in the caller's COO order and/or in the graph's CSR order; both
// orders use the same operands in the same order, so they are bit-identical.
#include "wave.h"

namespace tfg {
namespace {

// Weight of edge id e in the list with appended loops.
__device__ __forceinline__ float edge_w(const float* __restrict__ w, int64_t E_in, int64_t e) {
  return (w == nullptr || e >= E_in) ? 1.0f : w[e];
}

// Unit weights: the degree is the row length (exact in float32 below 2^24,
// and rounded once above it).
__global__ __launch_bounds__(kBlock) void degree_unit(const int* __restrict__ rowptr, int64_t N,
                                                      float* __restrict__ deg,
                                                      float* __restrict__ dinv) {
  int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= N) return;
  float d = (float)(rowptr[t + 1] - rowptr[t]);
  if (deg) deg[t] = d;
  dinv[t] = d > 0.0f ? 1.0f / sqrtf(d) : 0.0f;
}

// General weights: one wavefront per row, each lane summing a strided part of
// the row in double, then a fixed-order tree across the lanes.
__global__ __launch_bounds__(kBlock) void degree_weighted(const int* __restrict__ rowptr,
                                                          const int* __restrict__ perm,
                                                          const float* __restrict__ w,
                                                          int64_t E_in, int64_t N,
                                                          float* __restrict__ deg,
                                                          float* __restrict__ dinv) {
  const int64_t t = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
  if (t >= N) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int kb = uniform(rowptr[t]), ke = uniform(rowptr[t + 1]);
  double acc = 0.0;
  for (int k = kb + lane; k < ke; k += kWave) acc += (double)edge_w(w, E_in, perm[k]);
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) {
    float d = (float)acc;
    if (deg) deg[t] = d;
    dinv[t] = d > 0.0f ? 1.0f / sqrtf(d) : 0.0f;
  }
}

// CSR order: one wavefront per aggregation work item (row or row chunk); each
// lane handles four positions per step with their loads issued together.
__global__ __launch_bounds__(kBlock) void weights_csr(const WorkItem* __restrict__ heavy,
                                                      int n_heavy,
                                                      const WorkItem* __restrict__ light,
                                                      int n_light, const int* __restrict__ col,
                                                      const int* __restrict__ perm,
                                                      const float* __restrict__ w, int64_t E_in,
                                                      const float* __restrict__ dinv,
                                                      float* __restrict__ out) {
  const int wid = uniform(blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave);
  if (wid >= n_heavy + n_light) return;
  const int lane = threadIdx.x & (kWave - 1);
  const WorkItem* it = wid < n_heavy ? heavy + wid : light + (wid - n_heavy);
  const int row = uniform(it->row), kb = uniform(it->kbeg), ke = uniform(it->kend);
  const float dt = dinv[row];
  for (int k0 = kb + lane; k0 < ke; k0 += 4 * kWave) {
    int c[4];
    float we[4], ds[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k = k0 + j * kWave < ke ? k0 + j * kWave : k0;
      c[j] = col[k];
      we[j] = w ? edge_w(w, E_in, perm[k]) : 1.0f;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) ds[j] = dinv[c[j]];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k = k0 + j * kWave;
      if (k < ke) {
        const float a = ds[j] * we[j];
        out[k] = a * dt;
      }
    }
  }
}

// COO order (input edges, then loops), optionally writing the edge list; four
// edges per thread, strided by the block size, loads issued together.
template <typename IdxT>
__global__ __launch_bounds__(kBlock) void weights_coo(const IdxT* __restrict__ src,
                                                      const IdxT* __restrict__ tgt, int64_t E_in,
                                                      int64_t E, int64_t N,
                                                      const float* __restrict__ w,
                                                      const float* __restrict__ dinv,
                                                      int32_t* __restrict__ out_ei,
                                                      float* __restrict__ out_w) {
  const int64_t base = (int64_t)blockIdx.x * (4 * kBlock) + threadIdx.x;
  int s[4], t[4];
  float we[4], ds[4], dt[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t e = base + j * kBlock;
    const int64_t ec = e < E_in ? e : (E_in > 0 ? E_in - 1 : 0);
    const int64_t sv = E_in > 0 ? (int64_t)__builtin_nontemporal_load(src + ec) : 0;
    const int64_t tv = E_in > 0 ? (int64_t)__builtin_nontemporal_load(tgt + ec) : 0;
    const bool in = e < E_in;
    // ids were validated when the graph was built; clamped here all the same
    s[j] = in ? ((sv < 0 || sv >= N) ? 0 : (int)sv) : (int)(e - E_in);
    t[j] = in ? ((tv < 0 || tv >= N) ? 0 : (int)tv) : (int)(e - E_in);
    we[j] = (w != nullptr && in) ? w[ec] : 1.0f;
  }
  if (out_w) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool ok = base + j * kBlock < E;
      ds[j] = ok ? dinv[s[j]] : 0.0f;
      dt[j] = ok ? dinv[t[j]] : 0.0f;
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t e = base + j * kBlock;
    if (e >= E) break;
    if (out_ei) {
      __builtin_nontemporal_store(s[j], out_ei + e);
      __builtin_nontemporal_store(t[j], out_ei + E + e);
    }
    if (out_w) {
      const float a = ds[j] * we[j];
      __builtin_nontemporal_store(a * dt[j], out_w + e);
    }
  }
}

}  // namespace

int launch_gcn_norm(const Graph& g, const void* edge_index, int index_type,
                    const float* edge_weight, int32_t* out_edge_index, float* out_w,
                    float* out_w_csr, float* out_deg, float* dinv, hipStream_t s) {
  if (g.N == 0) return TFG_OK;
  const unsigned nb_rows = (unsigned)((g.N + kBlock - 1) / kBlock);
  if (edge_weight == nullptr) {
    degree_unit<<<nb_rows, kBlock, 0, s>>>(g.rowptr, g.N, out_deg, dinv);
  } else {
    degree_weighted<<<(unsigned)((g.N + 3) / 4), kBlock, 0, s>>>(g.rowptr, g.perm, edge_weight,
                                                                 g.E_in, g.N, out_deg, dinv);
  }
  TFG_LAUNCHED("gcn degree");
  const int waves = g.n_heavy + g.n_light;
  if (out_w_csr && waves > 0) {
    weights_csr<<<(unsigned)((waves + 3) / 4), kBlock, 0, s>>>(
        g.heavy, g.n_heavy, g.light, g.n_light, g.col, g.perm, edge_weight, g.E_in, dinv,
        out_w_csr);
    TFG_LAUNCHED("gcn weights (CSR order)");
  }
  if ((out_w || out_edge_index) && g.E > 0) {
    const unsigned nb = (unsigned)((g.E + 4 * kBlock - 1) / (4 * kBlock));
    if (index_type == TFG_I64) {
      const int64_t* ei = static_cast<const int64_t*>(edge_index);
      weights_coo<int64_t><<<nb, kBlock, 0, s>>>(ei, ei + g.E_in, g.E_in, g.E, g.N, edge_weight,
                                                  dinv, out_edge_index, out_w);
    } else {
      const int32_t* ei = static_cast<const int32_t*>(edge_index);
      weights_coo<int32_t><<<nb, kBlock, 0, s>>>(ei, ei + g.E_in, g.E_in, g.E, g.N, edge_weight,
                                                  dinv, out_edge_index, out_w);
    }
    TFG_LAUNCHED("gcn weights (COO order)");
  }
  return TFG_OK;
}

}  // namespace tfg
