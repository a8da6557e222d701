// Gradients of the aggregation and of the segment softmax (gfx950, wave64).
//
// For out = aggregate(w, x) and an incoming gradient dy = dL/d out:
//   dx  (sum)  = the sum aggregation of dy over the transposed graph (rows are
//                sources, columns targets) with the same edge weights;
//   dx  (mean) = the same with w_e / deg(t_e) as weights;
//   dx  (max)  = the masked gather of spmm_rows: element c of dy[t] reaches
//                source s only through the edge that won the forward max;
//   dw[e, k]   = sum over the columns c of head k of g[t_e, c] x[s_e, c] with
//                g = dy, dy / deg(t) or the masked dy: one dot product per
//                edge (edge_grad_rows), walking the forward graph so that the
//                dy row of a target is loaded once.
// Segment softmax: ds = alpha * (dalpha - sum over the segment of alpha * dalpha)
// per head, the sum accumulated in double (softmax_grad_items; long rows in
// chunks whose sums are added in chunk order).
// Every result has one writer and a fixed summation order: no atomics.
#include <cstdlib>

#include "softmax_stats.h"
#include "spmm.h"

namespace tfg {

namespace rows {

void dispatch_masked(bool part_plan, bool heads, int vec, int slots, dim3 grid, hipStream_t s,
                     const RowArgs& a) {
  if (part_plan) {
    if (heads)
      dispatch_vec<false, true, true, true>(vec, slots, grid, s, a);
    else
      dispatch_vec<false, false, true, true>(vec, slots, grid, s, a);
  } else {
    if (heads)
      dispatch_vec<false, true, false, true>(vec, slots, grid, s, a);
    else
      dispatch_vec<false, false, false, true>(vec, slots, grid, s, a);
  }
}

}  // namespace rows

namespace {

using namespace rows;

enum { kGradSum = 0, kGradMean = 1, kGradMax = 2 };

// Sums each of the U values of a lane over the LPS lanes of its slot, U <= LPS
// (powers of two), with log2(LPS) xor exchanges in which the values are also
// transposed: at an exchange over offset o while c > 1 values remain, the
// lane with bit o set keeps the upper half of its values and sends the lower
// half (the partner the reverse), so c halves. After log2(U) such steps each
// lane holds one value, the sum for index sl / (LPS / U) over its group; the
// remaining exchanges are plain butterflies. log2(LPS) + U - 1 shuffles in
// all, against U * log2(LPS) for U separate trees.
template <int U, int LPS>
__device__ __forceinline__ float transpose_sum(float (&p)[U], int sl) {
  int cnt = U;
#pragma unroll
  for (int o = LPS / 2; o >= 1; o >>= 1) {
    if (cnt > 1) {
      const bool up = (sl & o) != 0;
      const int half = cnt / 2;
#pragma unroll
      for (int j = 0; j < U / 2; ++j) {
        if (j < half) {
          const float send = up ? p[j] : p[j + half];
          const float keep = up ? p[j + half] : p[j];
          p[j] = keep + __shfl_xor(send, o);
        }
      }
      cnt = half;
    } else {
      p[0] += __shfl_xor(p[0], o);
    }
  }
  return p[0];
}

// dw for the work items of the forward graph. Lanes are (edge slot, V
// columns); each lane keeps its V columns of g[t] in registers. With one head
// (WHOLE) the U partial dot products of a lane are summed over the slot with
// transpose_sum; with several heads they are summed over the G lanes of each
// head with a shift-down tree (the head's first lane holds the result).
template <int V, int SLOTS, int MODE, bool WHOLE>
__global__ __launch_bounds__(kItemBlock) void edge_grad_rows(
    const WorkItem* __restrict__ items, int n_items, const int* __restrict__ rowptr,
    const int* __restrict__ col, const int* __restrict__ perm, const float* __restrict__ x,
    int64_t ldx, const float* __restrict__ dy, const int* __restrict__ arg, int F, int H, int G,
    float* __restrict__ dw, int dw_by_perm, float scale) {
  constexpr int LPS = kWave / SLOTS;
  // 4 gathers in flight per slot with the transposing reduction keeps the
  // kernel within 64 VGPRs (8 waves per SIMD); 8 would need 79
  constexpr int UMAX = WHOLE ? 4 : 8;
  constexpr int U = SLOTS * UMAX <= kWave ? UMAX : kWave / SLOTS;
  const int wid = uniform(blockIdx.x * (kItemBlock / kWave) + threadIdx.x / kWave);
  if (wid >= n_items) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int slot = lane / LPS, sl = lane % LPS;
  const WorkItem* itp = items + wid;
  const int row = uniform(itp->row), kbeg = uniform(itp->kbeg), kend = uniform(itp->kend);
  if (kbeg >= kend) return;
  const int f = sl * V;
  const bool fok = f < F;
  const int r = sl % G, head = sl / G;
  const bool need_perm = MODE == kGradMax || dw_by_perm;

  float gy[V];
  int ga[V];
#pragma unroll
  for (int v = 0; v < V; ++v) {
    gy[v] = 0.0f;
    ga[v] = -1;
  }
  if (fok) {
    load_row<V>(dy + (int64_t)row * F + f, gy);
    if constexpr (MODE == kGradMean) {
      const float cnt = (float)(rowptr[row + 1] - rowptr[row]);
#pragma unroll
      for (int v = 0; v < V; ++v) gy[v] = gy[v] / cnt;
    }
    if constexpr (MODE == kGradMax) load_irow<V>(arg + (int64_t)row * F + f, ga);
  }

  for (int kb = kbeg; kb < kend; kb += kWave) {
    const int n = min(kWave, kend - kb);
    const bool lok = lane < n;
    const int cj = lok ? __builtin_nontemporal_load(col + kb + lane) : 0;
    const int pj = (lok && need_perm) ? __builtin_nontemporal_load(perm + kb + lane) : 0;
    for (int s0 = 0; s0 < n; s0 += SLOTS * U) {
      float p[U];
      int pe[U];
      bool ok[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int jb = s0 + u * SLOTS;
        ok[u] = jb + slot < n;
        const int c = bcast<SLOTS>(cj, jb, slot);
        pe[u] = need_perm ? bcast<SLOTS>(pj, jb, slot) : 0;
        float xv[V];
        if (ok[u] && fok) {
          load_row<V>(x + (int64_t)c * ldx + f, xv);
        } else {
#pragma unroll
          for (int v = 0; v < V; ++v) xv[v] = 0.0f;
        }
        float acc = 0.0f;
#pragma unroll
        for (int v = 0; v < V; ++v) {
          const float t = (MODE == kGradMax && ga[v] != pe[u]) ? 0.0f : gy[v];
          acc = __builtin_fmaf(t, xv[v], acc);
        }
        p[u] = acc;
      }
      if constexpr (WHOLE) {
        // lane sl ends with the dot product of edge slot u = sl / (LPS / U)
        constexpr int STRIDE = LPS / U;
        const int u = sl / STRIDE;
        const int j = s0 + u * SLOTS + slot;
        const int pu = need_perm ? __shfl(pj, j & (kWave - 1)) : 0;
        const float val = transpose_sum<U, LPS>(p, sl);
        if (sl % STRIDE == 0 && j < n) {
          const int64_t e = dw_by_perm ? pu : kb + j;
          dw[e] = val * scale;
        }
      } else {
        for (int off = 1; off < G; off <<= 1)
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const float o = __shfl_down(p[u], off);
            if (r + off < G) p[u] += o;
          }
        if (r == 0 && fok) {
#pragma unroll
          for (int u = 0; u < U; ++u)
            if (ok[u]) {
              const int64_t e = dw_by_perm ? pe[u] : kb + s0 + u * SLOTS + slot;
              dw[e * H + head] = p[u] * scale;
            }
        }
      }
    }
  }
}

// Fallback for shapes the lane mapping above does not cover (more than 64
// vector columns, or heads that are not a whole number of vectors): one
// thread per (graph position, head), columns in order.
template <int MODE>
__global__ __launch_bounds__(kBlock) void edge_grad_simple(
    const int* __restrict__ rowptr, int64_t N, int64_t E, const int* __restrict__ col,
    const int* __restrict__ perm, const float* __restrict__ x, int64_t ldx,
    const float* __restrict__ dy, const int* __restrict__ arg, int F, int H,
    float* __restrict__ dw, int dw_by_perm, float scale) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= E * H) return;
  const int64_t k = i / H;
  const int h = (int)(i - k * H);
  int64_t lo = 0, hi = N;  // the row t with rowptr[t] <= k < rowptr[t + 1]
  while (hi - lo > 1) {
    const int64_t mid = (lo + hi) >> 1;
    if (rowptr[mid] <= k) lo = mid; else hi = mid;
  }
  const int64_t t = lo, s = col[k], e = perm[k];
  const int D = F / H;
  const float cnt = (float)(rowptr[t + 1] - rowptr[t]);
  float acc = 0.0f;
  for (int c = h * D; c < (h + 1) * D; ++c) {
    float g = dy[t * F + c];
    if (MODE == kGradMean) g = g / cnt;
    if (MODE == kGradMax && arg[t * F + c] != (int)e) g = 0.0f;
    acc = __builtin_fmaf(g, x[s * ldx + c], acc);
  }
  dw[(dw_by_perm ? e : k) * H + h] = acc * scale;
}

// Weights of the transposed graph for the mean gradient, in its graph order:
// wt[k, h] = w[e, h] / deg(t_k) (w = 1 when NULL) with e = perm[k] for
// weights in edge order, e = k for weights already in the transposed order;
// t_k = col[k].
__global__ __launch_bounds__(kBlock) void mean_weights(const int* __restrict__ tcol,
                                                       const int* __restrict__ tperm, int64_t E,
                                                       int H, const int* __restrict__ rowptr,
                                                       const float* __restrict__ w, int by_perm,
                                                       float* __restrict__ wt) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= E * H) return;
  const int64_t k = i / H;
  const int h = (int)(i - k * H);
  const int t = tcol[k];
  const float cnt = (float)(rowptr[t + 1] - rowptr[t]);
  const float wv = w ? w[(by_perm ? (int64_t)tperm[k] : k) * H + h] : 1.0f;
  wt[i] = wv / cnt;
}

// Graph order -> caller's edge order: out[perm[k], h] = in[k, h].
__global__ __launch_bounds__(kBlock) void to_edge_order(const int* __restrict__ perm, int64_t E,
                                                        int H, const float* __restrict__ in,
                                                        float* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= E * H) return;
  const int64_t k = i / H;
  const int h = (int)(i - k * H);
  out[(int64_t)perm[k] * H + h] = in[i];
}

// The same scatter for one value per edge on large graphs, in two passes
// through buckets of 2^kPermBits consecutive destinations (a random 4-byte
// store moves a whole line; these passes move whole lines):
//   perm_count   per tile of kPermTile positions, the count of each bucket
//                (one column of a bucket-major table);
//   (exclusive scan of the table: every (bucket, tile) its place)
//   perm_bucket  each position's (destination mod 2^kPermBits, value) pair
//                to its bucket's place for this tile, slots taken with LDS
//                atomics (the order inside a bucket does not matter);
//   perm_place   one block per bucket: the pairs into LDS at their offsets,
//                then the bucket's 2^kPermBits destinations written in order.
// perm is a permutation, so every destination of a bucket is written once.
constexpr int kPermBits = 15;                         // destinations per bucket (128 KB of LDS)
constexpr int kPermThreads = 1024;
constexpr int kPermItems = 64;                        // positions per thread and tile
constexpr int kPermTile = kPermThreads * kPermItems;  // 65536
constexpr int kPermMaxBuckets = 8192;                 // LDS counters (32 KB)
constexpr int kPermXcds = 8;

// tiles in XCD-contiguous order (blocks are dispatched round-robin over the
// XCDs), so that the bucket runs of neighbouring tiles meet in one L2
__device__ __forceinline__ int perm_tile_of(int bid, int ntiles) {
  const int q = ntiles / kPermXcds, r = ntiles % kPermXcds;
  const int x = bid % kPermXcds, i = bid / kPermXcds;
  return x * q + min(x, r) + i;
}

__global__ __launch_bounds__(kPermThreads) void perm_count(const int* __restrict__ perm, int64_t E,
                                                       int nbuckets, int ntiles,
                                                       int* __restrict__ table) {
  __shared__ int cnt[kPermMaxBuckets];
  for (int b = threadIdx.x; b < nbuckets; b += kPermThreads) cnt[b] = 0;
  __syncthreads();
  const int tile = perm_tile_of((int)blockIdx.x, ntiles);
  const int64_t base = (int64_t)tile * kPermTile;
  const int n = (int)min<int64_t>(kPermTile, E - base);
  for (int i0 = 0; i0 < kPermItems; i0 += 16) {
    int d[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int p = (i0 + i) * kPermThreads + (int)threadIdx.x;
      d[i] = p < n ? __builtin_nontemporal_load(perm + base + p) : -1;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (d[i] >= 0) atomicAdd(&cnt[d[i] >> kPermBits], 1);
  }
  __syncthreads();
  for (int b = threadIdx.x; b < nbuckets; b += kPermThreads)
    table[(int64_t)b * ntiles + tile] = cnt[b];
}

__global__ __launch_bounds__(kPermThreads) void perm_bucket(const int* __restrict__ perm,
                                                        const float* __restrict__ in, int64_t E,
                                                        int nbuckets, int ntiles,
                                                        const int* __restrict__ table,
                                                        int2* __restrict__ pairs) {
  __shared__ int cur[kPermMaxBuckets];
  const int tile = perm_tile_of((int)blockIdx.x, ntiles);
  for (int b = threadIdx.x; b < nbuckets; b += kPermThreads)
    cur[b] = table[(int64_t)b * ntiles + tile];
  __syncthreads();
  const int64_t base = (int64_t)tile * kPermTile;
  const int n = (int)min<int64_t>(kPermTile, E - base);
  for (int i0 = 0; i0 < kPermItems; i0 += 16) {
    int d[16];
    float v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int p = (i0 + i) * kPermThreads + (int)threadIdx.x;
      d[i] = p < n ? __builtin_nontemporal_load(perm + base + p) : -1;
      v[i] = p < n ? __builtin_nontemporal_load(in + base + p) : 0.0f;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (d[i] >= 0) {
        const int slot = atomicAdd(&cur[d[i] >> kPermBits], 1);
        pairs[slot] = make_int2(d[i] & ((1 << kPermBits) - 1), __float_as_int(v[i]));
      }
  }
}

__global__ __launch_bounds__(kPermThreads) void perm_place(const int2* __restrict__ pairs,
                                                       const int* __restrict__ table, int ntiles,
                                                       int64_t E, int nbuckets,
                                                       float* __restrict__ out) {
  __shared__ float buf[1 << kPermBits];
  const int b = (int)blockIdx.x;
  const int64_t start = table[(int64_t)b * ntiles];
  const int64_t end = b + 1 < nbuckets ? table[(int64_t)(b + 1) * ntiles] : E;
  typedef int i2v __attribute__((ext_vector_type(2)));
  const i2v* pv = reinterpret_cast<const i2v*>(pairs);
  for (int64_t j0 = start; j0 < end; j0 += 8 * kPermThreads) {
    i2v pr[8];  // eight loads in flight per thread
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int64_t j = j0 + u * kPermThreads + threadIdx.x;
      pr[u] = j < end ? __builtin_nontemporal_load(pv + j) : i2v{-1, 0};
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (pr[u].x >= 0) buf[pr[u].x] = __int_as_float(pr[u].y);
  }
  __syncthreads();
  const int64_t o = (int64_t)b << kPermBits;
  const int n = (int)min<int64_t>(int64_t(1) << kPermBits, E - o);
  for (int j = threadIdx.x; j < n; j += kPermThreads) __builtin_nontemporal_store(buf[j], out + o + j);
}

// Caller's edge order -> graph order: out[k, h] = in[perm[k], h].
__global__ __launch_bounds__(kBlock) void to_graph_order(const int* __restrict__ perm, int64_t E,
                                                         int H, const float* __restrict__ in,
                                                         float* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= E * H) return;
  const int64_t k = i / H;
  const int h = (int)(i - k * H);
  out[i] = in[(int64_t)perm[k] * H + h];
}

// Softmax gradient ds = alpha * (dalpha - sum over the row of alpha *
// dalpha), per head, with the products summed in double (exact products of
// floats), in the layouts of the softmax: short rows one lane per (row,
// head), other light rows and chunks one wavefront each with their values in
// registers (NST slot steps, the next power of two of the item's), split rows
// of at most kGradSplitWaves chunks one block each with the chunk sums added
// in chunk order in LDS. Chunks of longer split rows store their sums
// (pdot), which softmax_grad_split adds in chunk order before writing.
constexpr int kGradCap = 8;          // slot steps held in registers
constexpr int kGradSplitWaves = 16;  // chunks per split row done by one block

__device__ __forceinline__ void grad_short_row(const WorkItem& it, const int* __restrict__ perm,
                                               const float* __restrict__ alpha,
                                               const float* __restrict__ da, int H, int hh,
                                               int HP, float* __restrict__ ds) {
  const int kb = it.kbeg, n = it.kend - it.kbeg;  // 0 <= n <= kShortRow
  int nw = 0;  // the wavefront's longest row
#pragma unroll
  for (int j = 1; j <= kShortRow; ++j) nw = __any(n >= j) ? j : nw;
  int e[kShortRow];
#pragma unroll
  for (int j = 0; j < kShortRow; ++j) e[j] = j < n ? edge_at(perm, kb + j) : 0;
  for (int h = hh; h < H; h += HP) {
    float a[kShortRow], g[kShortRow];
#pragma unroll
    for (int j = 0; j < kShortRow; ++j) {
      a[j] = j < n ? alpha[(int64_t)e[j] * H + h] : 0.0f;
      g[j] = j < n ? da[(int64_t)e[j] * H + h] : 0.0f;
    }
    double dot = 0.0;
#pragma unroll
    for (int j = 0; j < kShortRow; ++j)
      if (j < nw) dot += (double)a[j] * (double)g[j];
#pragma unroll
    for (int j = 0; j < kShortRow; ++j)
      if (j < n) ds[(int64_t)e[j] * H + h] = (float)((double)a[j] * ((double)g[j] - dot));
  }
}

// alpha and dalpha of head h for the registers' ids (0 where there is none)
template <int NST>
__device__ __forceinline__ void grad_load(const float* __restrict__ alpha,
                                          const float* __restrict__ da, int H, int h, bool act,
                                          const int (&e)[NST], float (&a)[NST],
                                          float (&g)[NST]) {
#pragma unroll
  for (int u = 0; u < NST; ++u) {
    const bool ok = act && e[u] >= 0;
    a[u] = ok ? alpha[(int64_t)e[u] * H + h] : 0.0f;
    g[u] = ok ? da[(int64_t)e[u] * H + h] : 0.0f;
  }
}

template <int NST>
__device__ __forceinline__ double grad_dot(const float (&a)[NST], const float (&g)[NST], int HP) {
  double dot = 0.0;
#pragma unroll
  for (int u = 0; u < NST; ++u) dot += (double)a[u] * (double)g[u];
  return slots_sum(dot, HP);
}

template <int NST>
__device__ __forceinline__ void grad_write(const float (&a)[NST], const float (&g)[NST],
                                           const int (&e)[NST], double dot, int H, int h,
                                           bool act, float* __restrict__ ds) {
#pragma unroll
  for (int u = 0; u < NST; ++u)
    if (act && e[u] >= 0) ds[(int64_t)e[u] * H + h] = (float)((double)a[u] * ((double)g[u] - dot));
}

// A whole item's sum over [kb, ke) for head h, loading the values (the items
// longer than kGradCap slot steps), and its ds from a second sweep.
__device__ __forceinline__ double grad_sweep_dot(const int* __restrict__ perm,
                                                 const float* __restrict__ alpha,
                                                 const float* __restrict__ da, int H, int h,
                                                 bool act, int kb, int ke, int slot, int SL,
                                                 int HP) {
  double dot = 0.0;
  for (int k = kb + slot; k < ke; k += SL)
    if (act) {
      const int64_t i = (int64_t)edge_at(perm, k) * H + h;
      dot += (double)alpha[i] * (double)da[i];
    }
  return slots_sum(dot, HP);
}

__device__ __forceinline__ void grad_sweep_write(const int* __restrict__ perm,
                                                 const float* __restrict__ alpha,
                                                 const float* __restrict__ da, int H, int h,
                                                 bool act, int kb, int ke, int slot, int SL,
                                                 double dot, float* __restrict__ ds) {
  for (int k = kb + slot; k < ke; k += SL)
    if (act) {
      const int64_t i = (int64_t)edge_at(perm, k) * H + h;
      ds[i] = (float)((double)alpha[i] * ((double)da[i] - dot));
    }
}

template <int NST>
__device__ __forceinline__ void grad_item_regs(const int* __restrict__ perm,
                                               const float* __restrict__ alpha,
                                               const float* __restrict__ da, int H, int HP,
                                               int kb, int ke, int slot, int hh, int pslot,
                                               float* __restrict__ ds,
                                               double* __restrict__ pdot) {
  const int SL = kWave / HP;
  int e[NST];
  load_ids<NST>(perm, kb, ke, slot, SL, e);
  for (int hb = 0; hb < H; hb += HP) {
    const int h = hb + hh;
    const bool act = h < H;
    float a[NST], g[NST];
    grad_load<NST>(alpha, da, H, h, act, e, a, g);
    const double dot = grad_dot<NST>(a, g, HP);
    if (pslot >= 0) {
      if (slot == 0 && act) pdot[(int64_t)pslot * H + h] = dot;
      continue;
    }
    grad_write<NST>(a, g, e, dot, H, h, act, ds);
  }
}

// Wavefronts [0, short_waves) take 64 / HP short rows each; the next n_long
// one light row of more than kShortRow edges each; the rest one chunk of a
// split row of more than kGradSplitWaves chunks (the others are left to
// softmax_grad_split).
__global__ __launch_bounds__(kItemBlock) void softmax_grad_items(
    const WorkItem* __restrict__ short_rows, int n_short, int short_waves,
    const WorkItem* __restrict__ long_rows, int n_long, const WorkItem* __restrict__ heavy,
    int n_heavy, const int* __restrict__ rowptr, int chunk, const int* __restrict__ perm,
    const float* __restrict__ alpha, const float* __restrict__ da, int H, int HP,
    float* __restrict__ ds, double* __restrict__ pdot) {
  const int lane = threadIdx.x & (kWave - 1);
  int wid = uniform(blockIdx.x * (kItemBlock / kWave) + threadIdx.x / kWave);
  if (wid < short_waves) {
    const int i = wid * (kWave / HP) + lane / HP;
    if (i < n_short) grad_short_row(short_rows[i], perm, alpha, da, H, lane % HP, HP, ds);
    return;
  }
  wid -= short_waves;
  if (wid >= n_long + n_heavy) return;
  const int SL = kWave / HP;
  const int slot = lane / HP, hh = lane % HP;
  int kb, ke, pslot = -1;
  if (wid < n_long) {
    kb = uniform(long_rows[wid].kbeg);
    ke = uniform(long_rows[wid].kend);
  } else {
    const WorkItem* it = heavy + (wid - n_long);
    const int row = uniform(it->row);
    const int deg = uniform(rowptr[row + 1]) - uniform(rowptr[row]);
    if ((deg + chunk - 1) / chunk <= kGradSplitWaves) return;
    kb = uniform(it->kbeg);
    ke = uniform(it->kend);
    pslot = uniform(it->slot);
  }
  const int nst = (ke - kb + SL - 1) / SL;
  if (nst <= 1) {
    grad_item_regs<1>(perm, alpha, da, H, HP, kb, ke, slot, hh, pslot, ds, pdot);
  } else if (nst <= 2) {
    grad_item_regs<2>(perm, alpha, da, H, HP, kb, ke, slot, hh, pslot, ds, pdot);
  } else if (nst <= 4) {
    grad_item_regs<4>(perm, alpha, da, H, HP, kb, ke, slot, hh, pslot, ds, pdot);
  } else if (nst <= kGradCap) {
    grad_item_regs<kGradCap>(perm, alpha, da, H, HP, kb, ke, slot, hh, pslot, ds, pdot);
  } else {
    for (int hb = 0; hb < H; hb += HP) {
      const int h = hb + hh;
      const bool act = h < H;
      const double dot = grad_sweep_dot(perm, alpha, da, H, h, act, kb, ke, slot, SL, HP);
      if (pslot >= 0) {
        if (slot == 0 && act) pdot[(int64_t)pslot * H + h] = dot;
        continue;
      }
      grad_sweep_write(perm, alpha, da, H, h, act, kb, ke, slot, SL, dot, ds);
    }
  }
}

// Chunk w of a split row of at most kGradSplitWaves chunks (NST = 0: the
// values are loaded again to write); every wavefront runs the same head
// passes and barriers, with or without a chunk.
template <int NST>
__device__ __forceinline__ void grad_split_chunk(const int* __restrict__ perm,
                                                 const float* __restrict__ alpha,
                                                 const float* __restrict__ da, int H, int HP,
                                                 int kb, int ke, int nch, int w, int lane,
                                                 double (&lsum)[kGradSplitWaves][kWave],
                                                 float* __restrict__ ds) {
  const int SL = kWave / HP;
  const int slot = lane / HP, hh = lane % HP;
  const bool has = kb < ke;
  constexpr int R = NST > 0 ? NST : 1;
  int e[R];
  if constexpr (NST > 0) load_ids<NST>(perm, kb, ke, slot, SL, e);
  for (int hb = 0; hb < H; hb += HP) {
    const int h = hb + hh;
    const bool act = h < H;
    float a[R], g[R];
    double dot = 0.0;
    if (has) {
      if constexpr (NST > 0) {
        grad_load<NST>(alpha, da, H, h, act, e, a, g);
        dot = grad_dot<NST>(a, g, HP);
      } else {
        dot = grad_sweep_dot(perm, alpha, da, H, h, act, kb, ke, slot, SL, HP);
      }
    }
    lsum[w][lane] = dot;
    __syncthreads();
    double tot = 0.0;
    for (int c = 0; c < nch; ++c) tot += lsum[c][lane];
    __syncthreads();  // the sums are read before the next head pass writes
    if (!has) continue;
    if constexpr (NST > 0)
      grad_write<NST>(a, g, e, tot, H, h, act, ds);
    else
      grad_sweep_write(perm, alpha, da, H, h, act, kb, ke, slot, SL, tot, ds);
  }
}

// One block per split row (kGradSplitWaves wavefronts): grad_split_chunk for
// a row of at most kGradSplitWaves chunks; for a longer one the chunk sums
// from softmax_grad_items, added in chunk order, and wavefront w writes
// chunks w, w + kGradSplitWaves, ...
__global__ __launch_bounds__(kGradSplitWaves * kWave) void softmax_grad_split(
    const SplitRow* __restrict__ split, const int* __restrict__ rowptr, int chunk,
    const int* __restrict__ perm, const float* __restrict__ alpha, const float* __restrict__ da,
    int H, int HP, const double* __restrict__ pdot, float* __restrict__ ds) {
  __shared__ double lsum[kGradSplitWaves][kWave];
  const SplitRow* sr = split + blockIdx.x;
  const int row = uniform(sr->row), nch = uniform(sr->nchunks), s0 = uniform(sr->slot0);
  const int rb = uniform(rowptr[row]), re = uniform(rowptr[row + 1]);
  const int w = uniform((int)threadIdx.x / kWave);
  const int lane = threadIdx.x & (kWave - 1);
  const int SL = kWave / HP;
  if (nch <= kGradSplitWaves) {
    const int kb = rb + w * chunk, ke = min(re, kb + chunk);  // kb >= ke: no chunk
    const int cst = (chunk + SL - 1) / SL;  // slot steps of a whole chunk
    if (cst <= 2)
      grad_split_chunk<2>(perm, alpha, da, H, HP, kb, ke, nch, w, lane, lsum, ds);
    else if (cst <= 4)
      grad_split_chunk<4>(perm, alpha, da, H, HP, kb, ke, nch, w, lane, lsum, ds);
    else if (cst <= kGradCap)
      grad_split_chunk<kGradCap>(perm, alpha, da, H, HP, kb, ke, nch, w, lane, lsum, ds);
    else if (cst <= 2 * kGradCap)
      grad_split_chunk<2 * kGradCap>(perm, alpha, da, H, HP, kb, ke, nch, w, lane, lsum, ds);
    else
      grad_split_chunk<0>(perm, alpha, da, H, HP, kb, ke, nch, w, lane, lsum, ds);
    return;
  }
  const int slot = lane / HP, hh = lane % HP;
  for (int hb = 0; hb < H; hb += HP) {
    const int h = hb + hh;
    const bool act = h < H;
    double dot = 0.0;
    if (act)
      for (int c = 0; c < nch; ++c) dot += pdot[(int64_t)(s0 + c) * H + h];
    for (int c = w; c < nch; c += kGradSplitWaves) {
      const int kb = rb + c * chunk, ke = min(re, kb + chunk);
      grad_sweep_write(perm, alpha, da, H, h, act, kb, ke, slot, SL, dot, ds);
    }
  }
}

template <int V, int MODE, bool WHOLE>
void launch_edge_grad_slots(int slots, dim3 grid, hipStream_t s, const WorkItem* items,
                            int n_items, const Graph& g, const float* x, int64_t ldx,
                            const float* dy, const int* arg, int F, int H, int G, float* dw,
                            int by_perm, float scale) {
#define TFG_EG(SL)                                                                      \
  edge_grad_rows<V, SL, MODE, WHOLE><<<grid, kItemBlock, 0, s>>>(                       \
      items, n_items, g.rowptr, g.col, g.perm, x, ldx, dy, arg, F, H, G, dw, by_perm, scale)
  switch (slots) {
    case 1: TFG_EG(1); break;
    case 2: TFG_EG(2); break;
    case 4: TFG_EG(4); break;
    case 8: TFG_EG(8); break;
    default: TFG_EG(16); break;
  }
#undef TFG_EG
}

template <int MODE>
int launch_edge_grad(const Graph& g, const float* x, int64_t ldx, const float* dy,
                     const int* arg, int64_t F, int H, float* dw, int by_perm, hipStream_t s,
                     float scale = 1.0f) {
  const int D = (int)(F / H);
  auto fits = [&](int v) {
    return D % v == 0 && ldx % v == 0 && reinterpret_cast<uintptr_t>(x) % (4 * v) == 0 &&
           reinterpret_cast<uintptr_t>(dy) % (4 * v) == 0 &&
           (arg == nullptr || reinterpret_cast<uintptr_t>(arg) % (4 * v) == 0);
  };
  const int vec = fits(4) ? 4 : fits(2) ? 2 : 1;
  if (F / vec > kWave) {
    const int64_t n = g.E * H;
    edge_grad_simple<MODE><<<(unsigned)((n + kBlock - 1) / kBlock), kBlock, 0, s>>>(
        g.rowptr, g.N, g.E, g.col, g.perm, x, ldx, dy, arg, (int)F, H, dw, by_perm, scale);
    TFG_LAUNCHED("edge_grad_simple");
    return TFG_OK;
  }
  int p2 = 1;
  while (p2 < F / vec) p2 <<= 1;
  const int slots = std::min(kWave / p2, 16);
  // every edge belongs to exactly one work item of either plan (the row plan
  // keeps its long-row chunks and its whole rows in two lists)
  auto run = [&](const WorkItem* it, int n) {
    if (n <= 0) return;
    dim3 grid((unsigned)((n + kItemBlock / kWave - 1) / (kItemBlock / kWave)));
    const int G = D / vec;
    if (H == 1) {
      if (vec == 4)
        launch_edge_grad_slots<4, MODE, true>(slots, grid, s, it, n, g, x, ldx, dy, arg, (int)F,
                                              H, G, dw, by_perm, scale);
      else if (vec == 2)
        launch_edge_grad_slots<2, MODE, true>(slots, grid, s, it, n, g, x, ldx, dy, arg, (int)F,
                                              H, G, dw, by_perm, scale);
      else
        launch_edge_grad_slots<1, MODE, true>(slots, grid, s, it, n, g, x, ldx, dy, arg, (int)F,
                                              H, G, dw, by_perm, scale);
    } else {
      if (vec == 4)
        launch_edge_grad_slots<4, MODE, false>(slots, grid, s, it, n, g, x, ldx, dy, arg, (int)F,
                                               H, G, dw, by_perm, scale);
      else if (vec == 2)
        launch_edge_grad_slots<2, MODE, false>(slots, grid, s, it, n, g, x, ldx, dy, arg, (int)F,
                                               H, G, dw, by_perm, scale);
      else
        launch_edge_grad_slots<1, MODE, false>(slots, grid, s, it, n, g, x, ldx, dy, arg, (int)F,
                                               H, G, dw, by_perm, scale);
    }
  };
  if (use_part_plan(g, F)) {
    run(g.pexec, g.n_pexec);
  } else {
    run(g.heavy, g.n_heavy);
    run(g.light, g.n_light);
  }
  TFG_LAUNCHED("edge_grad_rows");
  return TFG_OK;
}

}  // namespace

// Bytes of the bucketed scatter's scratch (pairs, bucket table, scan sums);
// 0 where the plain scatter runs (several values per edge, small or very
// large graphs).
size_t perm_scatter_ws_bytes(int64_t E, int H) {
  if (H != 1 || E < (int64_t(1) << 20)) return 0;
  if (const char* v = std::getenv("TFG_PERM_BUCKETS"))  // "0": the plain scatter
    if (v[0] == '0') return 0;
  const int64_t nbuckets = (E + (int64_t(1) << kPermBits) - 1) >> kPermBits;
  if (nbuckets > kPermMaxBuckets) return 0;
  const int64_t ntiles = (E + kPermTile - 1) / kPermTile;
  const int64_t entries = nbuckets * ntiles;
  return align_up(sizeof(int2) * (size_t)E, 256) + align_up(sizeof(int) * (size_t)entries, 256) +
         align_up(sizeof(int) * (size_t)exclusive_scan_sums(entries), 256);
}

// out[perm[k], h] = in[k, h]; bucketed when ws holds perm_scatter_ws_bytes.
int launch_perm_scatter(const int* perm, int64_t E, int H, const float* in, float* out, void* ws,
                        size_t ws_bytes, hipStream_t s) {
  const int64_t n = E * H;
  if (n == 0) return TFG_OK;
  const size_t need = perm_scatter_ws_bytes(E, H);
  if (need == 0 || ws == nullptr || ws_bytes < need) {
    to_edge_order<<<(unsigned)((n + kBlock - 1) / kBlock), kBlock, 0, s>>>(perm, E, H, in, out);
    TFG_LAUNCHED("to_edge_order");
    return TFG_OK;
  }
  const int nbuckets = (int)((E + (int64_t(1) << kPermBits) - 1) >> kPermBits);
  const int ntiles = (int)((E + kPermTile - 1) / kPermTile);
  const int64_t entries = (int64_t)nbuckets * ntiles;
  char* c = static_cast<char*>(ws);
  int2* pairs = reinterpret_cast<int2*>(c);
  c += align_up(sizeof(int2) * (size_t)E, 256);
  int* table = reinterpret_cast<int*>(c);
  c += align_up(sizeof(int) * (size_t)entries, 256);
  int* sums = reinterpret_cast<int*>(c);
  perm_count<<<ntiles, kPermThreads, 0, s>>>(perm, E, nbuckets, ntiles, table);
  TFG_LAUNCHED("perm_count");
  if (int rc = exclusive_scan(table, table, entries, sums, s)) return rc;
  perm_bucket<<<ntiles, kPermThreads, 0, s>>>(perm, in, E, nbuckets, ntiles, table, pairs);
  TFG_LAUNCHED("perm_bucket");
  perm_place<<<nbuckets, kPermThreads, 0, s>>>(pairs, table, ntiles, E, nbuckets, out);
  TFG_LAUNCHED("perm_place");
  return TFG_OK;
}


int launch_edge_dot(const Graph& g, const float* q, const float* key, int64_t ldk, int64_t F,
                    int H, float scale, float* out, int by_perm, hipStream_t s) {
  if (g.E == 0 || F == 0) return TFG_OK;
  return launch_edge_grad<kGradSum>(g, key, ldk, q, nullptr, F, H, out, by_perm, s, scale);
}

// Graph -> graph goes through edge order in the first E * H floats of ws;
// the scatter's scratch follows.
size_t edge_reorder_ws_bytes(int64_t E, int H, bool from, bool to) {
  const size_t tmp = (from && to) ? align_up(sizeof(float) * (size_t)std::max<int64_t>(E * H, 1), 256) : 0;
  return tmp + (from ? perm_scatter_ws_bytes(E, H) : 0);
}

int launch_edge_reorder(const int* perm_from, const int* perm_to, int64_t E, int H,
                        const float* in, float* out, void* ws, size_t ws_bytes, hipStream_t s) {
  const int64_t n = E * H;
  if (n == 0) return TFG_OK;
  const unsigned nb = (unsigned)((n + kBlock - 1) / kBlock);
  if (perm_from != nullptr && perm_to != nullptr) {
    const size_t tb = align_up(sizeof(float) * (size_t)n, 256);
    float* tmp = static_cast<float*>(ws);
    const int rc = launch_perm_scatter(perm_from, E, H, in, tmp, static_cast<char*>(ws) + tb,
                                       ws_bytes > tb ? ws_bytes - tb : 0, s);
    if (rc) return rc;
    to_graph_order<<<nb, kBlock, 0, s>>>(perm_to, E, H, tmp, out);
  } else if (perm_from != nullptr) {
    return launch_perm_scatter(perm_from, E, H, in, out, ws, ws_bytes, s);
  } else {
    to_graph_order<<<nb, kBlock, 0, s>>>(perm_to, E, H, in, out);
  }
  TFG_LAUNCHED("edge reorder");
  return TFG_OK;
}

size_t aggregate_backward_ws_bytes(const Graph& g, const Graph* gt, int64_t F, int64_t H,
                                   int reduce, int w_order, bool has_w) {
  size_t b = 256;
  if (gt == nullptr) return b;
  const int64_t parts = use_part_plan(*gt, F) ? gt->n_pexec : gt->n_heavy;
  b += aggregate_partial_bytes(parts, F, TFG_SUM);
  const size_t ew = align_up(sizeof(float) * (size_t)std::max<int64_t>(g.E * H, 1), 256);
  // weights moved to edge order (and the bucketed scatter's scratch)
  if (has_w && w_order == TFG_CSR) b += ew + perm_scatter_ws_bytes(g.E, (int)H);
  if (reduce == TFG_MEAN) b += ew;           // weights / degree in transposed order
  return b;
}

int launch_aggregate_backward(const Graph& g, const Graph* gt, const float* w, int H, int w_order,
                              const float* x, int64_t ldx, const float* dy, int64_t F,
                              int reduce, const int32_t* argmax, float* dx, float* dw,
                              int dw_order, void* ws, hipStream_t s) {
  const int64_t EH = g.E * H;
  const unsigned eb = (unsigned)((EH + kBlock - 1) / kBlock);
  char* base = static_cast<char*>(ws);
  size_t off = 256;
  if (dx != nullptr && gt != nullptr) {
    const int64_t parts = use_part_plan(*gt, F) ? gt->n_pexec : gt->n_heavy;
    void* part = base + off;
    off += aggregate_partial_bytes(parts, F, TFG_SUM);
    const size_t ew = align_up(sizeof(float) * (size_t)std::max<int64_t>(EH, 1), 256);
    // weights for the gather over gt: in edge order (read through gt's perm)
    // or already in gt's order (read in sequence)
    const float* wg = w;
    int wg_order = w_order == TFG_CSR_T ? TFG_CSR : TFG_COO;
    if (w != nullptr && w_order == TFG_CSR && EH > 0) {
      float* t = reinterpret_cast<float*>(base + off);
      off += ew;
      const size_t sb = perm_scatter_ws_bytes(g.E, H);
      const int rc = launch_perm_scatter(g.perm, g.E, H, w, t, sb ? base + off : nullptr, sb, s);
      if (rc) return rc;
      off += sb;
      wg = t;
    }
    if (gt->N > 0 && F > 0) {
      int rc;
      if (reduce == TFG_MEAN) {
        float* wt = reinterpret_cast<float*>(base + off);
        off += ew;
        if (EH > 0) {
          mean_weights<<<eb, kBlock, 0, s>>>(gt->col, gt->perm, g.E, H, g.rowptr, wg,
                                             wg_order == TFG_COO ? 1 : 0, wt);
          TFG_LAUNCHED("mean_weights");
        }
        rc = launch_aggregate(*gt, wt, H, TFG_CSR, dy, F, F, TFG_SUM, dx, nullptr, part, s);
      } else {
        rc = launch_aggregate(*gt, wg, wg ? H : 1, wg_order, dy, F, F, TFG_SUM, dx, nullptr, part,
                              s, 1.0f, 0.0f, nullptr, 0, reduce == TFG_MAX ? argmax : nullptr);
      }
      if (rc) return rc;
    }
  }
  if (dw != nullptr && EH > 0 && F > 0) {
    const int by_perm = dw_order == TFG_COO ? 1 : 0;
    int rc;
    if (reduce == TFG_MEAN)
      rc = launch_edge_grad<kGradMean>(g, x, ldx, dy, nullptr, F, H, dw, by_perm, s);
    else if (reduce == TFG_MAX)
      rc = launch_edge_grad<kGradMax>(g, x, ldx, dy, argmax, F, H, dw, by_perm, s);
    else
      rc = launch_edge_grad<kGradSum>(g, x, ldx, dy, nullptr, F, H, dw, by_perm, s);
    if (rc) return rc;
  }
  return TFG_OK;
}

int launch_segment_softmax_backward(const Graph& g, const float* alpha, const float* dalpha,
                                    int H, float* ds, void* ws, hipStream_t s, bool graph_order) {
  if (g.N == 0 || g.E == 0 || H == 0) return TFG_OK;
  const int* perm = graph_order ? nullptr : g.perm;  // alpha, dalpha, ds in the graph order
  int hp = 1;
  while (hp * 2 <= std::min(H, kWave)) hp *= 2;
  // the double part of the per-chunk statistics (row_stats_bytes layout)
  double* pdot = reinterpret_cast<double*>(
      static_cast<char*>(ws) +
      align_up(sizeof(float) * (size_t)std::max<int64_t>((int64_t)g.n_heavy * H, 1), 256));
  const int64_t short_waves = (g.n_short + kWave / hp - 1) / (kWave / hp);
  const int64_t waves = short_waves + g.n_long + g.n_heavy;
  if (waves > INT32_MAX) return fail(TFG_ERR_TOO_LARGE, "softmax gradient: too many work items");
  if (waves > 0) {
    softmax_grad_items<<<(unsigned)((waves + (kItemBlock / kWave) - 1) / (kItemBlock / kWave)), kItemBlock, 0, s>>>(
        g.short_rows, g.n_short, (int)short_waves, g.long_rows, g.n_long, g.heavy, g.n_heavy,
        g.rowptr, g.chunk, perm, alpha, dalpha, H, hp, ds, pdot);
    TFG_LAUNCHED("softmax_grad_items");
  }
  if (g.n_split > 0) {
    softmax_grad_split<<<(unsigned)g.n_split, kGradSplitWaves * kWave, 0, s>>>(
        g.split, g.rowptr, g.chunk, perm, alpha, dalpha, H, hp, pdot, ds);
    TFG_LAUNCHED("softmax_grad_split");
  }
  return TFG_OK;
}

}  // namespace tfg
