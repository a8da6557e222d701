// Graph pooling over a sorted node -> graph index (gfx950): segment bounds
// from the sorted index (with range and order checks), then one wavefront per
// graph reducing its contiguous node rows (sum / mean / max + argmax); and its
// gradient, one thread per node and column vector.
#include "wave.h"

namespace tfg {
namespace {

typedef float f2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));

__global__ void zero_ints(int* __restrict__ p, int64_t n) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

__device__ __forceinline__ int64_t clamp_gid(int64_t g, int64_t G) {
  return g < -1 ? -1 : (g > G - 1 ? G - 1 : g);
}

// goff[g] = first node of graph g, goff[G] = Nb. Node n writes the starts of
// the graphs (gi[n-1], gi[n]]; the thread n = Nb writes the empty tail graphs.
// With valid sorted input every entry is written exactly once. Otherwise the
// error flag is set, and every entry is still written (so goff needs no
// clearing first) with a value in [0, Nb]: the clamped ids run from -1 (before
// node 0) to G (after node Nb - 1), so each g in [0, G] lies in (prev, cur] for
// the first n whose cur reaches g.
template <typename IdxT>
__global__ __launch_bounds__(kBlock) void segment_bounds(const IdxT* __restrict__ gi, int64_t Nb,
                                                         int64_t G, int* __restrict__ goff,
                                                         int* __restrict__ err) {
  int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n > Nb) return;
  int64_t prev = n > 0 ? (int64_t)gi[n - 1] : -1;
  int64_t cur;
  if (n < Nb) {
    cur = (int64_t)gi[n];
    int bad = 0;
    if (cur < 0 || cur >= G) bad |= kErrIndex;
    if (n > 0 && cur < prev) bad |= kErrUnsorted;
    if (bad) atomicOr(err, bad);
  } else {
    cur = G;  // the tail: graphs after the last node's graph start at Nb
  }
  int64_t a = clamp_gid(prev, G), b = n < Nb ? clamp_gid(cur, G) : G;
  for (int64_t g = a + 1; g <= b; ++g) goff[g] = (int)n;
}

template <int V>
__device__ __forceinline__ void load_row(const float* __restrict__ p, float (&v)[V]) {
  if constexpr (V == 4) {
    f4 t = *reinterpret_cast<const f4*>(p);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else if constexpr (V == 2) {
    f2 t = *reinterpret_cast<const f2*>(p);
    v[0] = t.x; v[1] = t.y;
  } else {
    v[0] = *p;
  }
}

__device__ __forceinline__ void max_combine(float& v, int& a, float vb, int ab) {
  bool take = ab >= 0 && (a < 0 || vb > v || (vb == v && ab < a));
  v = take ? vb : v;
  a = take ? ab : a;
}

// One wavefront per graph; SLOTS node slots of 64/SLOTS lanes, U nodes in
// flight per slot, pairwise combination (as in the aggregation kernel).
template <int V, int SLOTS, bool MAX>
__global__ __launch_bounds__(kItemBlock) void pool_rows(const float* __restrict__ x, int64_t ldx,
                                                    int F, const int* __restrict__ goff, int64_t G,
                                                    int64_t Nb, int mean, float* __restrict__ out,
                                                    int* __restrict__ argout) {
  constexpr int LPS = kWave / SLOTS;
  constexpr int FC = LPS * V;
  constexpr int U = SLOTS * 8 <= kWave ? 8 : kWave / SLOTS;
  const int64_t g = (int64_t)blockIdx.x * (kItemBlock / kWave) + threadIdx.x / kWave;
  if (g >= G) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int slot = lane / LPS, sl = lane % LPS;
  int b = uniform(goff[g]), e = uniform(goff[g + 1]);
  b = b < 0 ? 0 : (b > Nb ? (int)Nb : b);
  e = e < b ? b : (e > Nb ? (int)Nb : e);
  for (int f0 = 0; f0 < F; f0 += FC) {
    const int f = f0 + sl * V;
    const bool fok = f < F;
    float acc[U][V];
    int arg[U][V];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int v = 0; v < V; ++v) {
        acc[u][v] = 0.0f;
        arg[u][v] = -1;
      }
    for (int n0 = b; n0 < e; n0 += SLOTS * U) {
      float xv[U][V];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int n = n0 + u * SLOTS + slot;
        if (n < e && fok) {
          load_row<V>(x + (int64_t)n * ldx + f, xv[u]);
        } else {
#pragma unroll
          for (int v = 0; v < V; ++v) xv[u][v] = 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int n = n0 + u * SLOTS + slot;
        if (n < e) {
#pragma unroll
          for (int v = 0; v < V; ++v) {
            if constexpr (MAX) {
              if (arg[u][v] < 0 || xv[u][v] > acc[u][v]) {
                acc[u][v] = xv[u][v];
                arg[u][v] = n;
              }
            } else {
              acc[u][v] += xv[u][v];
            }
          }
        }
      }
    }
#pragma unroll
    for (int step = 1; step < U; step <<= 1)
#pragma unroll
      for (int u = 0; u + step < U; u += 2 * step)
#pragma unroll
        for (int v = 0; v < V; ++v) {
          if constexpr (MAX)
            max_combine(acc[u][v], arg[u][v], acc[u + step][v], arg[u + step][v]);
          else
            acc[u][v] += acc[u + step][v];
        }
#pragma unroll
    for (int off = LPS; off < kWave; off <<= 1)
#pragma unroll
      for (int v = 0; v < V; ++v) {
        const float ov = __shfl_xor(acc[0][v], off);
        if constexpr (MAX) {
          const int oa = __shfl_xor(arg[0][v], off);
          max_combine(acc[0][v], arg[0][v], ov, oa);
        } else {
          acc[0][v] += ov;
        }
      }
    if (slot == 0 && fok) {
#pragma unroll
      for (int v = 0; v < V; ++v) {
        float r = acc[0][v];
        if (!MAX && mean && e > b) r = r / (float)(e - b);
        if (MAX && arg[0][v] < 0) r = 0.0f;
        out[g * F + f + v] = r;
        if (MAX && argout != nullptr) argout[g * F + f + v] = arg[0][v];
      }
    }
  }
}

template <int V, bool MAX>
void launch_pool_slots(int slots, dim3 grid, hipStream_t s, const float* x, int64_t ldx, int F,
                       const int* goff, int64_t G, int64_t Nb, int mean, float* out, int* argout) {
  switch (slots) {
    case 1: pool_rows<V, 1, MAX><<<grid, kItemBlock, 0, s>>>(x, ldx, F, goff, G, Nb, mean, out, argout); break;
    case 2: pool_rows<V, 2, MAX><<<grid, kItemBlock, 0, s>>>(x, ldx, F, goff, G, Nb, mean, out, argout); break;
    case 4: pool_rows<V, 4, MAX><<<grid, kItemBlock, 0, s>>>(x, ldx, F, goff, G, Nb, mean, out, argout); break;
    case 8: pool_rows<V, 8, MAX><<<grid, kItemBlock, 0, s>>>(x, ldx, F, goff, G, Nb, mean, out, argout); break;
    default: pool_rows<V, 16, MAX><<<grid, kItemBlock, 0, s>>>(x, ldx, F, goff, G, Nb, mean, out, argout); break;
  }
}

template <bool MAX>
void launch_pool_vec(int vec, int slots, dim3 grid, hipStream_t s, const float* x, int64_t ldx,
                     int F, const int* goff, int64_t G, int64_t Nb, int mean, float* out,
                     int* argout) {
  if (vec == 4)
    launch_pool_slots<4, MAX>(slots, grid, s, x, ldx, F, goff, G, Nb, mean, out, argout);
  else if (vec == 2)
    launch_pool_slots<2, MAX>(slots, grid, s, x, ldx, F, goff, G, Nb, mean, out, argout);
  else
    launch_pool_slots<1, MAX>(slots, grid, s, x, ldx, F, goff, G, Nb, mean, out, argout);
}

}  // namespace

namespace {

// Gradient of the pooling: one thread per (node, V columns) writes
// dx[n, c] = dy[g, c] (sum), dy[g, c] / count(g) (mean), or dy[g, c] where
// node n won the forward max of (g, c), else 0. g = the clamped graph id; the
// counts come from the segment bounds.
template <typename IdxT, int V>
__global__ __launch_bounds__(kBlock) void pool_grad(const float* __restrict__ dy, int64_t G,
                                                    int F, const IdxT* __restrict__ gi,
                                                    int64_t Nb, const int* __restrict__ goff,
                                                    int reduce, const int* __restrict__ arg,
                                                    float* __restrict__ dx, int64_t ldx) {
  const int cols = F / V;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= Nb * cols) return;
  const int64_t n = i / cols;
  const int f = (int)(i - n * cols) * V;
  const int64_t g = clamp_gid((int64_t)gi[n], G);
  float v[V];
  if (g < 0) {
#pragma unroll
    for (int j = 0; j < V; ++j) v[j] = 0.0f;
  } else {
    load_row<V>(dy + g * F + f, v);
    if (reduce == TFG_MEAN) {
      const float cnt = (float)(goff[g + 1] - goff[g]);
#pragma unroll
      for (int j = 0; j < V; ++j) v[j] = cnt > 0.0f ? v[j] / cnt : 0.0f;
    } else if (reduce == TFG_MAX) {
#pragma unroll
      for (int j = 0; j < V; ++j) v[j] = arg[g * F + f + j] == (int)n ? v[j] : 0.0f;
    }
  }
#pragma unroll
  for (int j = 0; j < V; ++j) dx[n * ldx + f + j] = v[j];
}

template <typename IdxT>
void launch_pool_grad(int vec, const float* dy, int64_t G, int F, const void* gi, int64_t Nb,
                      const int* goff, int reduce, const int* arg, float* dx, int64_t ldx,
                      hipStream_t s) {
  const int64_t n = Nb * (F / vec);
  const unsigned nb = (unsigned)((n + kBlock - 1) / kBlock);
  const IdxT* g = static_cast<const IdxT*>(gi);
  if (vec == 4)
    pool_grad<IdxT, 4><<<nb, kBlock, 0, s>>>(dy, G, F, g, Nb, goff, reduce, arg, dx, ldx);
  else if (vec == 2)
    pool_grad<IdxT, 2><<<nb, kBlock, 0, s>>>(dy, G, F, g, Nb, goff, reduce, arg, dx, ldx);
  else
    pool_grad<IdxT, 1><<<nb, kBlock, 0, s>>>(dy, G, F, g, Nb, goff, reduce, arg, dx, ldx);
}

}  // namespace

int launch_segment_pool_backward(const float* dy, int64_t G, int64_t F, const void* graph_index,
                                 int index_type, int64_t Nb, int reduce, const int32_t* argmax,
                                 float* dx, int64_t ldx, int* goff, int* err, hipStream_t s) {
  zero_ints<<<1, 64, 0, s>>>(err, 1);
  if (Nb == 0 || F == 0) return TFG_OK;
  const unsigned nb = (unsigned)((Nb + 1 + kBlock - 1) / kBlock);
  if (index_type == TFG_I64)
    segment_bounds<int64_t><<<nb, kBlock, 0, s>>>(static_cast<const int64_t*>(graph_index), Nb, G,
                                                   goff, err);
  else
    segment_bounds<int32_t><<<nb, kBlock, 0, s>>>(static_cast<const int32_t*>(graph_index), Nb, G,
                                                   goff, err);
  TFG_LAUNCHED("segment_bounds");
  auto fits = [&](int v) {
    return F % v == 0 && ldx % v == 0 && reinterpret_cast<uintptr_t>(dx) % (4 * v) == 0 &&
           reinterpret_cast<uintptr_t>(dy) % (4 * v) == 0;
  };
  const int vec = fits(4) ? 4 : fits(2) ? 2 : 1;
  if (index_type == TFG_I64)
    launch_pool_grad<int64_t>(vec, dy, G, (int)F, graph_index, Nb, goff, reduce, argmax, dx, ldx,
                              s);
  else
    launch_pool_grad<int32_t>(vec, dy, G, (int)F, graph_index, Nb, goff, reduce, argmax, dx, ldx,
                              s);
  TFG_LAUNCHED("pool_grad");
  return TFG_OK;
}

int launch_segment_pool(const float* x, int64_t Nb, int64_t F, int64_t ldx, const void* graph_index,
                        int index_type, int64_t G, int reduce, float* out, int32_t* argmax,
                        int* goff, int* err, hipStream_t s) {
  zero_ints<<<1, 64, 0, s>>>(err, 1);
  if (G == 0 || F == 0) return TFG_OK;
  const unsigned nb = (unsigned)((Nb + 1 + kBlock - 1) / kBlock);
  if (index_type == TFG_I64)
    segment_bounds<int64_t><<<nb, kBlock, 0, s>>>(static_cast<const int64_t*>(graph_index), Nb, G,
                                                   goff, err);
  else
    segment_bounds<int32_t><<<nb, kBlock, 0, s>>>(static_cast<const int32_t*>(graph_index), Nb, G,
                                                   goff, err);
  TFG_LAUNCHED("segment_bounds");
  auto fits = [&](int v) {
    return F % v == 0 && ldx % v == 0 && reinterpret_cast<uintptr_t>(x) % (4 * v) == 0;
  };
  const int vec = fits(4) ? 4 : fits(2) ? 2 : 1;
  int lanes = (int)std::min<int64_t>((F + vec - 1) / vec, kWave);
  int p2 = 1;
  while (p2 < lanes) p2 <<= 1;
  const int slots = std::min(kWave / p2, 16);
  dim3 grid((unsigned)((G + kItemBlock / kWave - 1) / (kItemBlock / kWave)));
  if (reduce == TFG_MAX)
    launch_pool_vec<true>(vec, slots, grid, s, x, ldx, (int)F, goff, G, Nb, 0, out, argmax);
  else
    launch_pool_vec<false>(vec, slots, grid, s, x, ldx, (int)F, goff, G, Nb,
                           reduce == TFG_MEAN, out, argmax);
  TFG_LAUNCHED("pool_rows");
  return TFG_OK;
}

}  // namespace tfg
