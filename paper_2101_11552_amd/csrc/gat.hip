// Fused attention aggregation (gfx950): for every target row, the score map,
// the per-head segment softmax and the weighted per-head sum of Fig. 5(a) in
// one sweep over the row's edges. Nothing per edge is written to memory unless
// the attention coefficients are requested.
//
// Rows of at most kShortRow edges go one per edge slot (several per
// wavefront), with every gather of the row in flight at once. Otherwise one
// wavefront per work item of the graph's row plan (a whole row, or a chunk of
// a long row). Lanes are (edge slot, V features) as in the
// aggregation kernel: every lane gathers its V features of the source row and
// what its head's score needs (the source's projection a_s for the additive
// GAT score, its V columns of the key row for the scaled dot product), forms
// the score and folds it into a running triple (maximum m,
// denominator d in double, numerators acc): when the maximum grows, d and acc
// are rescaled by exp(m_old - m_new). Each lane keeps U independent triples;
// they are merged pairwise, then across the slots. A whole row writes
// out = acc / d; a chunk writes its triple and gat_merge combines the chunks
// of each long row in chunk order. The optional coefficients
// alpha = exp(s - m) / d are written in a second sweep with lanes = (slot,
// head). For the additive score the node projections a_s = a_src . h and
// a_d = a_dst . h come from node_projections() (softmax.hip) and sit in the
// workspace.
#include <initializer_list>

#include "softmax_stats.h"

namespace tfg {
namespace {

typedef float f2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kMaxHeads = 64;

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

// Value held by lane (jbase + slot); jbase is wave-uniform. Runs with the
// whole wave active.
template <int SLOTS>
__device__ __forceinline__ int bcast(int v, int jbase, int slot) {
  if constexpr (SLOTS == 1) {
    return __builtin_amdgcn_readlane(v, jbase);
  } else if constexpr (SLOTS == 2) {
    int a = __builtin_amdgcn_readlane(v, jbase);
    int b = __builtin_amdgcn_readlane(v, jbase + 1);
    return slot ? b : a;
  } else {
    return __shfl(v, jbase + slot);
  }
}

__device__ __forceinline__ float leaky(float z, float slope) { return z >= 0.0f ? z : slope * z; }

// Merges the triple (m2, d2, a2) into (m, d, a); an empty triple has m = -inf.
template <int V>
__device__ __forceinline__ void triple_merge(float& m, double& d, float (&a)[V], float m2,
                                             double d2, const float (&a2)[V]) {
#pragma clang fp contract(off)
  if (m2 == -__builtin_huge_valf()) return;
  if (m == -__builtin_huge_valf()) {
    m = m2;
    d = d2;
#pragma unroll
    for (int v = 0; v < V; ++v) a[v] = a2[v];
    return;
  }
  const float mn = m2 > m ? m2 : m;
  const float x = expf(m - mn), y = expf(m2 - mn);
  d = d * (double)x + d2 * (double)y;
#pragma unroll
  for (int v = 0; v < V; ++v) a[v] = a[v] * x + a2[v] * y;
  m = mn;
}

// The two score maps. Additive (GAT): s = LeakyReLU(a_s[src, k] + a_d[t, k])
// from the node projections. Scaled dot product (the Transformer-style GAT,
// Sec. 4.2): s = scale * <q[t, k], key[src, k]> over the D columns of head k;
// a lane holds V of them, and the partial products are summed over the G =
// D / V lanes of the head with xor shuffles (every lane of the head gets the
// score).
struct Scores {
  const float* as;  // additive: [N, H]
  const float* ad;
  float slope;
  const float* q;  // dot product: [N, H*D]
  const float* key;
  float scale;
  int G;  // lanes per head (dot product)
};

template <bool DOT>
__device__ __forceinline__ float group_sum(float v, int G) {
  for (int o = 1; o < G; o <<= 1) v += __shfl_xor(v, o);
  return v;
}

// Score of edge (c -> t) at head k for one lane holding all D columns (the
// coefficient sweeps, lanes = (slot, head)).
template <bool DOT>
__device__ __forceinline__ float lane_score(const Scores& sc, int64_t c, int64_t t, int k, int H,
                                            int D) {
  if constexpr (DOT) {
    const int64_t F = (int64_t)H * D;
    const float* qa = sc.q + t * F + (int64_t)k * D;
    const float* ka = sc.key + c * F + (int64_t)k * D;
    float acc = 0.0f;
    for (int d = 0; d < D; ++d) acc = __builtin_fmaf(qa[d], ka[d], acc);
    return sc.scale * acc;
  } else {
    return leaky(sc.as[c * H + k] + sc.ad[t * H + k], sc.slope);
  }
}

// A short row (at most kShortRow edges) per edge slot: the slot's lanes load
// the row's column ids, scores and feature rows at once, take the maximum,
// then the weighted sums (denominator in double) in graph order. valid = false
// (a slot past the list) runs the same steps on no edges, so that the
// shuffles of the dot-product scores see the whole wave.
template <int V, bool DOT>
__device__ __forceinline__ void gat_short_row(bool valid, int t, int kb, int n, int sl, int LPS,
                                              const int* __restrict__ col,
                                              const int* __restrict__ perm, int H, int D,
                                              const Scores& S, const float* __restrict__ h,
                                              float* __restrict__ out,
                                              float* __restrict__ alpha_out) {
  const int F = H * D;  // 0 <= n <= kShortRow (0 when !valid)
  int c[kShortRow];
#pragma unroll
  for (int j = 0; j < kShortRow; ++j) c[j] = j < n ? col[kb + j] : 0;
  for (int f0 = 0; f0 < F; f0 += LPS * V) {
    const int f = f0 + sl * V;
    const bool fok = f < F;
    const int head = fok ? f / D : 0;
    float qv[V];
    float adt = 0.0f;
    if constexpr (DOT) {
      if (fok && n > 0) {
        load_row<V>(S.q + (int64_t)t * F + f, qv);
      } else {
#pragma unroll
        for (int v = 0; v < V; ++v) qv[v] = 0.0f;
      }
    } else {
      adt = n > 0 ? S.ad[(int64_t)t * H + head] : 0.0f;
    }
    float sc[kShortRow], xv[kShortRow][V];
    float m = -__builtin_huge_valf();
#pragma unroll
    for (int j = 0; j < kShortRow; ++j) {
      const bool use = j < n && fok;
      if (use) {
        load_row<V>(h + (int64_t)c[j] * F + f, xv[j]);
      } else {
#pragma unroll
        for (int v = 0; v < V; ++v) xv[j][v] = 0.0f;
      }
      if constexpr (DOT) {
        float kv[V];
        if (use) {
          load_row<V>(S.key + (int64_t)c[j] * F + f, kv);
        } else {
#pragma unroll
          for (int v = 0; v < V; ++v) kv[v] = 0.0f;
        }
        float p = 0.0f;
#pragma unroll
        for (int v = 0; v < V; ++v) p = __builtin_fmaf(qv[v], kv[v], p);
        sc[j] = S.scale * group_sum<DOT>(p, S.G);
      } else {
        sc[j] = j < n ? leaky(S.as[(int64_t)c[j] * H + head] + adt, S.slope) : 0.0f;
      }
      if (j < n) m = sc[j] > m ? sc[j] : m;
    }
    double d = 0.0;
    float acc[V];
#pragma unroll
    for (int v = 0; v < V; ++v) acc[v] = 0.0f;
#pragma unroll
    for (int j = 0; j < kShortRow; ++j) {
      sc[j] = j < n ? expf(sc[j] - m) : 0.0f;
      d += (double)sc[j];
#pragma unroll
      for (int v = 0; v < V; ++v) acc[v] = __builtin_fmaf(sc[j], xv[j][v], acc[v]);
    }
    if (valid && fok) {
#pragma unroll
      for (int v = 0; v < V; ++v)
        out[(int64_t)t * F + f + v] = n > 0 ? (float)((double)acc[v] / d) : 0.0f;
      if (alpha_out != nullptr && f % D == 0)
#pragma unroll
        for (int j = 0; j < kShortRow; ++j)
          if (j < n) alpha_out[(int64_t)perm[kb + j] * H + head] = (float)((double)sc[j] / d);
    }
  }
}

// SLOTS short rows per wavefront, one per edge slot (gat_short_row). A kernel
// of its own: holding a whole short row in registers takes more of them than
// the sweep of gat_items, whose occupancy it would otherwise lower.
template <int V, int SLOTS, bool DOT>
__global__ __launch_bounds__(kItemBlock) void gat_short(
    const WorkItem* __restrict__ short_rows, int n_short,
    const int* __restrict__ col, const int* __restrict__ perm, int H, int D, Scores S,
    const float* __restrict__ h, float* __restrict__ out, float* __restrict__ alpha_out) {
  constexpr int LPS = kWave / SLOTS;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  const int64_t i = wave * SLOTS + lane / LPS;
  const bool valid = i < n_short;
  const WorkItem it = valid ? short_rows[i] : WorkItem{0, 0, 0, -1};
  gat_short_row<V, DOT>(valid, it.row, it.kbeg, it.kend - it.kbeg, lane % LPS, LPS, col, perm, H,
                        D, S, h, out, alpha_out);
}

// Wavefronts [0, n_heavy) take the chunks of long rows, [n_heavy, n_heavy +
// n_long) one other light row each, with the running-triple sweep.
template <int V, int SLOTS, bool DOT>
__global__ __launch_bounds__(kItemBlock) void gat_items(
    const WorkItem* __restrict__ heavy, int n_heavy, const WorkItem* __restrict__ long_rows,
    int n_long, const int* __restrict__ col, const int* __restrict__ perm, int H, int D, int HP,
    Scores S, const float* __restrict__ h,
    float* __restrict__ out, float* __restrict__ alpha_out, float* __restrict__ pacc,
    float* __restrict__ pm, double* __restrict__ pd) {
  constexpr int LPS = kWave / SLOTS;
  constexpr int FC = LPS * V;
  constexpr int U = SLOTS * 4 <= kWave ? 4 : kWave / SLOTS;
  __shared__ float s_max[kItemBlock / kWave][kMaxHeads];
  __shared__ double s_den[kItemBlock / kWave][kMaxHeads];
  const int wv = threadIdx.x / kWave;
  const int wid = uniform(blockIdx.x * (kItemBlock / kWave) + wv);
  if (wid >= n_heavy + n_long) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int slot = lane / LPS, sl = lane % LPS;
  int row, kb, ke, pslot;
  if (wid < n_heavy) {
    row = uniform(heavy[wid].row);
    kb = uniform(heavy[wid].kbeg);
    ke = uniform(heavy[wid].kend);
    pslot = uniform(heavy[wid].slot);
  } else {
    const WorkItem* it = long_rows + (wid - n_heavy);
    row = uniform(it->row);
    kb = uniform(it->kbeg);
    ke = uniform(it->kend);
    pslot = -1;
  }
  const int F = H * D;
  for (int f0 = 0; f0 < F; f0 += FC) {
    const int f = f0 + sl * V;
    const bool fok = f < F;
    const int head = fok ? f / D : 0;
    float qv[V];
    float adt = 0.0f;
    if constexpr (DOT) {
      if (fok) {
        load_row<V>(S.q + (int64_t)row * F + f, qv);
      } else {
#pragma unroll
        for (int v = 0; v < V; ++v) qv[v] = 0.0f;
      }
    } else {
      adt = S.ad[(int64_t)row * H + head];
    }
    float acc[U][V];
    double den[U];
    float mx[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      den[u] = 0.0;
      mx[u] = -__builtin_huge_valf();
#pragma unroll
      for (int v = 0; v < V; ++v) acc[u][v] = 0.0f;
    }
    for (int kc = kb; kc < ke; kc += kWave) {
      const int n = min(kWave, ke - kc);
      const int cj = lane < n ? __builtin_nontemporal_load(col + kc + lane) : 0;
      for (int s0 = 0; s0 < n; s0 += SLOTS * U) {
        float xv[U][V];
        float sc[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int jb = s0 + u * SLOTS;
          ok[u] = jb + slot < n;
          const int c = bcast<SLOTS>(cj, jb, slot);
          const bool use = ok[u] && fok;
          if (use) {
            load_row<V>(h + (int64_t)c * F + f, xv[u]);
          } else {
#pragma unroll
            for (int v = 0; v < V; ++v) xv[u][v] = 0.0f;
          }
          if constexpr (DOT) {
            float kv[V];
            if (use) {
              load_row<V>(S.key + (int64_t)c * F + f, kv);
            } else {
#pragma unroll
              for (int v = 0; v < V; ++v) kv[v] = 0.0f;
            }
            float p = 0.0f;
#pragma unroll
            for (int v = 0; v < V; ++v) p = __builtin_fmaf(qv[v], kv[v], p);
            sc[u] = S.scale * group_sum<DOT>(p, S.G);
          } else {
            sc[u] = ok[u] ? leaky(S.as[(int64_t)c * H + head] + adt, S.slope) : 0.0f;
          }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          // one exponential per edge: t = exp(-|s - m|) is the new edge's
          // weight when the maximum stays, and the rescale factor of the old
          // sums when it grows (then the new edge weighs 1); from m = -inf
          // the factor is 0
          const float dlt = sc[u] - mx[u];
          const float t = expf(-__builtin_fabsf(dlt));
          const bool up = dlt > 0.0f;
          const float r = ok[u] ? (up ? t : 1.0f) : 1.0f;
          const float w = ok[u] ? (up ? 1.0f : t) : 0.0f;
          mx[u] = (ok[u] && up) ? sc[u] : mx[u];
          den[u] = den[u] * (double)r + (double)w;
#pragma unroll
          for (int v = 0; v < V; ++v) acc[u][v] = __builtin_fmaf(acc[u][v], r, w * xv[u][v]);
        }
      }
    }
#pragma unroll
    for (int step = 1; step < U; step <<= 1)
#pragma unroll
      for (int u = 0; u + step < U; u += 2 * step)
        triple_merge<V>(mx[u], den[u], acc[u], mx[u + step], den[u + step], acc[u + step]);
#pragma unroll
    for (int off = LPS; off < kWave; off <<= 1) {
      float a2[V];
#pragma unroll
      for (int v = 0; v < V; ++v) a2[v] = __shfl_xor(acc[0][v], off);
      const float m2 = __shfl_xor(mx[0], off);
      const double d2 = __shfl_xor(den[0], off);
      triple_merge<V>(mx[0], den[0], acc[0], m2, d2, a2);
    }
    if (slot == 0 && fok) {
      if (pslot < 0) {
#pragma unroll
        for (int v = 0; v < V; ++v)
          out[(int64_t)row * F + f + v] = (float)((double)acc[0][v] / den[0]);
        if (alpha_out != nullptr && f % D == 0) {
          s_max[wv][head] = mx[0];
          s_den[wv][head] = den[0];
        }
      } else {
#pragma unroll
        for (int v = 0; v < V; ++v) pacc[(int64_t)pslot * F + f + v] = acc[0][v];
        if (f % D == 0) {
          pm[(int64_t)pslot * H + head] = mx[0];
          pd[(int64_t)pslot * H + head] = den[0];
        }
      }
    }
  }
  if (alpha_out == nullptr || pslot >= 0) return;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // attention coefficients of a whole row, in the caller's edge order
  const int SL = kWave / HP;
  const int slot3 = lane / HP, hh = lane % HP;
  if (hh < H) {
    const float mh = s_max[wv][hh];
    const double dn = s_den[wv][hh];
    for (int k = kb + slot3; k < ke; k += SL) {
      const float w = expf(lane_score<DOT>(S, col[k], row, hh, H, D) - mh);
      alpha_out[(int64_t)perm[k] * H + hh] = (float)((double)w / dn);
    }
  }
}

// One wavefront per long row: the chunks' triples merged in chunk order
// (lanes over the features, one column each), out = acc / d. With alpha
// requested the row's (m, d) per head is written back to every chunk slot.
__global__ __launch_bounds__(kItemBlock) void gat_merge(const SplitRow* __restrict__ split,
                                                    int n_split, int H, int D,
                                                    float* __restrict__ pacc,
                                                    float* __restrict__ pm,
                                                    double* __restrict__ pd,
                                                    float* __restrict__ out, int write_back) {
  const int wid = uniform(blockIdx.x * (kItemBlock / kWave) + threadIdx.x / kWave);
  if (wid >= n_split) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int row = uniform(split[wid].row), s0 = uniform(split[wid].slot0);
  const int nch = uniform(split[wid].nchunks);
  const int F = H * D;
  for (int f = lane; f < F; f += kWave) {
    const int head = f / D;
    float m = -__builtin_huge_valf();
    double d = 0.0;
    float a[1] = {0.0f};
    for (int j = 0; j < nch; ++j) {
      const float a2[1] = {pacc[(int64_t)(s0 + j) * F + f]};
      triple_merge<1>(m, d, a, pm[(int64_t)(s0 + j) * H + head], pd[(int64_t)(s0 + j) * H + head],
                      a2);
    }
    out[(int64_t)row * F + f] = (float)((double)a[0] / d);
    if (write_back && f % D == 0)
      for (int j = 0; j < nch; ++j) {
        pm[(int64_t)(s0 + j) * H + head] = m;
        pd[(int64_t)(s0 + j) * H + head] = d;
      }
  }
}

// Attention coefficients of the chunks of long rows, from their row's (m, d).
template <bool DOT>
__global__ __launch_bounds__(kItemBlock) void gat_alpha_chunks(
    const WorkItem* __restrict__ heavy, int n_heavy, const int* __restrict__ col,
    const int* __restrict__ perm, int H, int D, int HP, Scores S, const float* __restrict__ pm,
    const double* __restrict__ pd, float* __restrict__ alpha_out) {
  const int wid = uniform(blockIdx.x * (kItemBlock / kWave) + threadIdx.x / kWave);
  if (wid >= n_heavy) return;
  const WorkItem* itp = heavy + wid;
  const int row = uniform(itp->row), kb = uniform(itp->kbeg), ke = uniform(itp->kend);
  const int pslot = uniform(itp->slot);
  const int lane = threadIdx.x & (kWave - 1);
  const int SL = kWave / HP;
  const int slot = lane / HP, hh = lane % HP;
  if (hh >= H) return;
  const float mh = pm[(int64_t)pslot * H + hh];
  const double dn = pd[(int64_t)pslot * H + hh];
  for (int k = kb + slot; k < ke; k += SL) {
    const float w = expf(lane_score<DOT>(S, col[k], row, hh, H, D) - mh);
    alpha_out[(int64_t)perm[k] * H + hh] = (float)((double)w / dn);
  }
}

struct GatArgs {
  const Graph* g;
  int H, D, HP;
  Scores S;
  const float* h;  // the rows that are summed (h, or the values)
  float* out;
  float* alpha_out;
  float* pacc;
  float* pm;
  double* pd;
};

template <int V, bool DOT>
void launch_slots(int slots, dim3 grid, hipStream_t s, const GatArgs& a) {
  const Graph& g = *a.g;
  const int waves = g.n_heavy + g.n_long;
  const int64_t short_waves = (g.n_short + slots - 1) / slots;
  const dim3 sgrid((unsigned)((short_waves + kItemBlock / kWave - 1) / (kItemBlock / kWave)));
#define TFG_GAT(SL)                                                                              \
  do {                                                                                           \
    if (g.n_short > 0)                                                                           \
      gat_short<V, SL, DOT><<<sgrid, kItemBlock, 0, s>>>(g.short_rows, g.n_short, g.col,         \
                                                     g.perm, a.H, a.D, a.S, a.h, a.out,          \
                                                     a.alpha_out);                               \
    if (waves > 0)                                                                               \
      gat_items<V, SL, DOT><<<grid, kItemBlock, 0, s>>>(g.heavy, g.n_heavy, g.long_rows,         \
                                                    g.n_long, g.col, g.perm, a.H,                \
                                                    a.D, a.HP, a.S, a.h, a.out, a.alpha_out,     \
                                                    a.pacc, a.pm, a.pd);                         \
  } while (0)
  switch (slots) {
    case 1: TFG_GAT(1); break;
    case 2: TFG_GAT(2); break;
    case 4: TFG_GAT(4); break;
    case 8: TFG_GAT(8); break;
    default: TFG_GAT(16); break;
  }
#undef TFG_GAT
}

struct GatLayout {
  size_t as, ad, pacc, pm, pd, total;
};

GatLayout gat_layout(int64_t N, int64_t H, int64_t F, int64_t n_chunks) {
  GatLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  L.as = take(sizeof(float) * (size_t)std::max<int64_t>(N * H, 1));
  L.ad = take(sizeof(float) * (size_t)std::max<int64_t>(N * H, 1));
  L.pacc = take(sizeof(float) * (size_t)std::max<int64_t>(n_chunks * F, 1));
  L.pm = take(sizeof(float) * (size_t)std::max<int64_t>(n_chunks * H, 1));
  L.pd = take(sizeof(double) * (size_t)std::max<int64_t>(n_chunks * H, 1));
  L.total = off + 256;
  return L;
}

}  // namespace

size_t gat_aggregate_ws_bytes(const Graph& g, int64_t H, int64_t D) {
  return gat_layout(g.N, H, H * D, g.n_heavy).total;
}

int max_fused_heads() { return kMaxHeads; }

namespace {

// Vector width for rows of D columns at these addresses (every row read or
// written with V-wide accesses).
int gat_vec(int D, std::initializer_list<const float*> ptrs) {
  for (int v : {4, 2}) {
    bool ok = D % v == 0;
    for (const float* p : ptrs) ok = ok && reinterpret_cast<uintptr_t>(p) % (4 * v) == 0;
    if (ok) return v;
  }
  return 1;
}

template <bool DOT>
int run_attention(const Graph& g, GatArgs& a, int vec, hipStream_t s) {
  const int H = a.H, D = a.D;
  const int64_t F = (int64_t)H * D;
  const int lanes = (int)std::min<int64_t>((F + vec - 1) / vec, kWave);
  int p2 = 1;
  while (p2 < lanes) p2 <<= 1;
  const int slots = std::min(kWave / p2, 16);
  int hp = 1;
  while (hp < H) hp <<= 1;  // heads per pass (a power of two, at most 64)
  a.HP = hp;
  const int waves = g.n_heavy + g.n_long;
  if (waves > 0 || g.n_short > 0) {
    dim3 grid((unsigned)((std::max(waves, 1) + kItemBlock / kWave - 1) / (kItemBlock / kWave)));
    if (vec == 4)
      launch_slots<4, DOT>(slots, grid, s, a);
    else if (vec == 2)
      launch_slots<2, DOT>(slots, grid, s, a);
    else
      launch_slots<1, DOT>(slots, grid, s, a);
    TFG_LAUNCHED("gat_items");
  }
  if (g.n_split > 0) {
    dim3 mgrid((unsigned)((g.n_split + (kItemBlock / kWave) - 1) / (kItemBlock / kWave)));
    gat_merge<<<mgrid, kItemBlock, 0, s>>>(g.split, g.n_split, H, D, a.pacc, a.pm, a.pd, a.out,
                                       a.alpha_out != nullptr ? 1 : 0);
    TFG_LAUNCHED("gat_merge");
    if (a.alpha_out != nullptr) {
      dim3 agrid((unsigned)((g.n_heavy + kItemBlock / kWave - 1) / (kItemBlock / kWave)));
      gat_alpha_chunks<DOT><<<agrid, kItemBlock, 0, s>>>(g.heavy, g.n_heavy, g.col, g.perm, H, D, hp,
                                                     a.S, a.pm, a.pd, a.alpha_out);
      TFG_LAUNCHED("gat_alpha_chunks");
    }
  }
  return TFG_OK;
}

GatArgs make_args(const Graph& g, int H, int D, float* out, float* alpha_out, void* ws) {
  const GatLayout L = gat_layout(g.N, H, (int64_t)H * D, g.n_heavy);
  char* base = static_cast<char*>(ws);
  GatArgs a{};
  a.g = &g;
  a.H = H;
  a.D = D;
  a.out = out;
  a.alpha_out = alpha_out;
  a.pacc = reinterpret_cast<float*>(base + L.pacc);
  a.pm = reinterpret_cast<float*>(base + L.pm);
  a.pd = reinterpret_cast<double*>(base + L.pd);
  a.S.as = reinterpret_cast<float*>(base + L.as);
  a.S.ad = reinterpret_cast<float*>(base + L.ad);
  return a;
}

}  // namespace

int launch_gat_aggregate(const Graph& g, const float* h, int H, int D, const float* a_src,
                         const float* a_dst, float slope, float* out, float* alpha_out, void* ws,
                         hipStream_t s) {
  if (g.N == 0 || H == 0 || D == 0) return TFG_OK;
  GatArgs a = make_args(g, H, D, out, alpha_out, ws);
  a.S.slope = slope;
  a.h = h;
  int rc = launch_node_projections(h, g.N, H, D, a_src, a_dst, const_cast<float*>(a.S.as),
                                   const_cast<float*>(a.S.ad), s);
  if (rc) return rc;
  return run_attention<false>(g, a, gat_vec(D, {h, out}), s);
}

bool dot_attention_shape_ok(int64_t D) { return D >= 1 && D <= 64 && (D & (D - 1)) == 0; }

int launch_gat_dot_aggregate(const Graph& g, const float* q, const float* key, const float* v,
                             int H, int D, float scale, float* out, float* alpha_out, void* ws,
                             hipStream_t s) {
  if (g.N == 0 || H == 0 || D == 0) return TFG_OK;
  GatArgs a = make_args(g, H, D, out, alpha_out, ws);
  a.h = v;
  a.S.q = q;
  a.S.key = key;
  a.S.scale = scale;
  const int vec = gat_vec(D, {q, key, v, out});
  a.S.G = D / vec;  // lanes of one head, a power of two that divides the slot width
  return run_attention<true>(g, a, vec, s);
}

}  // namespace tfg
