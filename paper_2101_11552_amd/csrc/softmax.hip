// Attention map -> reduce -> map (gfx950):
//   gat scores: per node and head, the dot products with a_src / a_dst; per
//               edge, LeakyReLU of their sum (the first map);
//   segment softmax: per target row and head, the maximum and the sum of the
//               shifted exponentials (the reduce, in one online sweep) and the
//               division (the last map), one wavefront per work item of the
//               graph's row plan.
#include "softmax_stats.h"

namespace tfg {
namespace {

typedef float f2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));

// a_s[n, k] = sum_d a_src[k, d] h[n, k*D + d]; a_d likewise (float32, d ascending).
__global__ __launch_bounds__(kBlock) void node_projections(const float* __restrict__ h, int64_t N,
                                                           int H, int D,
                                                           const float* __restrict__ a_src,
                                                           const float* __restrict__ a_dst,
                                                           float* __restrict__ as,
                                                           float* __restrict__ ad) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (node, head)
  if (i >= N * H) return;
  const int k = (int)(i % H);
  const float* hv = h + i * D;  // h[n, k*D ...] == h + (n*H + k) * D
  const float* s = a_src + (int64_t)k * D;
  const float* t = a_dst + (int64_t)k * D;
  float x = 0.0f, y = 0.0f;
  for (int d = 0; d < D; ++d) {
    const float v = hv[d];
    x = __builtin_fmaf(s[d], v, x);
    y = __builtin_fmaf(t[d], v, y);
  }
  as[i] = x;
  ad[i] = y;
}

// The same projections with lanes = (node, V columns): 64 / LPS nodes per
// wave, the V-column partial dots summed over the G = D / V lanes of each
// head with xor butterflies (G a power of two dividing LPS).
template <int V>
__global__ __launch_bounds__(kBlock) void node_projections_vec(
    const float* __restrict__ h, int64_t N, int H, int D, int LPS, int G,
    const float* __restrict__ a_src, const float* __restrict__ a_dst, float* __restrict__ as,
    float* __restrict__ ad) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  const int64_t n = wave * (kWave / LPS) + lane / LPS;
  const int sl = lane % LPS;
  const int F = H * D;
  const int f = sl * V;
  const bool ok = n < N && f < F;
  float x = 0.0f, y = 0.0f;
  if (ok) {
    float t[V];
    const float* hv = h + n * F + f;
    if constexpr (V == 4) {
      const f4 q = *reinterpret_cast<const f4*>(hv);
      t[0] = q.x; t[1] = q.y; t[2] = q.z; t[3] = q.w;
    } else if constexpr (V == 2) {
      const f2 q = *reinterpret_cast<const f2*>(hv);
      t[0] = q.x; t[1] = q.y;
    } else {
      t[0] = hv[0];
    }
#pragma unroll
    for (int v = 0; v < V; ++v) {
      x = __builtin_fmaf(a_src[f + v], t[v], x);
      y = __builtin_fmaf(a_dst[f + v], t[v], y);
    }
  }
  for (int off = 1; off < G; off <<= 1) {
    x += __shfl_xor(x, off);
    y += __shfl_xor(y, off);
  }
  if (ok && sl % G == 0) {
    as[n * H + sl / G] = x;
    ad[n * H + sl / G] = y;
  }
}

// Launches the vectorised projections when the shape allows, else the simple ones.
void projections(const float* h, int64_t N, int H, int D, const float* a_src, const float* a_dst,
                 float* as, float* ad, hipStream_t s) {
  const int F = H * D;
  int vec = 1;
  for (int v : {4, 2}) {
    if (D % v == 0 && reinterpret_cast<uintptr_t>(h) % (4 * v) == 0) {
      vec = v;
      break;
    }
  }
  const int G = D / vec;
  const int lanes = F / vec;
  if ((G & (G - 1)) == 0 && lanes <= kWave) {
    int lps = 1;
    while (lps < lanes) lps <<= 1;
    const int64_t waves = (N + kWave / lps - 1) / (kWave / lps);
    const unsigned nb = (unsigned)((waves * kWave + kBlock - 1) / kBlock);
    if (vec == 4)
      node_projections_vec<4><<<nb, kBlock, 0, s>>>(h, N, H, D, lps, G, a_src, a_dst, as, ad);
    else if (vec == 2)
      node_projections_vec<2><<<nb, kBlock, 0, s>>>(h, N, H, D, lps, G, a_src, a_dst, as, ad);
    else
      node_projections_vec<1><<<nb, kBlock, 0, s>>>(h, N, H, D, lps, G, a_src, a_dst, as, ad);
  } else {
    node_projections<<<(unsigned)((N * H + kBlock - 1) / kBlock), kBlock, 0, s>>>(h, N, H, D, a_src,
                                                                                 a_dst, as, ad);
  }
}

template <typename IdxT>
__global__ __launch_bounds__(kBlock) void edge_scores(const IdxT* __restrict__ src,
                                                      const IdxT* __restrict__ tgt, int64_t E,
                                                      int64_t N, int H,
                                                      const float* __restrict__ as,
                                                      const float* __restrict__ ad, float slope,
                                                      float* __restrict__ out,
                                                      int* __restrict__ err) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (edge, head)
  if (i >= E * H) return;
  const int64_t e = i / H;
  const int k = (int)(i - e * H);
  int64_t s = (int64_t)src[e], t = (int64_t)tgt[e];
  if (s < 0 || s >= N || t < 0 || t >= N) {
    atomicOr(err, kErrIndex);
    s = (s < 0 || s >= N) ? 0 : s;
    t = (t < 0 || t >= N) ? 0 : t;
  }
  const float z = as[s * H + k] + ad[t * H + k];
  out[i] = z >= 0.0f ? z : slope * z;
}

// Short rows (at most kShortRow edges), 64 / HP per wavefront: lane (r, hh)
// takes row short_rows[i] and heads hh, hh + HP, ...; the row's scores are
// loaded at once and kept in registers: maximum, then the sum of exp(s - m)
// in double in graph order, then alpha. No cross-lane traffic.
__device__ __forceinline__ void softmax_short_row(const WorkItem& it,
                                                  const int* __restrict__ perm,
                                                  const float* __restrict__ s, int H, int hh,
                                                  int HP, float* __restrict__ out,
                                                  float* __restrict__ out_csr) {
  const int kb = it.kbeg, n = it.kend - it.kbeg;  // 0 <= n <= kShortRow
  int e[kShortRow];
#pragma unroll
  for (int j = 0; j < kShortRow; ++j) e[j] = j < n ? perm[kb + j] : 0;
  for (int h = hh; h < H; h += HP) {
    float v[kShortRow];
    float m = -__builtin_huge_valf();
#pragma unroll
    for (int j = 0; j < kShortRow; ++j) {
      v[j] = j < n ? s[(int64_t)e[j] * H + h] : 0.0f;
      if (j < n) m = v[j] > m ? v[j] : m;
    }
    double d = 0.0;
#pragma unroll
    for (int j = 0; j < kShortRow; ++j) {
      v[j] = expf(v[j] - m);
      if (j < n) d += (double)v[j];
    }
#pragma unroll
    for (int j = 0; j < kShortRow; ++j)
      if (j < n) {
        const float a = (float)((double)v[j] / d);
        out[(int64_t)e[j] * H + h] = a;
        if (out_csr) out_csr[(int64_t)(kb + j) * H + h] = a;
      }
  }
}

// Short rows, 64 / HP per wavefront (a kernel of its own: its registers would
// lower the occupancy of the sweep below).
__global__ __launch_bounds__(kItemBlock) void softmax_short(const WorkItem* __restrict__ short_rows,
                                                        int n_short,
                                                        const int* __restrict__ perm,
                                                        const float* __restrict__ s, int H, int HP,
                                                        float* __restrict__ out,
                                                        float* __restrict__ out_csr) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  const int64_t i = wave * (kWave / HP) + lane / HP;
  if (i < n_short) softmax_short_row(short_rows[i], perm, s, H, lane % HP, HP, out, out_csr);
}

// kSmSteps slot steps (positions k0, k0 + SL, ...) at a time: the edge ids,
// then the scores, issued together (e < 0: past the item or an inactive head).
constexpr int kSmSteps = 4;
__device__ __forceinline__ void load_steps(const int* __restrict__ perm,
                                           const float* __restrict__ s, int H, int h, bool act,
                                           int k0, int SL, int ke, int64_t (&e)[kSmSteps],
                                           float (&v)[kSmSteps]) {
#pragma unroll
  for (int u = 0; u < kSmSteps; ++u) {
    const int k = k0 + u * SL;
    e[u] = (act && k < ke) ? (int64_t)perm[k] : -1;
  }
#pragma unroll
  for (int u = 0; u < kSmSteps; ++u) v[u] = e[u] >= 0 ? s[e[u] * H + h] : 0.0f;
}

// The other buckets of the row plan: wavefronts [0, n_heavy) take the chunks
// of long rows, the rest one other light row each. Lanes are (slot, head) pairs: HP
// heads (a power of two) per pass and 64 / HP edge slots; each lane keeps the
// maximum m of the scores it has seen and d = sum of exp(s - m) (in double),
// rescaling d when m grows, so the maximum and the denominator come out of
// one sweep; the slots are combined with xor butterflies (every lane of a
// head ends with the same pair). A whole row then writes alpha = exp(s - m) /
// d; a chunk stores its pair, and softmax_write combines the pairs of each
// long row in chunk order and writes the chunk's outputs.
__global__ __launch_bounds__(kItemBlock) void softmax_items(
    const WorkItem* __restrict__ heavy, int n_heavy, const WorkItem* __restrict__ long_rows,
    int n_long, const int* __restrict__ perm, const float* __restrict__ s, int H, int HP,
    float* __restrict__ out, float* __restrict__ out_csr, float* __restrict__ pm,
    double* __restrict__ pd) {
  const int wid = uniform(blockIdx.x * (kItemBlock / kWave) + threadIdx.x / kWave);
  if (wid >= n_heavy + n_long) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int SL = kWave / HP;
  const int slot = lane / HP, hh = lane % HP;
  int kb, ke, pslot;
  if (wid < n_heavy) {
    kb = uniform(heavy[wid].kbeg);
    ke = uniform(heavy[wid].kend);
    pslot = uniform(heavy[wid].slot);
  } else {
    kb = uniform(long_rows[wid - n_heavy].kbeg);
    ke = uniform(long_rows[wid - n_heavy].kend);
    pslot = -1;
  }
  for (int hb = 0; hb < H; hb += HP) {
    const int h = hb + hh;
    const bool act = h < H;
    float m = -__builtin_huge_valf();
    double d = 0.0;
    for (int k0 = kb + slot; k0 < ke; k0 += kSmSteps * SL) {
      int64_t e[kSmSteps];
      float v[kSmSteps];
      load_steps(perm, s, H, h, act, k0, SL, ke, e, v);
#pragma unroll
      for (int u = 0; u < kSmSteps; ++u)
        if (e[u] >= 0) stat_add(m, d, v[u]);
    }
    for (int off = HP; off < kWave; off <<= 1) {
      const float m2 = __shfl_xor(m, off);
      const double d2 = __shfl_xor(d, off);
      stat_merge(m, d, m2, d2);
    }
    if (pslot >= 0) {
      if (slot == 0 && act) {
        pm[(int64_t)pslot * H + h] = m;
        pd[(int64_t)pslot * H + h] = d;
      }
      continue;
    }
    for (int k0 = kb + slot; k0 < ke; k0 += kSmSteps * SL) {
      int64_t e[kSmSteps];
      float v[kSmSteps];
      load_steps(perm, s, H, h, act, k0, SL, ke, e, v);
#pragma unroll
      for (int u = 0; u < kSmSteps; ++u)
        if (e[u] >= 0) {
          const float a = (float)((double)expf(v[u] - m) / d);
          out[e[u] * H + h] = a;
          if (out_csr) out_csr[(int64_t)(k0 + u * SL) * H + h] = a;
        }
    }
  }
}

// The outputs of the chunks of long rows. Each chunk combines the pairs of
// all chunks of its row in chunk order (the chunks of a row are consecutive
// slots of `chunk` edges each, the last one shorter), so every chunk of the
// row gets the same pair, then writes its alpha.
__global__ __launch_bounds__(kItemBlock) void softmax_write(
    const WorkItem* __restrict__ heavy, int n_heavy, const int* __restrict__ rowptr, int chunk,
    const int* __restrict__ perm, const float* __restrict__ s, int H, int HP,
    const float* __restrict__ pm, const double* __restrict__ pd, float* __restrict__ out,
    float* __restrict__ out_csr) {
  const int wid = uniform(blockIdx.x * (kItemBlock / kWave) + threadIdx.x / kWave);
  if (wid >= n_heavy) return;
  const WorkItem* itp = heavy + wid;
  const int kb = uniform(itp->kbeg), ke = uniform(itp->kend), pslot = uniform(itp->slot);
  const int row = uniform(itp->row);
  const int rb = uniform(rowptr[row]), re = uniform(rowptr[row + 1]);
  const int s0 = pslot - (kb - rb) / chunk, nch = (re - rb + chunk - 1) / chunk;
  const int lane = threadIdx.x & (kWave - 1);
  const int SL = kWave / HP;
  const int slot = lane / HP, hh = lane % HP;
  for (int hb = 0; hb < H; hb += HP) {
    const int h = hb + hh;
    if (h >= H) continue;
    float m = -__builtin_huge_valf();
    double d = 0.0;
    for (int j = 0; j < nch; ++j)
      stat_merge(m, d, pm[(int64_t)(s0 + j) * H + h], pd[(int64_t)(s0 + j) * H + h]);
    for (int k0 = kb + slot; k0 < ke; k0 += kSmSteps * SL) {
      int64_t e[kSmSteps];
      float v[kSmSteps];
      load_steps(perm, s, H, h, true, k0, SL, ke, e, v);
#pragma unroll
      for (int u = 0; u < kSmSteps; ++u)
        if (e[u] >= 0) {
          const float a = (float)((double)expf(v[u] - m) / d);
          out[e[u] * H + h] = a;
          if (out_csr) out_csr[(int64_t)(k0 + u * SL) * H + h] = a;
        }
    }
  }
}

}  // namespace

int launch_node_projections(const float* h, int64_t N, int H, int D, const float* a_src,
                            const float* a_dst, float* as, float* ad, hipStream_t s) {
  if (N * H == 0) return TFG_OK;
  projections(h, N, H, D, a_src, a_dst, as, ad, s);
  TFG_LAUNCHED("node_projections");
  return TFG_OK;
}

int launch_gat_scores(const void* edge_index, int index_type, int64_t E, const float* h, int64_t N,
                      int H, int D, const float* a_src, const float* a_dst, float slope,
                      float* out, float* proj, int* err, hipStream_t s) {
  float* as = proj;
  float* ad = proj + N * H;
  if (N * H > 0) {
    projections(h, N, H, D, a_src, a_dst, as, ad, s);
    TFG_LAUNCHED("node_projections");
  }
  if (E * H > 0) {
    const unsigned nb = (unsigned)((E * H + kBlock - 1) / kBlock);
    if (index_type == TFG_I64) {
      const int64_t* ei = static_cast<const int64_t*>(edge_index);
      edge_scores<int64_t><<<nb, kBlock, 0, s>>>(ei, ei + E, E, N, H, as, ad, slope, out, err);
    } else {
      const int32_t* ei = static_cast<const int32_t*>(edge_index);
      edge_scores<int32_t><<<nb, kBlock, 0, s>>>(ei, ei + E, E, N, H, as, ad, slope, out, err);
    }
    TFG_LAUNCHED("edge_scores");
  }
  return TFG_OK;
}

size_t row_stats_bytes(int64_t n_chunks, int64_t H) {
  const size_t n = (size_t)std::max<int64_t>(n_chunks * H, 1);
  return align_up(sizeof(float) * n, 256) + align_up(sizeof(double) * n, 256);
}

int launch_segment_softmax(const Graph& g, const float* scores, int H, float* out, float* out_csr,
                           void* ws, hipStream_t s) {
  if (g.N == 0 || g.E == 0 || H == 0) return TFG_OK;
  int hp = 1;
  while (hp * 2 <= std::min(H, kWave)) hp *= 2;
  float* pm = static_cast<float*>(ws);
  double* pd = reinterpret_cast<double*>(
      static_cast<char*>(ws) + align_up(sizeof(float) * (size_t)std::max<int64_t>((int64_t)g.n_heavy * H, 1), 256));
  const int64_t short_waves = (g.n_short + kWave / hp - 1) / (kWave / hp);
  if (short_waves > 0) {
    softmax_short<<<(unsigned)((short_waves + (kItemBlock / kWave) - 1) / (kItemBlock / kWave)), kItemBlock, 0, s>>>(
        g.short_rows, g.n_short, g.perm, scores, H, hp, out, out_csr);
    TFG_LAUNCHED("softmax_short");
  }
  const int waves = g.n_heavy + g.n_long;
  if (waves > 0) {
    softmax_items<<<(unsigned)((waves + (kItemBlock / kWave) - 1) / (kItemBlock / kWave)), kItemBlock, 0, s>>>(
        g.heavy, g.n_heavy, g.long_rows, g.n_long, g.perm, scores, H, hp, out, out_csr, pm, pd);
    TFG_LAUNCHED("softmax_items");
  }
  if (g.n_split > 0) {
    softmax_write<<<(unsigned)((g.n_heavy + (kItemBlock / kWave) - 1) / (kItemBlock / kWave)), kItemBlock, 0, s>>>(
        g.heavy, g.n_heavy, g.rowptr, g.chunk, g.perm, scores, H, hp, pm, pd, out, out_csr);
    TFG_LAUNCHED("softmax_write");
  }
  return TFG_OK;
}

}  // namespace tfg
