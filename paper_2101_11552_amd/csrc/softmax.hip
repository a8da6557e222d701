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

// The same scores over a graph handle: one thread per (graph position, head),
// the source from col, the target from the stored sort key (target * parts +
// part), written at the position (graph order) or at the edge id perm[k]
// (the caller's order). Same operands and operations as edge_scores.
__global__ __launch_bounds__(kBlock) void edge_scores_graph(const int* __restrict__ col,
                                                            const int* __restrict__ key,
                                                            const int* __restrict__ perm,
                                                            int parts, int64_t E, int H,
                                                            const float* __restrict__ as,
                                                            const float* __restrict__ ad,
                                                            float slope, float* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (position, head)
  if (i >= E * H) return;
  const int64_t k = i / H;
  const int h = (int)(i - k * H);
  const int64_t sv = col[k], t = key[k] / parts;
  const float z = as[sv * H + h] + ad[t * H + h];
  out[(int64_t)edge_at(perm, (int)k) * H + h] = z >= 0.0f ? z : slope * z;
}

// Short rows (at most kShortRow edges), 64 / HP per wavefront: lane (r, hh)
// takes row short_rows[i] and heads hh, hh + HP, ...; the row's scores are
// loaded at once and kept in registers: maximum, then the sum of exp(s - m)
// in graph order (at most kShortRow terms of at most 1, one of them 1: float
// keeps it within a few units of 2^-24), then alpha = exp(s - m) * (1 / sum).
// No cross-lane traffic.
__device__ __forceinline__ void softmax_short_row(const WorkItem& it,
                                                  const int* __restrict__ perm,
                                                  const float* __restrict__ s, int H, int hh,
                                                  int HP, float* __restrict__ out,
                                                  float* __restrict__ out_csr) {
  const int kb = it.kbeg, n = it.kend - it.kbeg;  // 0 <= n <= kShortRow
  // the wavefront's longest row: steps past it are skipped by all lanes
  int nw = 0;
#pragma unroll
  for (int j = 1; j <= kShortRow; ++j) nw = __any(n >= j) ? j : nw;
  int e[kShortRow];
#pragma unroll
  for (int j = 0; j < kShortRow; ++j) e[j] = j < n ? edge_at(perm, kb + j) : 0;
  for (int h = hh; h < H; h += HP) {
    float v[kShortRow];
    float m = -__builtin_huge_valf();
#pragma unroll
    for (int j = 0; j < kShortRow; ++j) {
      v[j] = j < n ? s[(int64_t)e[j] * H + h] : 0.0f;
      if (j < n) m = v[j] > m ? v[j] : m;
    }
    float d = 0.0f;
#pragma unroll
    for (int j = 0; j < kShortRow; ++j)
      if (j < nw) {
        v[j] = expf(v[j] - m);
        if (j < n) d += v[j];
      }
    const float r = 1.0f / d;
#pragma unroll
    for (int j = 0; j < kShortRow; ++j)
      if (j < n) {
        const float a = v[j] * r;
        out[(int64_t)e[j] * H + h] = a;
        if (out_csr) out_csr[(int64_t)(kb + j) * H + h] = a;
      }
  }
}

// The other rows go one work item (a whole row, or a chunk of a long row)
// per wavefront. Lanes are (slot, head) pairs: HP heads (a power of two) per
// pass and SL = 64 / HP edge slots; slot step u of an item starting at kb is
// position kb + slot + u * SL.
//
// Items of at most kSmCap slot steps are swept once, over NST steps (the
// next power of two, a template argument chosen per item, so that the
// wavefront runs no step that holds none of its edges): their edge ids and
// scores are loaded together and stay in registers, the maximum comes from
// the registers and a butterfly over the slots, then each score is replaced
// by exp(s - m) and summed in double (butterfly again), and alpha is written
// from the registers. Longer items keep a running pair instead (stat_add:
// maximum and rescaled sum in one sweep of loads) and load the scores again
// to write alpha.
constexpr int kSmCap = 8;    // slot steps held in registers
constexpr int kSmSteps = 4;  // slot steps per round of loads (the running sweep)

// Scores of head h for the ids (-inf where there is no edge or no head).
template <int NST>
__device__ __forceinline__ void load_scores(const float* __restrict__ s, int H, int h, bool act,
                                            const int (&e)[NST], float (&v)[NST]) {
#pragma unroll
  for (int u = 0; u < NST; ++u)
    v[u] = (act && e[u] >= 0) ? s[(int64_t)e[u] * H + h] : -__builtin_huge_valf();
}

__device__ __forceinline__ float slots_max(float m, int HP) {
  for (int off = HP; off < kWave; off <<= 1) {
    const float o = __shfl_xor(m, off);
    m = o > m ? o : m;
  }
  return m;
}

__device__ __forceinline__ void slots_merge(float& m, double& d, int HP) {
  for (int off = HP; off < kWave; off <<= 1) {
    const float m2 = __shfl_xor(m, off);
    const double d2 = __shfl_xor(d, off);
    stat_merge(m, d, m2, d2);
  }
}

// Maximum of the registers, over all slots of the head.
template <int NST>
__device__ __forceinline__ float regs_max(const float (&v)[NST], int HP) {
  float m = -__builtin_huge_valf();
#pragma unroll
  for (int u = 0; u < NST; ++u) m = v[u] > m ? v[u] : m;
  return slots_max(m, HP);
}

// Sum of exp(v - m) over all slots of the head (a missing edge, v = -inf,
// adds exp(-inf) = 0): at most kSmCap terms per lane in float, then the
// lanes' sums in double; with KEEP the registers become exp(v - m).
template <int NST, bool KEEP>
__device__ __forceinline__ double regs_exp_sum(float (&v)[NST], float m, int HP) {
  float d = 0.0f;
#pragma unroll
  for (int u = 0; u < NST; ++u) {
    const float x = expf(v[u] - m);
    if (KEEP) v[u] = x;
    d += x;
  }
  return slots_sum((double)d, HP);
}

// alpha = x * r for the registers' edges (x = exp(s - m), r = 1 / sum).
template <int NST>
__device__ __forceinline__ void regs_write(const float (&x)[NST], const int (&e)[NST], float r,
                                           int kb, int slot, int SL, int H, int h, bool act,
                                           float* __restrict__ out,
                                           float* __restrict__ out_csr) {
#pragma unroll
  for (int u = 0; u < NST; ++u)
    if (act && e[u] >= 0) {
      const float a = x[u] * r;
      out[(int64_t)e[u] * H + h] = a;
      if (out_csr) out_csr[(int64_t)(kb + slot + u * SL) * H + h] = a;
    }
}

// kSmSteps slot steps (positions k0, k0 + SL, ...) at a time: the edge ids,
// then the scores, issued together (e < 0: past the item or an inactive head).
__device__ __forceinline__ void load_steps(const int* __restrict__ perm,
                                           const float* __restrict__ s, int H, int h, bool act,
                                           int k0, int SL, int ke, int64_t (&e)[kSmSteps],
                                           float (&v)[kSmSteps]) {
#pragma unroll
  for (int u = 0; u < kSmSteps; ++u) {
    const int k = k0 + u * SL;
    e[u] = (act && k < ke) ? (int64_t)edge_at(perm, k) : -1;
  }
#pragma unroll
  for (int u = 0; u < kSmSteps; ++u) v[u] = e[u] >= 0 ? s[e[u] * H + h] : 0.0f;
}

// The running pair of [kb, ke) for head h, combined over the slots.
__device__ __forceinline__ void sweep_stats(const int* __restrict__ perm,
                                            const float* __restrict__ s, int H, int h, bool act,
                                            int kb, int ke, int slot, int SL, int HP, float& m,
                                            double& d) {
  m = -__builtin_huge_valf();
  d = 0.0;
  for (int k0 = kb + slot; k0 < ke; k0 += kSmSteps * SL) {
    int64_t e[kSmSteps];
    float v[kSmSteps];
    load_steps(perm, s, H, h, act, k0, SL, ke, e, v);
#pragma unroll
    for (int u = 0; u < kSmSteps; ++u)
      if (e[u] >= 0) stat_add(m, d, v[u]);
  }
  slots_merge(m, d, HP);
}

// alpha = exp(s - m) * r over [kb, ke), loading the scores again.
__device__ __forceinline__ void sweep_write(const int* __restrict__ perm,
                                            const float* __restrict__ s, int H, int h, bool act,
                                            int kb, int ke, int slot, int SL, float m, double r,
                                            float* __restrict__ out,
                                            float* __restrict__ out_csr) {
  for (int k0 = kb + slot; k0 < ke; k0 += kSmSteps * SL) {
    int64_t e[kSmSteps];
    float v[kSmSteps];
    load_steps(perm, s, H, h, act, k0, SL, ke, e, v);
#pragma unroll
    for (int u = 0; u < kSmSteps; ++u)
      if (e[u] >= 0) {
        const float a = (float)((double)expf(v[u] - m) * r);
        out[e[u] * H + h] = a;
        if (out_csr) out_csr[(int64_t)(k0 + u * SL) * H + h] = a;
      }
  }
}

// One item from the registers: a whole row (pslot < 0) writes alpha, a chunk
// of a split row its pair.
template <int NST>
__device__ __forceinline__ void item_regs(const int* __restrict__ perm,
                                          const float* __restrict__ s, int H, int HP, int kb,
                                          int ke, int slot, int hh, int pslot,
                                          float* __restrict__ out, float* __restrict__ out_csr,
                                          float* __restrict__ pm, double* __restrict__ pd) {
  const int SL = kWave / HP;
  int e[NST];
  load_ids<NST>(perm, kb, ke, slot, SL, e);
  for (int hb = 0; hb < H; hb += HP) {
    const int h = hb + hh;
    const bool act = h < H;
    float v[NST];
    load_scores<NST>(s, H, h, act, e, v);
    const float m = regs_max<NST>(v, HP);
    const double d = regs_exp_sum<NST, true>(v, m, HP);
    if (pslot >= 0) {
      if (slot == 0 && act) {
        pm[(int64_t)pslot * H + h] = m;
        pd[(int64_t)pslot * H + h] = d;
      }
      continue;
    }
    regs_write<NST>(v, e, (float)(1.0 / d), kb, slot, SL, H, h, act, out, out_csr);
  }
}

// Split rows: a row of more than kSplitWaves chunks has its chunks' pairs
// written here (pm, pd at the chunk's slot) and combined by softmax_split;
// the chunks of the other split rows are left to softmax_split entirely.
constexpr int kSplitWaves = 16;

// Wavefronts [0, short_waves) take 64 / HP short rows each; the next n_long
// one whole light row of more than kShortRow edges each, the rest one chunk
// of a split row.
__global__ __launch_bounds__(kItemBlock) void softmax_items(
    const WorkItem* __restrict__ short_rows, int n_short, int short_waves,
    const WorkItem* __restrict__ long_rows, int n_long, const WorkItem* __restrict__ heavy,
    int n_heavy, const int* __restrict__ rowptr, int chunk, const int* __restrict__ perm,
    const float* __restrict__ s, int H, int HP, float* __restrict__ out,
    float* __restrict__ out_csr, float* __restrict__ pm, double* __restrict__ pd) {
  const int lane = threadIdx.x & (kWave - 1);
  int wid = uniform(blockIdx.x * (kItemBlock / kWave) + threadIdx.x / kWave);
  if (wid < short_waves) {
    const int i = wid * (kWave / HP) + lane / HP;
    if (i < n_short) softmax_short_row(short_rows[i], perm, s, H, lane % HP, HP, out, out_csr);
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
    if ((deg + chunk - 1) / chunk <= kSplitWaves) return;
    kb = uniform(it->kbeg);
    ke = uniform(it->kend);
    pslot = uniform(it->slot);
  }
  const int nst = (ke - kb + SL - 1) / SL;
  if (nst <= 1) {
    item_regs<1>(perm, s, H, HP, kb, ke, slot, hh, pslot, out, out_csr, pm, pd);
  } else if (nst <= 2) {
    item_regs<2>(perm, s, H, HP, kb, ke, slot, hh, pslot, out, out_csr, pm, pd);
  } else if (nst <= 4) {
    item_regs<4>(perm, s, H, HP, kb, ke, slot, hh, pslot, out, out_csr, pm, pd);
  } else if (nst <= kSmCap) {
    item_regs<kSmCap>(perm, s, H, HP, kb, ke, slot, hh, pslot, out, out_csr, pm, pd);
  } else {
    for (int hb = 0; hb < H; hb += HP) {
      const int h = hb + hh;
      const bool act = h < H;
      float m;
      double d;
      sweep_stats(perm, s, H, h, act, kb, ke, slot, SL, HP, m, d);
      if (pslot >= 0) {
        if (slot == 0 && act) {
          pm[(int64_t)pslot * H + h] = m;
          pd[(int64_t)pslot * H + h] = d;
        }
        continue;
      }
      sweep_write(perm, s, H, h, act, kb, ke, slot, SL, m, 1.0 / d, out, out_csr);
    }
  }
}

// A split row of at most kSplitWaves chunks, by one block: wavefront w takes
// chunk w, finds its pair (from the registers, or a running sweep), leaves it
// in LDS, and after the barrier every wavefront combines the pairs in chunk
// order and writes its chunk's alpha (from the registers when they hold the
// chunk). Every wavefront runs the same head passes and barriers, with or
// without a chunk.
template <int NST>
__device__ __forceinline__ void split_chunk(const int* __restrict__ perm,
                                            const float* __restrict__ s, int H, int HP, int kb,
                                            int ke, int nch, int w, int lane,
                                            float (&lm)[kSplitWaves][kWave],
                                            double (&ld)[kSplitWaves][kWave],
                                            float* __restrict__ out,
                                            float* __restrict__ out_csr) {
  const int SL = kWave / HP;
  const int slot = lane / HP, hh = lane % HP;
  const bool has = kb < ke;
  constexpr int R = NST > 0 ? NST : 1;  // registers (NST = 0: the running sweep)
  int e[R];
  if constexpr (NST > 0) load_ids<NST>(perm, kb, ke, slot, SL, e);
  for (int hb = 0; hb < H; hb += HP) {
    const int h = hb + hh;
    const bool act = h < H;
    float v[R];
    float m = -__builtin_huge_valf();
    double d = 0.0;
    if (has) {
      if constexpr (NST > 0) {
        load_scores<NST>(s, H, h, act, e, v);
        m = regs_max<NST>(v, HP);
        d = regs_exp_sum<NST, false>(v, m, HP);
      } else {
        sweep_stats(perm, s, H, h, act, kb, ke, slot, SL, HP, m, d);
      }
    }
    lm[w][lane] = m;
    ld[w][lane] = d;
    __syncthreads();
    // the row's maximum, then the chunks' sums rescaled to it, in chunk order
    float mr = -__builtin_huge_valf();
    for (int c = 0; c < nch; ++c) mr = lm[c][lane] > mr ? lm[c][lane] : mr;
    double dr = 0.0;
    for (int c = 0; c < nch; ++c) dr += ld[c][lane] * (double)expf(lm[c][lane] - mr);
    __syncthreads();  // the pairs are read before the next head pass writes
    if (!has) continue;
    const double r = 1.0 / dr;
    if constexpr (NST > 0) {
#pragma unroll
      for (int u = 0; u < NST; ++u) v[u] = expf(v[u] - mr);
      regs_write<NST>(v, e, (float)r, kb, slot, SL, H, h, act, out, out_csr);
    } else {
      sweep_write(perm, s, H, h, act, kb, ke, slot, SL, mr, r, out, out_csr);
    }
  }
}

// One block per split row (kSplitWaves wavefronts). A row of at most
// kSplitWaves chunks goes through split_chunk (the register sweep when a
// whole chunk fits, the same choice for every chunk of the launch). A longer
// row: the chunks' pairs come from softmax_items and are combined in chunk
// order the same way, and wavefront w writes chunks w, w + kSplitWaves, ...
__global__ __launch_bounds__(kSplitWaves * kWave) void softmax_split(
    const SplitRow* __restrict__ split, const int* __restrict__ rowptr, int chunk,
    const int* __restrict__ perm, const float* __restrict__ s, int H, int HP,
    const float* __restrict__ pm, const double* __restrict__ pd, float* __restrict__ out,
    float* __restrict__ out_csr) {
  __shared__ float lm[kSplitWaves][kWave];
  __shared__ double ld[kSplitWaves][kWave];
  const SplitRow* sr = split + blockIdx.x;
  const int row = uniform(sr->row), nch = uniform(sr->nchunks), s0 = uniform(sr->slot0);
  const int rb = uniform(rowptr[row]), re = uniform(rowptr[row + 1]);
  const int w = uniform((int)threadIdx.x / kWave);
  const int lane = threadIdx.x & (kWave - 1);
  const int SL = kWave / HP;
  if (nch <= kSplitWaves) {
    const int kb = rb + w * chunk, ke = min(re, kb + chunk);  // kb >= ke: no chunk
    const int cst = (chunk + SL - 1) / SL;  // slot steps of a whole chunk
    if (cst <= 2)
      split_chunk<2>(perm, s, H, HP, kb, ke, nch, w, lane, lm, ld, out, out_csr);
    else if (cst <= 4)
      split_chunk<4>(perm, s, H, HP, kb, ke, nch, w, lane, lm, ld, out, out_csr);
    else if (cst <= kSmCap)
      split_chunk<kSmCap>(perm, s, H, HP, kb, ke, nch, w, lane, lm, ld, out, out_csr);
    else if (cst <= 2 * kSmCap)
      split_chunk<2 * kSmCap>(perm, s, H, HP, kb, ke, nch, w, lane, lm, ld, out, out_csr);
    else
      split_chunk<0>(perm, s, H, HP, kb, ke, nch, w, lane, lm, ld, out, out_csr);
    return;
  }
  const int slot = lane / HP, hh = lane % HP;
  for (int hb = 0; hb < H; hb += HP) {
    const int h = hb + hh;
    const bool act = h < H;
    float m = -__builtin_huge_valf();
    double d = 0.0;
    if (act)
      for (int c = 0; c < nch; ++c)
        stat_merge(m, d, pm[(int64_t)(s0 + c) * H + h], pd[(int64_t)(s0 + c) * H + h]);
    const double r = 1.0 / d;
    for (int c = w; c < nch; c += kSplitWaves) {
      const int kb = rb + c * chunk, ke = min(re, kb + chunk);
      sweep_write(perm, s, H, h, act, kb, ke, slot, SL, m, r, out, out_csr);
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

int launch_gat_graph_scores(const Graph& g, const float* h, int H, int D, const float* a_src,
                            const float* a_dst, float slope, float* out, int by_perm,
                            float* proj, hipStream_t s) {
  float* as = proj;
  float* ad = proj + g.N * H;
  if (g.N * H > 0) {
    projections(h, g.N, H, D, a_src, a_dst, as, ad, s);
    TFG_LAUNCHED("node_projections");
  }
  if (g.E * H > 0) {
    const unsigned nb = (unsigned)((g.E * H + kBlock - 1) / kBlock);
    edge_scores_graph<<<nb, kBlock, 0, s>>>(g.col, g.key, by_perm ? g.perm : nullptr, g.parts, g.E,
                                            H, as, ad, slope, out);
    TFG_LAUNCHED("edge_scores_graph");
  }
  return TFG_OK;
}

size_t row_stats_bytes(int64_t n_chunks, int64_t H) {
  const size_t n = (size_t)std::max<int64_t>(n_chunks * H, 1);
  return align_up(sizeof(float) * n, 256) + align_up(sizeof(double) * n, 256);
}

int launch_segment_softmax(const Graph& g, const float* scores, int H, float* out, float* out_csr,
                           void* ws, hipStream_t s, bool graph_order) {
  if (g.N == 0 || g.E == 0 || H == 0) return TFG_OK;
  // scores and alpha in the graph order: position k is edge k, one output
  const int* perm = graph_order ? nullptr : g.perm;
  if (graph_order) out_csr = nullptr;
  int hp = 1;
  while (hp * 2 <= std::min(H, kWave)) hp *= 2;
  float* pm = static_cast<float*>(ws);
  double* pd = reinterpret_cast<double*>(
      static_cast<char*>(ws) + align_up(sizeof(float) * (size_t)std::max<int64_t>((int64_t)g.n_heavy * H, 1), 256));
  const int64_t short_waves = (g.n_short + kWave / hp - 1) / (kWave / hp);
  const int64_t waves = short_waves + g.n_long + g.n_heavy;
  if (waves > INT32_MAX) return fail(TFG_ERR_TOO_LARGE, "segment softmax: too many work items");
  if (waves > 0) {
    softmax_items<<<(unsigned)((waves + (kItemBlock / kWave) - 1) / (kItemBlock / kWave)), kItemBlock, 0, s>>>(
        g.short_rows, g.n_short, (int)short_waves, g.long_rows, g.n_long, g.heavy, g.n_heavy,
        g.rowptr, g.chunk, perm, scores, H, hp, out, out_csr, pm, pd);
    TFG_LAUNCHED("softmax_items");
  }
  if (g.n_split > 0) {
    softmax_split<<<(unsigned)g.n_split, kSplitWaves * kWave, 0, s>>>(
        g.split, g.rowptr, g.chunk, perm, scores, H, hp, pm, pd, out, out_csr);
    TFG_LAUNCHED("softmax_split");
  }
  return TFG_OK;
}

}  // namespace tfg
