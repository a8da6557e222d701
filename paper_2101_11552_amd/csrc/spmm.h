// The row kernel of the message aggregation (gfx950, wave64), shared by the
// forward aggregation (aggregate.hip) and the masked gather of the max
// gradient (backward.hip), which instantiate it in separate translation units.
//
// out[t, :] = reduce over the edges k of row t of w_k * x[col_k, :].
//
// One wavefront processes one work item (a whole row, or a chunk of at most
// `chunk` edges of a long row). The 64 lanes are split into SLOTS edge slots of
// 64/SLOTS lanes; each slot gathers one source row per step with V-wide vector
// loads, so a wave has SLOTS * U row gathers in flight (U independent
// accumulators per lane). Edge indices and weights are read once per 64 edges
// with coalesced loads and broadcast from registers. Partial chains are short
// (row length / (SLOTS * U)) and are combined pairwise, so the float32 error
// stays small for long rows too; long rows are cut into chunks whose partial
// results a fix-up pass combines in chunk order. No floating-point atomics:
// every output is reproducible bit for bit.
#pragma once

#include "wave.h"

namespace tfg {
namespace rows {

typedef float f2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef int i2 __attribute__((ext_vector_type(2)));
typedef int i4 __attribute__((ext_vector_type(4)));

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

// The same, for data read once (streamed past the L2).
template <int V>
__device__ __forceinline__ void load_row_once(const float* __restrict__ p, float (&v)[V]) {
  if constexpr (V == 4) {
    f4 t = __builtin_nontemporal_load(reinterpret_cast<const f4*>(p));
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else if constexpr (V == 2) {
    f2 t = __builtin_nontemporal_load(reinterpret_cast<const f2*>(p));
    v[0] = t.x; v[1] = t.y;
  } else {
    v[0] = __builtin_nontemporal_load(p);
  }
}

template <int V>
__device__ __forceinline__ void load_irow(const int* __restrict__ p, int (&v)[V]) {
  if constexpr (V == 4) {
    i4 t = *reinterpret_cast<const i4*>(p);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else if constexpr (V == 2) {
    i2 t = *reinterpret_cast<const i2*>(p);
    v[0] = t.x; v[1] = t.y;
  } else {
    v[0] = *p;
  }
}

template <int V>
__device__ __forceinline__ void store_row(float* __restrict__ p, const float (&v)[V]) {
  if constexpr (V == 4) {
    f4 t = {v[0], v[1], v[2], v[3]};
    __builtin_nontemporal_store(t, reinterpret_cast<f4*>(p));
  } else if constexpr (V == 2) {
    f2 t = {v[0], v[1]};
    __builtin_nontemporal_store(t, reinterpret_cast<f2*>(p));
  } else {
    __builtin_nontemporal_store(v[0], p);
  }
}

// Value held by lane (jbase + slot); jbase is wave-uniform.
template <int SLOTS>
__device__ __forceinline__ int bcast(int v, int jbase, int slot) {
  if constexpr (SLOTS == 1) {
    return __builtin_amdgcn_readlane(v, jbase);
  } else if constexpr (SLOTS == 2) {
    int a = __builtin_amdgcn_readlane(v, jbase);
    int b = __builtin_amdgcn_readlane(v, jbase + 1);
    return slot ? b : a;
  } else if constexpr (SLOTS == 4) {
    int a = __builtin_amdgcn_readlane(v, jbase);
    int b = __builtin_amdgcn_readlane(v, jbase + 1);
    int c = __builtin_amdgcn_readlane(v, jbase + 2);
    int d = __builtin_amdgcn_readlane(v, jbase + 3);
    return slot == 0 ? a : slot == 1 ? b : slot == 2 ? c : d;
  } else {
    return __shfl(v, jbase + slot);
  }
}
template <int SLOTS>
__device__ __forceinline__ float bcastf(float v, int jbase, int slot) {
  return __int_as_float(bcast<SLOTS>(__float_as_int(v), jbase, slot));
}

// Output transform of a propagation step: y = scale * sum + alpha * h[row]
// (APPNP, SGC); the identity (scale 1, no h) for a plain aggregation.
struct Epilogue {
  float scale, alpha;
  const float* h;
  int64_t ldh;
};

template <int V>
__device__ __forceinline__ void apply_epilogue(const Epilogue& ep, int row, int f, float (&v)[V]) {
  if (ep.h != nullptr) {
    float t[V];
    load_row<V>(ep.h + (int64_t)row * ep.ldh + f, t);
#pragma unroll
    for (int i = 0; i < V; ++i) v[i] = ep.scale * v[i] + ep.alpha * t[i];
  } else if (ep.scale != 1.0f) {
#pragma unroll
    for (int i = 0; i < V; ++i) v[i] = ep.scale * v[i];
  }
}

// Max with the smallest edge id winning ties; arg < 0 marks "no edge yet".
__device__ __forceinline__ void max_combine(float& v, int& a, float vb, int ab) {
  bool take = ab >= 0 && (a < 0 || vb > v || (vb == v && ab < a));
  v = take ? vb : v;
  a = take ? ab : a;
}

// Independent row gathers in flight per edge slot: 8 for whole rows, 4 for
// the short (row, source part) segments of the part plan.
template <int SLOTS, bool SHORT>
constexpr int unroll_for() {
  constexpr int u = SLOTS * 8 <= kWave ? 8 : kWave / SLOTS;
  return SHORT && u > 4 ? 4 : u;
}

// Threads per block of the row kernel: one wavefront. Its wavefronts are
// independent, and single-wavefront blocks let a CU start the next item as
// soon as any wavefront ends (aggregation on the power-law graph: 3.60 ms,
// against 3.65 / 3.71 / 4.10 / 4.98 ms with 128- to 1024-thread blocks).
constexpr int kRowBlock = kItemBlock;

// MASK (sum only): element c of the gathered row x[col_k] counts only where
// mask[col_k, c] equals the edge id perm[k] (the gradient of a max
// aggregation, gathered over the transposed graph).

template <int V, int SLOTS, bool MAX, bool HEADS, bool SHORT, bool MASK>
__global__ __launch_bounds__(kRowBlock) void spmm_rows(
    const WorkItem* __restrict__ heavy, int n_heavy, const WorkItem* __restrict__ light,
    int n_light, const int* __restrict__ col, const int* __restrict__ perm,
    const float* __restrict__ w, int w_by_perm, int H, int per_head, const float* __restrict__ x,
    int64_t ldx, const int* __restrict__ mask, int F, int mean, float* __restrict__ out,
    int* __restrict__ argout, float* __restrict__ part, int* __restrict__ part_arg, Epilogue ep) {
  static_assert(!(MASK && MAX), "a masked gather is a sum");
  constexpr int LPS = kWave / SLOTS;  // lanes per edge slot
  constexpr int FC = LPS * V;         // feature columns per pass
  constexpr int U = unroll_for<SLOTS, SHORT>();
  const int wid = uniform(blockIdx.x * (kRowBlock / kWave) + threadIdx.x / kWave);
  if (wid >= n_heavy + n_light) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int slot = lane / LPS, sl = lane % LPS;
  const WorkItem* itp = wid < n_heavy ? heavy + wid : light + (wid - n_heavy);
  const int row = uniform(itp->row), kbeg = uniform(itp->kbeg), kend = uniform(itp->kend);
  const int pslot = uniform(itp->slot);
  const bool need_perm = MAX || MASK || w_by_perm;

  for (int f0 = 0; f0 < F; f0 += FC) {
    const int f = f0 + sl * V;
    const bool fok = f < F;
    const float* __restrict__ xf = x + (fok ? f : 0);
    const int head = HEADS ? (fok ? f / per_head : 0) : 0;
    float acc[U][V];
    int arg[U][V];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int v = 0; v < V; ++v) {
        acc[u][v] = 0.0f;
        arg[u][v] = -1;
      }

    for (int kb = kbeg; kb < kend; kb += kWave) {
      const int n = min(kWave, kend - kb);
      const bool lok = lane < n;
      const int cj = lok ? __builtin_nontemporal_load(col + kb + lane) : 0;
      const int pj = (lok && need_perm) ? __builtin_nontemporal_load(perm + kb + lane) : 0;
      float wj = 1.0f;
      if (!HEADS && w != nullptr && lok)
        wj = __builtin_nontemporal_load(w + (w_by_perm ? pj : kb + lane));
      for (int s0 = 0; s0 < n; s0 += SLOTS * U) {
        float xv[U][V];
        float wv[U];
        int ev[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int jb = s0 + u * SLOTS;
          ok[u] = jb + slot < n;
          // cross-lane reads run with the whole wave active (a bpermute from an
          // inactive lane does not return that lane's value)
          const int c = bcast<SLOTS>(cj, jb, slot);
          const int pe = need_perm ? bcast<SLOTS>(pj, jb, slot) : 0;
          if constexpr (HEADS) {
            wv[u] = 1.0f;
            const int e = w_by_perm ? pe : kb + jb + slot;
            if (w != nullptr && ok[u]) wv[u] = w[(int64_t)e * H + head];
          } else {
            wv[u] = bcastf<SLOTS>(wj, jb, slot);
          }
          if constexpr (MAX) ev[u] = pe;
          if (ok[u] && fok) {
            load_row<V>(xf + (int64_t)c * ldx, xv[u]);
            if constexpr (MASK) {
              int mv[V];
              load_irow<V>(mask + (int64_t)c * F + f, mv);
#pragma unroll
              for (int v = 0; v < V; ++v) xv[u][v] = mv[v] == pe ? xv[u][v] : 0.0f;
            }
          } else {
#pragma unroll
            for (int v = 0; v < V; ++v) xv[u][v] = 0.0f;
          }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (ok[u]) {
#pragma unroll
            for (int v = 0; v < V; ++v) {
              if constexpr (MAX) {
                // edge ids need not increase along a row (rows may be grouped
                // by source range), so ties compare the ids
                const float m = wv[u] * xv[u][v];
                if (arg[u][v] < 0 || m > acc[u][v] || (m == acc[u][v] && ev[u] < arg[u][v])) {
                  acc[u][v] = m;
                  arg[u][v] = ev[u];
                }
              } else {
                acc[u][v] = __builtin_fmaf(wv[u], xv[u][v], acc[u][v]);
              }
            }
          }
        }
      }
    }

    // Pairwise combination of the U accumulators, then across the slots.
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
      if (pslot < 0) {
        if (!MAX && mean && kend > kbeg) {
          const float cnt = (float)(kend - kbeg);
#pragma unroll
          for (int v = 0; v < V; ++v) acc[0][v] = acc[0][v] / cnt;
        }
        if (MAX) {
#pragma unroll
          for (int v = 0; v < V; ++v)
            if (arg[0][v] < 0) acc[0][v] = 0.0f;
        }
        if (!MAX) apply_epilogue<V>(ep, row, f, acc[0]);
        store_row<V>(out + (int64_t)row * F + f, acc[0]);
        if (MAX && argout != nullptr)
#pragma unroll
          for (int v = 0; v < V; ++v) argout[(int64_t)row * F + f + v] = arg[0][v];
      } else {
        // partial rows are read back once, by the fix-up, long after: streamed
        // past the L2, which they would otherwise share with the gathered rows
        store_row<V>(part + (int64_t)pslot * F + f, acc[0]);
        if (MAX)
#pragma unroll
          for (int v = 0; v < V; ++v) part_arg[(int64_t)pslot * F + f + v] = arg[0][v];
      }
    }
  }
}

// The kernel arguments shared by every instantiation.
struct RowArgs {
  const WorkItem* heavy;
  int n_heavy;
  const WorkItem* light;
  int n_light;
  const int* col;
  const int* perm;
  const float* w;
  int w_by_perm, H, per_head;
  const float* x;
  int64_t ldx;
  const int* mask;
  int F, mean;
  float* out;
  int* argout;
  float* part;
  int* part_arg;
  Epilogue ep;
};

template <int V, int SLOTS, bool MAX, bool HEADS, bool SHORT, bool MASK>
void launch_rows(dim3 grid, hipStream_t s, const RowArgs& a) {
  spmm_rows<V, SLOTS, MAX, HEADS, SHORT, MASK><<<grid, dim3(kRowBlock), 0, s>>>(
      a.heavy, a.n_heavy, a.light, a.n_light, a.col, a.perm, a.w, a.w_by_perm, a.H, a.per_head,
      a.x, a.ldx, a.mask, a.F, a.mean, a.out, a.argout, a.part, a.part_arg, a.ep);
}

template <int V, bool MAX, bool HEADS, bool SHORT, bool MASK>
void dispatch_slots(int slots, dim3 grid, hipStream_t s, const RowArgs& a) {
  switch (slots) {
    case 1: launch_rows<V, 1, MAX, HEADS, SHORT, MASK>(grid, s, a); break;
    case 2: launch_rows<V, 2, MAX, HEADS, SHORT, MASK>(grid, s, a); break;
    case 4: launch_rows<V, 4, MAX, HEADS, SHORT, MASK>(grid, s, a); break;
    case 8: launch_rows<V, 8, MAX, HEADS, SHORT, MASK>(grid, s, a); break;
    default: launch_rows<V, 16, MAX, HEADS, SHORT, MASK>(grid, s, a); break;
  }
}

template <bool MAX, bool HEADS, bool SHORT, bool MASK>
void dispatch_vec(int vec, int slots, dim3 grid, hipStream_t s, const RowArgs& a) {
  if (vec == 4)
    dispatch_slots<4, MAX, HEADS, SHORT, MASK>(slots, grid, s, a);
  else if (vec == 2)
    dispatch_slots<2, MAX, HEADS, SHORT, MASK>(slots, grid, s, a);
  else
    dispatch_slots<1, MAX, HEADS, SHORT, MASK>(slots, grid, s, a);
}

// Short rows of the row plan, one per edge slot (aggregate_short.hip).
void dispatch_short(bool mx, int vec, int slots, const Graph& g, const RowArgs& a,
                    hipStream_t s);

// Masked sum gathers (backward.hip).
void dispatch_masked(bool part_plan, bool heads, int vec, int slots, dim3 grid, hipStream_t s,
                     const RowArgs& a);

}  // namespace rows
}  // namespace tfg
