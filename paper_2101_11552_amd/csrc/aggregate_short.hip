// Short rows of the aggregation (gfx950): rows of at most kShortRow edges,
// one per edge slot and SLOTS per wavefront (one weight per edge; per-head
// weights keep the one-row-per-wavefront kernel, which measured faster). The slot's lanes load the row's
// column ids (and edge ids, weights) at once and gather every source row of
// the row together; each lane then reduces its V columns over the edges in
// graph order (sum / mean with one float32 chain, max with the smallest edge
// id winning ties) and applies the epilogue. No cross-lane traffic. On graphs
// of low average degree most rows are short, and one wavefront per row would
// spend most of its time waiting on one or two dependent loads.
#include "spmm.h"

namespace tfg {
namespace rows {
namespace {

template <int V, int SLOTS, bool MAX>
__global__ __launch_bounds__(kItemBlock) void spmm_short(
    const WorkItem* __restrict__ short_rows, int n_short, const int* __restrict__ col,
    const int* __restrict__ perm, const float* __restrict__ w,
    int w_by_perm, const float* __restrict__ x, int64_t ldx, int F, int mean,
    float* __restrict__ out, int* __restrict__ argout, Epilogue ep) {
  constexpr int LPS = kWave / SLOTS;
  constexpr int FC = LPS * V;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  const int64_t i = wave * SLOTS + lane / LPS;
  if (i >= n_short) return;  // nothing crosses lanes: a lane may leave early
  const int sl = lane % LPS;
  const WorkItem it = short_rows[i];
  const int t = it.row, kb = it.kbeg, n = it.kend - it.kbeg;  // 0 <= n <= kShortRow
  const bool need_perm = MAX || w_by_perm;
  int c[kShortRow], e[kShortRow];
  float wr[kShortRow];
#pragma unroll
  for (int j = 0; j < kShortRow; ++j) {
    const bool ok = j < n;
    c[j] = ok ? col[kb + j] : 0;
    e[j] = (ok && need_perm) ? perm[kb + j] : kb + j;
    wr[j] = (w != nullptr && ok) ? w[w_by_perm ? e[j] : kb + j] : 1.0f;
  }
  for (int f0 = 0; f0 < F; f0 += FC) {
    const int f = f0 + sl * V;
    if (f >= F) break;
    float xv[kShortRow][V];
#pragma unroll
    for (int j = 0; j < kShortRow; ++j) {
      if (j < n) {
        load_row<V>(x + (int64_t)c[j] * ldx + f, xv[j]);
      } else {
#pragma unroll
        for (int v = 0; v < V; ++v) xv[j][v] = 0.0f;
      }
    }
    float acc[V];
    int arg[V];
#pragma unroll
    for (int v = 0; v < V; ++v) {
      acc[v] = 0.0f;
      arg[v] = -1;
    }
#pragma unroll
    for (int j = 0; j < kShortRow; ++j)
      if (j < n) {
#pragma unroll
        for (int v = 0; v < V; ++v) {
          if constexpr (MAX) {
            const float m = wr[j] * xv[j][v];
            if (arg[v] < 0 || m > acc[v] || (m == acc[v] && e[j] < arg[v])) {
              acc[v] = m;
              arg[v] = e[j];
            }
          } else {
            acc[v] = __builtin_fmaf(wr[j], xv[j][v], acc[v]);
          }
        }
      }
    if constexpr (MAX) {
#pragma unroll
      for (int v = 0; v < V; ++v)
        if (arg[v] < 0) acc[v] = 0.0f;
    } else {
      if (mean && n > 0) {
        const float cnt = (float)n;
#pragma unroll
        for (int v = 0; v < V; ++v) acc[v] = acc[v] / cnt;
      }
      apply_epilogue<V>(ep, t, f, acc);
    }
    store_row<V>(out + (int64_t)t * F + f, acc);
    if (MAX && argout != nullptr)
#pragma unroll
      for (int v = 0; v < V; ++v) argout[(int64_t)t * F + f + v] = arg[v];
  }
}

template <int V, int SLOTS, bool MAX>
void run(const Graph& g, const RowArgs& a, hipStream_t s) {
  const int64_t waves = (g.n_short + SLOTS - 1) / SLOTS;
  const dim3 grid((unsigned)((waves + kItemBlock / kWave - 1) / (kItemBlock / kWave)));
  spmm_short<V, SLOTS, MAX><<<grid, kItemBlock, 0, s>>>(g.short_rows, g.n_short, a.col,
                                                    a.perm, a.w, a.w_by_perm, a.x, a.ldx, a.F,
                                                    a.mean, a.out, a.argout, a.ep);
}

template <int V, bool MAX>
void by_slots(int slots, const Graph& g, const RowArgs& a, hipStream_t s) {
  switch (slots) {
    case 1: run<V, 1, MAX>(g, a, s); break;
    case 2: run<V, 2, MAX>(g, a, s); break;
    case 4: run<V, 4, MAX>(g, a, s); break;
    case 8: run<V, 8, MAX>(g, a, s); break;
    default: run<V, 16, MAX>(g, a, s); break;
  }
}

template <bool MAX>
void by_vec(int vec, int slots, const Graph& g, const RowArgs& a, hipStream_t s) {
  if (vec == 4)
    by_slots<4, MAX>(slots, g, a, s);
  else if (vec == 2)
    by_slots<2, MAX>(slots, g, a, s);
  else
    by_slots<1, MAX>(slots, g, a, s);
}

}  // namespace

void dispatch_short(bool mx, int vec, int slots, const Graph& g, const RowArgs& a,
                    hipStream_t s) {
  if (mx)
    by_vec<true>(vec, slots, g, a, s);
  else
    by_vec<false>(vec, slots, g, a, s);
}

}  // namespace rows
}  // namespace tfg
