// Message aggregation over the CSR-by-target graph (gfx950, wave64):
// out[t, :] = reduce over the edges k of row t of w_k * x[col_k, :].
// The row kernel (spmm_rows, spmm.h) runs over the work items of the graph's
// plan; long rows and source-part segments leave partial rows that
// fixup_rows combines in a fixed order. No floating-point atomics: every
// output is reproducible bit for bit.
#include <cstdlib>
#include <mutex>

#include "spmm.h"

namespace tfg {
namespace {

// Device memory of the no-allocation aggregation (tfg_aggregate_noalloc): the
// partial rows that tfg_aggregate keeps in its workspace. Every GPU the
// library runs on holds its own copy until the process ends. In host code the
// name only stands for the symbol: kernels get the device address that
// hipGetSymbolAddress returns for the current device.
__device__ __align__(256) unsigned char scratch[TFG_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

using namespace rows;

// Combines the partial results of each split row in chunk order: sums with
// kFixAcc interleaved accumulators combined pairwise, maxima with the tie rule.
constexpr int kFixAcc = 8;
// Lanes cover V consecutive features each.
template <bool MAX, int V>
__global__ __launch_bounds__(kItemBlock) void fixup_rows(const SplitRow* __restrict__ split,
                                                     int n_split, const float* __restrict__ part,
                                                     const int* __restrict__ part_arg, int F,
                                                     int mean, float* __restrict__ out,
                                                     int* __restrict__ argout, Epilogue ep) {
  const int wid = uniform(blockIdx.x * (kItemBlock / kWave) + threadIdx.x / kWave);
  if (wid >= n_split) return;
  const int lane = threadIdx.x & (kWave - 1);
  const SplitRow* sr = split + wid;
  const int row = uniform(sr->row), slot0 = uniform(sr->slot0), nch = uniform(sr->nchunks);
  const int deg = uniform(sr->deg);
  for (int f = lane * V; f < F; f += kWave * V) {
    if constexpr (MAX) {
#pragma unroll
      for (int v = 0; v < V; ++v) {
        float best = 0.0f;
        int a = -1;
        for (int j = 0; j < nch; ++j)
          max_combine(best, a, part[(int64_t)(slot0 + j) * F + f + v],
                      part_arg[(int64_t)(slot0 + j) * F + f + v]);
        out[(int64_t)row * F + f + v] = a < 0 ? 0.0f : best;
        if (argout != nullptr) argout[(int64_t)row * F + f + v] = a;
      }
    } else {
      // kFixAcc partial rows in flight, one accumulator each
      float a4[kFixAcc][V];
#pragma unroll
      for (int i = 0; i < kFixAcc; ++i)
#pragma unroll
        for (int v = 0; v < V; ++v) a4[i][v] = 0.0f;
      for (int j = 0; j < nch; j += kFixAcc) {
        float t[kFixAcc][V];
#pragma unroll
        for (int i = 0; i < kFixAcc; ++i) {
          if (j + i < nch) {
            load_row_once<V>(part + (int64_t)(slot0 + j + i) * F + f, t[i]);
          } else {
#pragma unroll
            for (int v = 0; v < V; ++v) t[i][v] = 0.0f;
          }
        }
#pragma unroll
        for (int i = 0; i < kFixAcc; ++i)
#pragma unroll
          for (int v = 0; v < V; ++v) a4[i][v] += t[i][v];
      }
#pragma unroll
      for (int step = 1; step < kFixAcc; step <<= 1)
#pragma unroll
        for (int i = 0; i + step < kFixAcc; i += 2 * step)
#pragma unroll
          for (int v = 0; v < V; ++v) a4[i][v] += a4[i + step][v];
      float s[V];
#pragma unroll
      for (int v = 0; v < V; ++v) {
        s[v] = a4[0][v];
        if (mean && deg > 0) s[v] = s[v] / (float)deg;
      }
      apply_epilogue<V>(ep, row, f, s);
      store_row<V>(out + (int64_t)row * F + f, s);
    }
  }
}

template <bool SHORT>
void dispatch_kind(bool mx, bool heads, int vec, int slots, dim3 grid, hipStream_t s,
                   const RowArgs& a) {
  if (mx && heads)
    dispatch_vec<true, true, SHORT, false>(vec, slots, grid, s, a);
  else if (mx)
    dispatch_vec<true, false, SHORT, false>(vec, slots, grid, s, a);
  else if (heads)
    dispatch_vec<false, true, SHORT, false>(vec, slots, grid, s, a);
  else
    dispatch_vec<false, false, SHORT, false>(vec, slots, grid, s, a);
}

}  // namespace

int noalloc_scratch(void** ptr) {
  int dev = 0;
  TFG_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(TFG_ERR_INVALID_ARG, "device id out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_addr[dev] == nullptr) {
    void* p = nullptr;
    TFG_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (p == nullptr) return fail(TFG_ERR_HIP, "no device address for the static scratch");
    g_scratch_addr[dev] = p;
  }
  *ptr = g_scratch_addr[dev];
  return TFG_OK;
}

size_t aggregate_partial_bytes(int64_t n_partials, int64_t F, int reduce) {
  size_t per = sizeof(float) + (reduce == TFG_MAX ? sizeof(int) : 0);
  return align_up((size_t)std::max<int64_t>(n_partials, 1) * (size_t)F * per + 256, 256);
}

bool use_part_plan(const Graph& g, int64_t F) {
  if (g.parts <= 1 || g.n_pexec == 0) return false;
  const char* v = std::getenv("TFG_PART_PLAN");  // "0": never, "1": always, unset: by size
  if (v && v[0] == '0') return false;
  if (v && v[0] == '1') return true;
  // the gathered table must be much larger than the L2 caches (8 x 4 MB)
  return (double)g.N_src * (double)F * 4.0 >= 32.0 * (1 << 20);
}

int launch_aggregate(const Graph& g, const float* w, int H, int w_order, const float* x,
                     int64_t F, int64_t ldx, int reduce, float* out, int32_t* argmax, void* ws,
                     hipStream_t s, float scale, float alpha, const float* h, int64_t ldh,
                     const int32_t* mask) {
  if (g.N == 0 || F == 0) return TFG_OK;
  if (mask != nullptr && reduce != TFG_SUM) return fail(TFG_ERR_INVALID_ARG, "masked max");
  const bool heads = H > 1 && w != nullptr;
  const int per_head = (int)(F / H);
  // every row of x, out (and h, mask) is read or written with v-wide accesses
  auto fits = [&](int v) {
    return F % v == 0 && ldx % v == 0 && reinterpret_cast<uintptr_t>(x) % (4 * v) == 0 &&
           reinterpret_cast<uintptr_t>(out) % (4 * v) == 0 && (!heads || per_head % v == 0) &&
           (h == nullptr || (ldh % v == 0 && reinterpret_cast<uintptr_t>(h) % (4 * v) == 0)) &&
           (mask == nullptr || reinterpret_cast<uintptr_t>(mask) % (4 * v) == 0);
  };
  const int vec = fits(4) ? 4 : fits(2) ? 2 : 1;
  const int lanes = (int)std::min<int64_t>((F + vec - 1) / vec, kWave);
  int p2 = 1;
  while (p2 < lanes) p2 <<= 1;
  const int slots = std::min(kWave / p2, 16);
  const bool mx = reduce == TFG_MAX;
  const bool part_plan = use_part_plan(g, F);
  const bool short_rows = !part_plan && mask == nullptr && !heads && g.n_short > 0;

  RowArgs a;
  a.col = g.col;
  a.perm = g.perm;
  a.w = w;
  a.w_by_perm = (w != nullptr && w_order == TFG_COO) ? 1 : 0;
  a.H = H;
  a.per_head = per_head;
  a.x = x;
  a.ldx = ldx;
  a.mask = mask;
  a.F = (int)F;
  a.mean = reduce == TFG_MEAN;
  a.out = out;
  a.argout = argmax;
  a.ep = Epilogue{scale, alpha, h, ldh};
  const int n_partials = part_plan ? g.n_pexec : g.n_heavy;
  a.part = static_cast<float*>(ws);
  a.part_arg = reinterpret_cast<int*>(a.part + (size_t)std::max(n_partials, 1) * F);
  const SplitRow* rows;
  int n_rows;
  if (part_plan) {
    // every (part, row) item writes a partial; each row is reduced in part order
    a.heavy = g.pexec;
    a.n_heavy = g.n_pexec;
    a.light = nullptr;
    a.n_light = 0;
    rows = g.prows;
    n_rows = (int)g.N;
  } else {
    a.heavy = g.heavy;
    a.n_heavy = g.n_heavy;
    rows = g.split;
    n_rows = g.n_split;
    if (short_rows) {
      // rows of at most kShortRow edges several per wavefront, the rest one each
      a.light = g.long_rows;
      a.n_light = g.n_long;
    } else {
      a.light = g.light;
      a.n_light = g.n_light;
    }
  }
  if (short_rows) {
    dispatch_short(mx, vec, slots, g, a, s);
    TFG_LAUNCHED("spmm_short");
  }
  const int waves = a.n_heavy + a.n_light;
  if (waves > 0) {
    dim3 grid((unsigned)((waves + kRowBlock / kWave - 1) / (kRowBlock / kWave)));
    if (mask != nullptr)
      dispatch_masked(part_plan, heads, vec, slots, grid, s, a);
    else if (part_plan)
      dispatch_kind<true>(mx, heads, vec, slots, grid, s, a);
    else
      dispatch_kind<false>(mx, heads, vec, slots, grid, s, a);
    TFG_LAUNCHED("spmm_rows");
  }
  if (n_rows > 0) {
    dim3 fgrid((unsigned)((n_rows + kItemBlock / kWave - 1) / (kItemBlock / kWave)));
    // partials are dense [slot, F] rows: 16-byte accesses when F is a multiple of 4
    const bool f4 = F % 4 == 0 && reinterpret_cast<uintptr_t>(out) % 16 == 0;
    if (mx)
      fixup_rows<true, 1><<<fgrid, dim3(kItemBlock), 0, s>>>(rows, n_rows, a.part, a.part_arg, a.F,
                                                         a.mean, out, argmax, a.ep);
    else if (f4)
      fixup_rows<false, 4><<<fgrid, dim3(kItemBlock), 0, s>>>(rows, n_rows, a.part, a.part_arg, a.F,
                                                          a.mean, out, argmax, a.ep);
    else
      fixup_rows<false, 1><<<fgrid, dim3(kItemBlock), 0, s>>>(rows, n_rows, a.part, a.part_arg, a.F,
                                                          a.mean, out, argmax, a.ep);
    TFG_LAUNCHED("fixup_rows");
  }
  return TFG_OK;
}

}  // namespace tfg
