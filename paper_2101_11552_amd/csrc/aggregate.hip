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

// Sum and mean with scalar edge ids: one wavefront per work item, SL edge
// slots of 64 / SL lanes (SL = 1 or 2), lane l of a slot holding columns
// V l .. V l + V - 1 of a 64 V / SL-column pass. The item's edge ids and
// weights come in with one coalesced load per 64 edges and are read out edge
// by edge into scalar registers (readlane); the scalar unit forms each row's
// 32-bit byte offset (NARROW: the table below 4 GB; else 64-bit per lane), so
// a lane adds its own offset and selects between the slots' values, and the
// load takes the table's base from scalar registers. Edges go in groups of U
// per slot, every load of a group issued before its first multiply-add; the
// last group repeats the item's last edge in its unused places (a row already
// loaded) and adds only the item's own edges. One accumulator chain per
// group place, combined pairwise, then across the slots.
template <int SL>
__device__ __forceinline__ int pick(int a, int b, int slot) {
  if constexpr (SL == 1) return a;
  else return slot ? b : a;
}

template <int V, int SL, int U, bool FULL, bool NARROW>
__device__ __forceinline__ void wide_pass(int kbeg, int kend, const int* __restrict__ col,
                                          const int* __restrict__ perm,
                                          const float* __restrict__ w, int w_by_perm,
                                          const char* __restrict__ xb, int64_t row_bytes,
                                          unsigned lane_off, int slot, bool fok,
                                          float (&acc)[U][V]) {
  const int lane = lane_id();
  for (int kb = kbeg; kb < kend; kb += kWave) {
    const int n = min(kWave, kend - kb);
    const bool lok = lane < n;
    const int cj = lok ? __builtin_nontemporal_load(col + kb + lane) : 0;
    float wf = 1.0f;
    if (w != nullptr && lok)  // weights in graph order, or in the caller's edge order
      wf = w_by_perm ? w[__builtin_nontemporal_load(perm + kb + lane)]
                     : __builtin_nontemporal_load(w + kb + lane);
    const int wj = __float_as_int(wf);
    auto group = [&](int j0, bool tail) {
      float xv[U][V];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ja = j0 + u * SL;
        const int ca = __builtin_amdgcn_readlane(cj, tail ? min(ja, n - 1) : ja);
        const int cb = SL > 1 ? __builtin_amdgcn_readlane(cj, tail ? min(ja + 1, n - 1) : ja + 1) : 0;
        if (FULL || fok) {
          if constexpr (NARROW) {
            const unsigned off =
                (unsigned)pick<SL>(ca * (int)row_bytes, cb * (int)row_bytes, slot) + lane_off;
            load_row<V>(reinterpret_cast<const float*>(xb + off), xv[u]);
          } else {
            const int64_t off = (int64_t)pick<SL>(ca, cb, slot) * row_bytes + lane_off;
            load_row<V>(reinterpret_cast<const float*>(xb + off), xv[u]);
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ja = j0 + u * SL;
        if (tail && ja >= n) continue;  // uniform
        const int wa = __builtin_amdgcn_readlane(wj, ja);
        const int wb = SL > 1 ? __builtin_amdgcn_readlane(wj, tail ? min(ja + 1, n - 1) : ja + 1) : 0;
        const float wt = __int_as_float(pick<SL>(wa, wb, slot));
        if ((FULL || fok) && (!tail || ja + slot < n))
#pragma unroll
          for (int v = 0; v < V; ++v) acc[u][v] = __builtin_fmaf(wt, xv[u][v], acc[u][v]);
      }
    };
    int j0 = 0;
    for (; j0 + U * SL <= n; j0 += U * SL) group(j0, false);
    if (j0 < n) group(j0, true);
  }
}

template <int V, int SL, int U, bool NARROW>
__global__ __launch_bounds__(kRowBlock) void spmm_wide(
    const WorkItem* __restrict__ heavy, int n_heavy, const WorkItem* __restrict__ light,
    int n_light, const int* __restrict__ col, const int* __restrict__ perm,
    const float* __restrict__ w, int w_by_perm, const float* __restrict__ x, int64_t ldx, int F,
    int mean, float* __restrict__ out, float* __restrict__ part, Epilogue ep) {
  constexpr int LPS = kWave / SL;  // lanes per slot
  constexpr int FC = LPS * V;      // columns per pass
  const int wid = uniform(blockIdx.x * (kRowBlock / kWave) + threadIdx.x / kWave);
  if (wid >= n_heavy + n_light) return;
  const int lane = lane_id();
  const int slot = lane / LPS, sl = lane % LPS;
  const WorkItem* itp = wid < n_heavy ? heavy + wid : light + (wid - n_heavy);
  const int row = uniform(itp->row), kbeg = uniform(itp->kbeg), kend = uniform(itp->kend);
  const int pslot = uniform(itp->slot);
  const char* xc = reinterpret_cast<const char*>(x);
  const int64_t row_bytes = ldx * (int64_t)sizeof(float);
  for (int f0 = 0; f0 < F; f0 += FC) {
    const int f = f0 + sl * V;
    const bool fok = f < F;
    float acc[U][V];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int v = 0; v < V; ++v) acc[u][v] = 0.0f;
    // the pass's column offset in scalar registers, the lane's in a 32-bit offset
    const char* xb = xc + (int64_t)f0 * (int64_t)sizeof(float);
    const unsigned lane_off = (unsigned)(sl * V) * (unsigned)sizeof(float);
    if (f0 + FC <= F)
      wide_pass<V, SL, U, true, NARROW>(kbeg, kend, col, perm, w, w_by_perm, xb, row_bytes,
                                        lane_off, slot, fok, acc);
    else
      wide_pass<V, SL, U, false, NARROW>(kbeg, kend, col, perm, w, w_by_perm, xb, row_bytes,
                                         lane_off, slot, fok, acc);
#pragma unroll
    for (int step = 1; step < U; step <<= 1)
#pragma unroll
      for (int u = 0; u + step < U; u += 2 * step)
#pragma unroll
        for (int v = 0; v < V; ++v) acc[u][v] += acc[u + step][v];
#pragma unroll
    for (int off = LPS; off < kWave; off <<= 1)
#pragma unroll
      for (int v = 0; v < V; ++v) acc[0][v] += __shfl_xor(acc[0][v], off);
    if (slot != 0 || !fok) continue;
    if (pslot < 0) {
      if (mean && kend > kbeg) {
        const float cnt = (float)(kend - kbeg);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[0][v] = acc[0][v] / cnt;
      }
      apply_epilogue<V>(ep, row, f, acc[0]);
      store_row<V>(out + (int64_t)row * F + f, acc[0]);
    } else {
      // partial rows are read back once, by the fix-up, long after: streamed
      // past the L2, which they would otherwise share with the gathered rows
      store_row<V>(part + (int64_t)pslot * F + f, acc[0]);
    }
  }
}

// Whether the sum / mean goes through spmm_wide: rows of at least 64
// columns (every lane busy), one weight per edge; the layout: two slots of
// four columns per lane where 128 columns fit the alignment, else one slot of
// two or one. TFG_WIDE_ROWS=0 keeps every aggregation on spmm_rows.
struct WideShape {
  int v, slots;
};
WideShape wide_shape(int64_t F, int vec, bool sum_like, bool heads, bool masked) {
  if (!sum_like || heads || masked || F < kWave) return {0, 0};
  if (const char* v = std::getenv("TFG_WIDE_ROWS"))
    if (v[0] == '0') return {0, 0};
  if (vec == 4 && F % 128 == 0) return {4, 2};
  return {vec % 2 == 0 && F >= 2 * kWave ? 2 : 1, 1};
}

void launch_wide(WideShape ws, dim3 grid, hipStream_t s, const RowArgs& a, int64_t n_src) {
  // the whole table within 32-bit byte offsets of its base
  const bool narrow = (double)n_src * (double)a.ldx * 4.0 < 2147483648.0;
#define TFG_WIDE(VV, SS, UU, NN)                                                       \
  spmm_wide<VV, SS, UU, NN><<<grid, dim3(kRowBlock), 0, s>>>(                          \
      a.heavy, a.n_heavy, a.light, a.n_light, a.col, a.perm, a.w, a.w_by_perm, a.x, a.ldx, \
      a.F, a.mean, a.out, a.part, a.ep)
  if (ws.slots == 2) {  // U = 4 (the power-law aggregation: 3.51 ms; U = 8: 3.69, U = 2: 3.51)
    if (narrow) TFG_WIDE(4, 2, 4, true); else TFG_WIDE(4, 2, 4, false);
  } else if (ws.v == 2) {
    if (narrow) TFG_WIDE(2, 1, 8, true); else TFG_WIDE(2, 1, 8, false);
  } else {
    if (narrow) TFG_WIDE(1, 1, 8, true); else TFG_WIDE(1, 1, 8, false);
  }
#undef TFG_WIDE
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
    const WideShape wsh = wide_shape(F, vec, !mx, heads, mask != nullptr);
    if (wsh.v > 0)
      launch_wide(wsh, grid, s, a, g.N_src);
    else if (mask != nullptr)
      dispatch_masked(part_plan, heads, vec, slots, grid, s, a);
    else if (part_plan)
      dispatch_kind<true>(mx, heads, vec, slots, grid, s, a);
    else
      dispatch_kind<false>(mx, heads, vec, slots, grid, s, a);
    TFG_LAUNCHED("spmm_rows");
  }
  if (n_rows > 0) {
    dim3 fgrid((unsigned)((n_rows + kItemBlock / kWave - 1) / (kItemBlock / kWave)));
    // partials are dense [slot, F] rows: 16-byte accesses when F is a multiple
    // of 4 and the output (and the epilogue's h rows) allow them
    const bool f4 = F % 4 == 0 && reinterpret_cast<uintptr_t>(out) % 16 == 0 &&
                    (h == nullptr || (ldh % 4 == 0 && reinterpret_cast<uintptr_t>(h) % 16 == 0));
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
