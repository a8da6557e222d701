// COO -> CSR by target on the GPU (gfx950): validation + target histogram,
// exclusive scans, a stable LSD radix sort of the edge ids by target, and the
// aggregation work list. The result is the unique stable permutation (edges
// sorted by target, input order kept among equal targets), so it is
// bit-identical to a sequential counting sort.
#include <algorithm>
#include <cstdlib>

#include "tfg_internal.h"

namespace tfg {
namespace {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;  // 2048

constexpr int kSortThreads = 512;                // 8 waves
constexpr int kSortItems = 8;                    // items per thread
constexpr int kSortTile = kSortThreads * kSortItems;  // 4096 edges per block
constexpr int kSortWaves = kSortThreads / kWave;
constexpr int kMaxDigitBits = 9;
constexpr int kMaxRadix = 1 << kMaxDigitBits;    // 512 = kSortThreads

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    int t = __shfl_up(v, off);
    if (lane >= off) v += t;
  }
  return v;
}

// Exclusive scan of one value per thread over a block of NW waves.
template <int NW>
__device__ __forceinline__ int block_excl_scan(int v, int* tmp, int* total) {
  const int wave = threadIdx.x / kWave;
  int incl = wave_incl_scan(v);
  if (lane_id() == kWave - 1) tmp[wave] = incl;
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    int t = tmp[w];
    if (w < wave) off += t;
    tot += t;
  }
  __syncthreads();
  if (total) *total = tot;
  return off + incl - v;
}

// Edge e of the list with appended loops: ids < E_in come from edge_index
// (clamped into range, with *bad set when out of range), ids >= E_in are the
// loops (i, i), i = e - E_in.
template <typename IdxT>
__device__ __forceinline__ void load_edge(const IdxT* __restrict__ src, const IdxT* __restrict__ tgt,
                                          int64_t E_in, int64_t N_src, int64_t N, int64_t e,
                                          int* s, int* t, bool* bad) {
  if (e < E_in) {
    int64_t sv = src ? (int64_t)src[e] : 0;
    int64_t tv = (int64_t)tgt[e];
    bool sbad = src && (sv < 0 || sv >= N_src);
    bool tbad = tv < 0 || tv >= N;
    *bad = sbad || tbad;
    *s = sbad ? 0 : (int)sv;
    *t = tbad ? 0 : (int)tv;
  } else {
    *bad = false;
    *s = *t = (int)(e - E_in);
  }
}

__global__ void fill_int(int* __restrict__ p, int64_t n, int v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// ---------------------------------------------------------------------------
// Device-wide exclusive scan of int32 (three kernels).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kScanThreads) void scan_tile_sums(const int* __restrict__ in, int64_t n,
                                                               int* __restrict__ sums) {
  __shared__ int tmp[kScanThreads / kWave];
  int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  int v = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i)
    if (base + i < n) v += in[base + i];
  int total;
  block_excl_scan<kScanThreads / kWave>(v, tmp, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// In-place exclusive scan of the tile sums by one block.
__global__ __launch_bounds__(1024) void scan_sums(int* __restrict__ sums, int64_t n) {
  __shared__ int tmp[1024 / kWave];
  int carry = 0;
  for (int64_t base = 0; base < n; base += 1024) {
    int64_t i = base + threadIdx.x;
    int v = i < n ? sums[i] : 0;
    int total;
    int ex = block_excl_scan<1024 / kWave>(v, tmp, &total);
    if (i < n) sums[i] = carry + ex;
    carry += total;
  }
}

__global__ __launch_bounds__(kScanThreads) void scan_apply(const int* in, int* out, int64_t n,
                                                           const int* __restrict__ sums) {
  __shared__ int tmp[kScanThreads / kWave];
  int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  int v[kScanItems];
  int tsum = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    v[i] = base + i < n ? in[base + i] : 0;
    tsum += v[i];
  }
  int run = sums[blockIdx.x] + block_excl_scan<kScanThreads / kWave>(tsum, tmp, nullptr);
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    if (base + i < n) out[base + i] = run;
    run += v[i];
  }
}

int64_t scan_tiles(int64_t n) { return (n + kScanTile - 1) / kScanTile; }

int exclusive_scan(const int* in, int* out, int64_t n, int* tile_sums, hipStream_t s) {
  if (n <= 0) return TFG_OK;
  int64_t nt = scan_tiles(n);
  scan_tile_sums<<<dim3((unsigned)nt), dim3(kScanThreads), 0, s>>>(in, n, tile_sums);
  scan_sums<<<1, 1024, 0, s>>>(tile_sums, nt);
  scan_apply<<<dim3((unsigned)nt), dim3(kScanThreads), 0, s>>>(in, out, n, tile_sums);
  TFG_LAUNCHED("exclusive scan");
  return TFG_OK;
}

// ---------------------------------------------------------------------------
// Radix sort passes.
// ---------------------------------------------------------------------------

// First upsweep: validates every edge, counts edges per target (global
// integer atomics: exact, order-free) and builds the block's digit histogram
// for the first pass. hist is digit-major: hist[d * nblocks + block].
template <typename IdxT>
__global__ __launch_bounds__(kSortThreads) void first_upsweep(
    const IdxT* __restrict__ src, const IdxT* __restrict__ tgt, int64_t E_in, int64_t N_src,
    int64_t N, int64_t E, int shift, int dbits, int* __restrict__ cnt, int* __restrict__ hist,
    int nblocks, int* __restrict__ err) {
  __shared__ int h[kMaxRadix];
  const int radix = 1 << dbits;
  for (int d = threadIdx.x; d < radix; d += kSortThreads) h[d] = 0;
  __syncthreads();
  int64_t base = (int64_t)blockIdx.x * kSortTile;
  bool any_bad = false;
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    int64_t e = base + (int64_t)i * kSortThreads + threadIdx.x;
    if (e < E) {
      int s, t;
      bool bad;
      load_edge(src, tgt, E_in, N_src, N, e, &s, &t, &bad);
      any_bad |= bad;
      atomicAdd(&cnt[t], 1);
      atomicAdd(&h[(t >> shift) & (radix - 1)], 1);
    }
  }
  if (any_bad) atomicOr(err, kErrIndex);
  __syncthreads();
  for (int d = threadIdx.x; d < radix; d += kSortThreads) hist[(int64_t)d * nblocks + blockIdx.x] = h[d];
}

__global__ __launch_bounds__(kSortThreads) void upsweep(const int* __restrict__ keys, int64_t E,
                                                        int shift, int dbits,
                                                        int* __restrict__ hist, int nblocks) {
  __shared__ int h[kMaxRadix];
  const int radix = 1 << dbits;
  for (int d = threadIdx.x; d < radix; d += kSortThreads) h[d] = 0;
  __syncthreads();
  int64_t base = (int64_t)blockIdx.x * kSortTile;
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    int64_t e = base + (int64_t)i * kSortThreads + threadIdx.x;
    if (e < E) atomicAdd(&h[(keys[e] >> shift) & (radix - 1)], 1);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < radix; d += kSortThreads) hist[(int64_t)d * nblocks + blockIdx.x] = h[d];
}

// Stable scatter of one tile by one digit. Wave w owns tile positions
// [w*512, (w+1)*512), visited in rounds of 64 consecutive positions, so the
// (wave, round, lane) order is the input order. Within a round, lanes with the
// same digit find each other with one ballot per digit bit; their rank is the
// number of such lanes below them plus the wave's running count of the digit.
// The tile is then staged in LDS in digit order and written out so that
// consecutive threads write consecutive addresses of a digit's run.
//   FIRST: keys/payloads come from edge_index (payload = edge id, source id)
//   LAST : writes perm (edge id) and col (source id) only
template <bool FIRST, bool LAST, typename IdxT>
__global__ __launch_bounds__(kSortThreads) void scatter(
    const IdxT* __restrict__ src, const IdxT* __restrict__ tgt, int64_t E_in, int64_t N_src,
    int64_t N, const int* __restrict__ kin, const int* __restrict__ ein,
    const int* __restrict__ sin, int64_t E, int shift, int dbits,
    const int* __restrict__ hist, int nblocks, int* __restrict__ kout, int* __restrict__ eout,
    int* __restrict__ sout) {
  __shared__ int wcnt[kSortWaves][kMaxRadix];
  __shared__ int loff[kMaxRadix];
  __shared__ int goff[kMaxRadix];
  __shared__ int skey[kSortTile];
  __shared__ int sedge[kSortTile];
  __shared__ int ssrc[kSortTile];
  __shared__ int tmp[kSortWaves];

  const int radix = 1 << dbits;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  const int tile_n = (int)min<int64_t>(kSortTile, E - base);
  const unsigned long long lt = (1ull << lane) - 1ull;

  for (int d = lane; d < kMaxRadix; d += kWave) wcnt[wave][d] = 0;
  __syncthreads();

  int key[kSortItems], edge[kSortItems], sv[kSortItems], rank[kSortItems];
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    int p = wave * (kWave * kSortItems) + i * kWave + lane;  // position in tile
    bool valid = p < tile_n;
    int64_t e = base + p;
    if (valid) {
      if constexpr (FIRST) {
        bool bad;
        load_edge(src, tgt, E_in, N_src, N, e, &sv[i], &key[i], &bad);
        edge[i] = (int)e;
      } else {
        key[i] = kin[e];
        edge[i] = ein[e];
        sv[i] = sin[e];
      }
    } else {
      key[i] = 0;
      edge[i] = 0;
      sv[i] = 0;
    }
    int d = (key[i] >> shift) & (radix - 1);
    unsigned long long peers = __ballot(valid);
    for (int b = 0; b < dbits; ++b) {
      int bit = (d >> b) & 1;
      unsigned long long bb = __ballot(bit);
      peers &= bit ? bb : ~bb;
    }
    int below = __popcll(peers & lt);
    int run = valid ? wcnt[wave][d] : 0;
    rank[i] = run + below;
    if (valid && below == 0) wcnt[wave][d] = run + __popcll(peers);
  }
  __syncthreads();

  // Per digit: exclusive offsets of the waves, the block total, the block's
  // start in LDS (scan over digits) and its start in the output (scanned hist).
  {
    int d = threadIdx.x;  // kSortThreads == kMaxRadix
    int tot = 0;
    if (d < radix) {
#pragma unroll
      for (int w = 0; w < kSortWaves; ++w) {
        int c = wcnt[w][d];
        wcnt[w][d] = tot;
        tot += c;
      }
    }
    int ex = block_excl_scan<kSortWaves>(d < radix ? tot : 0, tmp, nullptr);
    if (d < radix) {
      loff[d] = ex;
      goff[d] = hist[(int64_t)d * nblocks + blockIdx.x];
    }
  }
  __syncthreads();

#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    int p = wave * (kWave * kSortItems) + i * kWave + lane;
    if (p < tile_n) {
      int d = (key[i] >> shift) & (radix - 1);
      int lp = loff[d] + wcnt[wave][d] + rank[i];
      skey[lp] = key[i];
      sedge[lp] = edge[i];
      ssrc[lp] = sv[i];
    }
  }
  __syncthreads();

#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    int p = i * kSortThreads + threadIdx.x;
    if (p < tile_n) {
      int k = skey[p];
      int d = (k >> shift) & (radix - 1);
      int64_t gp = (int64_t)goff[d] + (p - loff[d]);
      if (gp >= 0 && gp < E) {  // always true for a consistent histogram
        if constexpr (!LAST) kout[gp] = k;
        eout[gp] = sedge[p];
        sout[gp] = ssrc[p];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Aggregation work list.
// ---------------------------------------------------------------------------

// Reserves v entries of *ctr for this lane with one atomic per wave; returns
// the lane's first entry.
__device__ __forceinline__ int wave_reserve(int* ctr, int v) {
  int incl = wave_incl_scan(v);
  int total = __shfl(incl, kWave - 1);
  int base = 0;
  if (lane_id() == kWave - 1 && total > 0) base = atomicAdd(ctr, total);
  base = __shfl(base, kWave - 1);
  return base + incl - v;
}

// Rows with at most `chunk` edges become one light item; longer rows are cut
// into ceil(deg / chunk) heavy items whose partial results are combined by
// the fix-up pass. Item order within each list is arbitrary (it only affects
// scheduling, never values).
__global__ __launch_bounds__(kBlock) void build_worklist(const int* __restrict__ rowptr, int64_t N,
                                                         int chunk, int* __restrict__ counters,
                                                         WorkItem* __restrict__ heavy,
                                                         WorkItem* __restrict__ light,
                                                         SplitRow* __restrict__ split) {
  int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int beg = 0, deg = 0;
  if (r < N) {
    beg = rowptr[r];
    deg = rowptr[r + 1] - beg;
  }
  bool valid = r < N;
  bool is_split = valid && deg > chunk;
  int nch = is_split ? (deg + chunk - 1) / chunk : 0;
  int h0 = wave_reserve(&counters[0], nch);
  int l0 = wave_reserve(&counters[1], valid && !is_split ? 1 : 0);
  int s0 = wave_reserve(&counters[2], is_split ? 1 : 0);
  if (!valid) return;
  if (is_split) {
    for (int j = 0; j < nch; ++j) {
      int kb = beg + j * chunk;
      heavy[h0 + j] = WorkItem{(int)r, kb, min(kb + chunk, beg + deg), h0 + j};
    }
    split[s0] = SplitRow{(int)r, h0, nch, deg};
  } else {
    light[l0] = WorkItem{(int)r, beg, beg + deg, -1};
  }
}

int ceil_log2(int64_t n) {
  int b = 0;
  while ((int64_t(1) << b) < n) ++b;
  return b;
}

struct SortPlan {
  int bits, passes, dbits;
  int64_t nblocks;
};

SortPlan sort_plan(int64_t E, int64_t N) {
  SortPlan p;
  p.bits = std::max(1, ceil_log2(std::max<int64_t>(N, 2)));
  p.passes = (p.bits + kMaxDigitBits - 1) / kMaxDigitBits;
  p.dbits = (p.bits + p.passes - 1) / p.passes;
  p.nblocks = (E + kSortTile - 1) / kSortTile;
  return p;
}

struct ScratchLayout {
  size_t cnt, hist, sums, bufA, bufB, total;
};

ScratchLayout scratch_layout(int64_t E, int64_t N) {
  SortPlan p = sort_plan(E, N);
  ScratchLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  int64_t hist_n = (int64_t)(1 << p.dbits) * p.nblocks;
  int64_t scan_n = std::max<int64_t>(hist_n, N + 1);
  L.cnt = take(sizeof(int) * (N + 1));
  L.hist = take(sizeof(int) * std::max<int64_t>(hist_n, 1));
  L.sums = take(sizeof(int) * std::max<int64_t>(scan_tiles(scan_n), 1));
  L.bufA = take(sizeof(int) * 3 * std::max<int64_t>(E, 1));
  L.bufB = take(p.passes >= 3 ? sizeof(int) * 3 * std::max<int64_t>(E, 1) : 0);
  L.total = off;
  return L;
}

template <typename IdxT>
int sort_edges(Graph& g, const IdxT* src, const IdxT* tgt, char* scratch, const ScratchLayout& L,
               hipStream_t s) {
  const int64_t E = g.E;
  SortPlan p = sort_plan(E, g.N);
  int* cnt = reinterpret_cast<int*>(scratch + L.cnt);
  int* hist = reinterpret_cast<int*>(scratch + L.hist);
  int* sums = reinterpret_cast<int*>(scratch + L.sums);
  int* bufs[2][3];
  for (int b = 0; b < 2; ++b) {
    int* base = reinterpret_cast<int*>(scratch + (b == 0 ? L.bufA : L.bufB));
    for (int j = 0; j < 3; ++j) bufs[b][j] = base + j * E;
  }
  int* err = g.counters + 3;
  const unsigned nb = (unsigned)p.nblocks;
  const int64_t hist_n = (int64_t)(1 << p.dbits) * p.nblocks;

  fill_int<<<dim3((unsigned)((g.N + 1 + 255) / 256)), dim3(256), 0, s>>>(cnt, g.N + 1, 0);
  if (E > 0) {
    first_upsweep<IdxT><<<nb, kSortThreads, 0, s>>>(src, tgt, g.E_in, g.N_src, g.N, E, 0, p.dbits,
                                                    cnt, hist, (int)p.nblocks, err);
    TFG_LAUNCHED("first_upsweep");
    int rc = exclusive_scan(hist, hist, hist_n, sums, s);
    if (rc) return rc;
    int cur = 0;  // which scratch buffer holds the current keys
    for (int pass = 0; pass < p.passes; ++pass) {
      const int shift = pass * p.dbits;
      const bool first = pass == 0, last = pass == p.passes - 1;
      if (!first) {
        upsweep<<<nb, kSortThreads, 0, s>>>(bufs[cur][0], E, shift, p.dbits, hist, (int)p.nblocks);
        rc = exclusive_scan(hist, hist, hist_n, sums, s);
        if (rc) return rc;
      }
      int nxt = first ? 0 : 1 - cur;
      int* ko = last ? nullptr : bufs[nxt][0];
      int* eo = last ? g.perm : bufs[nxt][1];
      int* so = last ? g.col : bufs[nxt][2];
      const int *ki = bufs[cur][0], *ei = bufs[cur][1], *si = bufs[cur][2];
      if (first && last)
        scatter<true, true, IdxT><<<nb, kSortThreads, 0, s>>>(src, tgt, g.E_in, g.N_src, g.N, ki, ei,
                                                             si, E, shift, p.dbits, hist,
                                                             (int)p.nblocks, ko, eo, so);
      else if (first)
        scatter<true, false, IdxT><<<nb, kSortThreads, 0, s>>>(src, tgt, g.E_in, g.N_src, g.N, ki, ei,
                                                              si, E, shift, p.dbits, hist,
                                                              (int)p.nblocks, ko, eo, so);
      else if (last)
        scatter<false, true, IdxT><<<nb, kSortThreads, 0, s>>>(src, tgt, g.E_in, g.N_src, g.N, ki, ei,
                                                              si, E, shift, p.dbits, hist,
                                                              (int)p.nblocks, ko, eo, so);
      else
        scatter<false, false, IdxT><<<nb, kSortThreads, 0, s>>>(src, tgt, g.E_in, g.N_src, g.N, ki,
                                                               ei, si, E, shift, p.dbits, hist,
                                                               (int)p.nblocks, ko, eo, so);
      TFG_LAUNCHED("radix scatter");
      cur = nxt;
    }
  }
  // rowptr = exclusive scan of the per-target counts (cnt[N] = 0 gives rowptr[N] = E)
  return exclusive_scan(cnt, g.rowptr, g.N + 1, sums, s);
}

}  // namespace

int default_chunk() {
  static int chunk = [] {
    const char* v = std::getenv("TFG_ROW_CHUNK");
    int c = v ? std::atoi(v) : kDefaultChunk;
    return c >= 64 ? c : kDefaultChunk;
  }();
  return chunk;
}

GraphLayout graph_layout(int64_t E, int64_t N, int chunk) {
  GraphLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  // split rows have > chunk edges each: at most E / chunk of them, and their
  // chunks number at most 2 * E / chunk
  L.cap_split = std::min<int64_t>(N, E / chunk + 1);
  L.cap_heavy = 2 * (E / chunk) + 2;
  L.cap_light = N;
  L.rowptr = take(sizeof(int) * (N + 1));
  L.col = take(sizeof(int) * std::max<int64_t>(E, 1));
  L.perm = take(sizeof(int) * std::max<int64_t>(E, 1));
  L.heavy = take(sizeof(WorkItem) * L.cap_heavy);
  L.light = take(sizeof(WorkItem) * std::max<int64_t>(L.cap_light, 1));
  L.split = take(sizeof(SplitRow) * std::max<int64_t>(L.cap_split, 1));
  L.counters = take(sizeof(int) * 4);
  L.total = off;
  return L;
}

size_t graph_scratch_bytes(int64_t E, int64_t N) { return scratch_layout(E, N).total; }

int build_graph(Graph& g, const void* src, const void* tgt, int index_type, void* scratch,
                size_t scratch_bytes, hipStream_t s) {
  ScratchLayout L = scratch_layout(g.E, g.N);
  if (scratch_bytes < L.total) return fail(TFG_ERR_WORKSPACE, "graph scratch buffer too small");
  char* sc = static_cast<char*>(scratch);
  fill_int<<<1, 64, 0, s>>>(g.counters, 4, 0);
  int rc;
  if (index_type == TFG_I64)
    rc = sort_edges<int64_t>(g, static_cast<const int64_t*>(src), static_cast<const int64_t*>(tgt),
                             sc, L, s);
  else
    rc = sort_edges<int32_t>(g, static_cast<const int32_t*>(src), static_cast<const int32_t*>(tgt),
                             sc, L, s);
  if (rc) return rc;
  if (g.N > 0) {
    build_worklist<<<dim3((unsigned)((g.N + kBlock - 1) / kBlock)), dim3(kBlock), 0, s>>>(
        g.rowptr, g.N, g.chunk, g.counters, g.heavy, g.light, g.split);
    TFG_LAUNCHED("build_worklist");
  }
  int host[4];
  TFG_HIP(hipMemcpyAsync(host, g.counters, sizeof(host), hipMemcpyDeviceToHost, s));
  TFG_HIP(hipStreamSynchronize(s));
  if (host[3] & kErrIndex) return fail(TFG_ERR_INDEX_RANGE, "edge_index holds an id outside [0, N)");
  g.n_heavy = host[0];
  g.n_light = host[1];
  g.n_split = host[2];
  return TFG_OK;
}

}  // namespace tfg
