// COO -> CSR by target on the GPU (gfx950).
//
// The edges are sorted by the key (target, source part) with a stable LSD
// radix sort, so the permutation is the unique one that orders the keys and
// keeps the input order among equal keys (bit-identical to a sequential
// counting sort). With one source part this is the CSR by target.
//
// Per radix pass: an upsweep counts the digits of every 8192-edge tile into
// one column of a digit-major table, one device-wide exclusive scan of the
// table turns the counts into output offsets, and a scatter ranks each tile
// stably (one ballot per digit bit per 64 edges), stages it in LDS in digit
// order and writes every digit's run with consecutive addresses. Row pointers
// come from the run boundaries of the sorted keys; the aggregation work lists
// from the row pointers (per-block counts and a scan, no atomics).
#include <algorithm>
#include <cmath>
#include <cstdlib>

#include "wave.h"

namespace tfg {
namespace {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;  // 2048

constexpr int kSortThreads = 1024;                    // 16 waves
constexpr int kSortItems = 8;                         // items per thread
constexpr int kSortTile = kSortThreads * kSortItems;  // 8192 edges per tile
constexpr int kSortWaves = kSortThreads / kWave;
constexpr int kUpThreads = 512;                       // counting pass: threads per tile
constexpr int kUpItems = kSortTile / kUpThreads;
constexpr int kMaxDigitBits = 8;
constexpr int kMaxRadix = 1 << kMaxDigitBits;         // 256
constexpr int kXcds = 8;

// Blocks are dispatched round-robin over the XCDs; tile_of() gives each XCD a
// contiguous range of tiles, so neighbouring tiles (whose runs of one digit
// are adjacent in the output) share an L2.
__device__ __forceinline__ int tile_of(int bid, int ntiles) {
  const int q = ntiles / kXcds, r = ntiles % kXcds;
  const int x = bid % kXcds, i = bid / kXcds;
  return x * q + min(x, r) + i;
}

// Number of lanes below this one whose bit is set in mask.
__device__ __forceinline__ int lanes_below(unsigned long long mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((unsigned)(mask >> 32),
                                        __builtin_amdgcn_mbcnt_lo((unsigned)mask, 0u));
}

// Edge e of the list with appended loops, as (source, sort key). Ids < E_in
// come from edge_index (an out-of-range id is replaced by 0 and flagged), ids
// >= E_in are the loops (i, i), i = e - E_in. key = target * P + source part.
struct KeyMap {
  int64_t E_in, N_src, N;
  int part_rows, parts;
  double inv_part_rows, half_inv_part_rows;  // 1 / part_rows and 0.5 / part_rows
};

// floor(s / part_rows) for 0 <= s < 2^31, as the truncation of
// (s + 1/2) / part_rows in double: the fraction of s / part_rows is at most
// (part_rows - 1) / part_rows, so adding 1 / (2 part_rows) never reaches the
// next integer, and the double's relative error (a few 2^-53) is far below
// that margin of 1 / (2 part_rows) for every s < 2^51.
__device__ __forceinline__ int source_part(int s, const KeyMap& m) {
  return (int)fma((double)s, m.inv_part_rows, m.half_inv_part_rows);
}

// Edges are addressed inside a tile: position p is edge base + p, and
// d = E_in - base (the tile's count of input edges when 0 <= d <= tile size)
// makes the input / loop test and the loop id 32-bit: p < d is an input
// edge, otherwise the loop on node p - d.
__device__ __forceinline__ int input_edges_before(int64_t E_in, int64_t base) {
  return (int)(E_in - base);  // |E_in - base| < 2^31: both below 2^31
}

// The raw ids of the N tile positions p0 + i * step, every load issued
// before any is used (the conditions are uniform: they depend on the tile
// only; values of positions past the tile are never used).
template <int N, typename IdxT>
__device__ __forceinline__ void load_raw_all(const IdxT* __restrict__ sb,
                                             const IdxT* __restrict__ tb, int p0, int step,
                                             int tile_n, int d, IdxT (&s)[N], IdxT (&t)[N]) {
  // byte offsets from the tile's base addresses, 32-bit (positions < 2^13),
  // shared by the source and target loads; positions past the input edges
  // (loops) read the last input edge, and a tile of loops only reads nothing
  const bool any = d > 0, has_src = sb != nullptr;
  const int last = min(tile_n, d) - 1;
  const char* sc = reinterpret_cast<const char*>(sb);
  const char* tc = reinterpret_cast<const char*>(tb);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const unsigned q = (unsigned)min(p0 + i * step, last) * (unsigned)sizeof(IdxT);
    s[i] = (any && has_src) ? __builtin_nontemporal_load(reinterpret_cast<const IdxT*>(sc + q))
                            : IdxT(0);
    t[i] = any ? __builtin_nontemporal_load(reinterpret_cast<const IdxT*>(tc + q)) : IdxT(0);
  }
}

template <typename IdxT>
__device__ __forceinline__ void decode_ids(const KeyMap& m, int p, int d, IdxT s, IdxT t,
                                           bool has_src, int* sv, int* tv, bool* bad) {
  const bool in = p < d;
  bool sbad, tbad;
  if constexpr (sizeof(IdxT) == 4) {  // counts are below 2^31: one unsigned compare
    sbad = has_src && (unsigned)s >= (unsigned)m.N_src;
    tbad = (unsigned)t >= (unsigned)m.N;
  } else {
    sbad = has_src && (s < 0 || (int64_t)s >= m.N_src);
    tbad = t < 0 || (int64_t)t >= m.N;
  }
  const int loop = p - d;
  *sv = in ? (sbad ? 0 : (int)s) : loop;
  *tv = in ? (tbad ? 0 : (int)t) : loop;
  *bad = in && (sbad || tbad);
}

template <typename IdxT>
__device__ __forceinline__ void decode_edge(const KeyMap& m, int p, int d, IdxT s, IdxT t,
                                            bool has_src, int* sv, int* key, bool* bad) {
  int tv;
  decode_ids(m, p, d, s, t, has_src, sv, &tv, bad);
  *key = m.parts == 1 ? tv : tv * m.parts + source_part(*sv, m);
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

// In-place exclusive scan of a short array by one block, 8 consecutive
// values per thread (for the small tables of small graphs: one launch
// instead of three).
constexpr int kSmallScan = 32768;
__global__ __launch_bounds__(1024) void scan_small(int* __restrict__ a, int64_t n) {
  __shared__ int tmp[1024 / kWave];
  int carry = 0;
  for (int64_t base = 0; base < n; base += 1024 * 8) {
    const int64_t i0 = base + (int64_t)threadIdx.x * 8;
    int v[8], t = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      v[j] = i0 + j < n ? a[i0 + j] : 0;
      t += v[j];
    }
    int total;
    int run = carry + block_excl_scan<1024 / kWave>(t, tmp, &total);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (i0 + j < n) a[i0 + j] = run;
      run += v[j];
    }
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

// ---------------------------------------------------------------------------
// Radix sort passes.
// ---------------------------------------------------------------------------

// Digit counts of one tile, written as column `tile` of the digit-major table
// hist[d * ntiles + tile]; an exclusive scan of the whole table then gives
// every (digit, tile) its output offset. The first pass also validates the
// ids.
template <bool FIRST, typename IdxT>
__global__ __launch_bounds__(kUpThreads) void upsweep(const IdxT* __restrict__ src,
                                                        const IdxT* __restrict__ tgt, KeyMap m,
                                                        const int* __restrict__ keys, int64_t E,
                                                        int shift, int dbits,
                                                        int* __restrict__ hist,
                                                        int* __restrict__ err) {
  // one histogram per wave: equal digits (a hub target's edges) then contend
  // only within a wave
  __shared__ int h[kUpThreads / kWave][kMaxRadix];
  const int radix = 1 << dbits;
  const int wave = threadIdx.x / kWave;
  for (int d = lane_id(); d < radix; d += kWave) h[wave][d] = 0;
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  const int tile_n = (int)min<int64_t>(kSortTile, E - base);
  const int d = input_edges_before(m.E_in, base);
  const IdxT* sb = src ? src + base : nullptr;
  const IdxT* tb = tgt + base;
  IdxT rs[kUpItems], rt[kUpItems];
  if constexpr (FIRST) {
    // read for every position (clamped to the tile's last input edge, or not
    // read when the tile has none), so that all loads are issued together
#pragma unroll
    for (int i = 0; i < kUpItems; ++i) {
      const int p = i * kUpThreads + (int)threadIdx.x;
      const int c = p < d ? p : d - 1;
      rs[i] = (sb && d > 0) ? __builtin_nontemporal_load(sb + c) : IdxT(0);
      rt[i] = d > 0 ? __builtin_nontemporal_load(tb + c) : IdxT(0);
    }
  } else {
#pragma unroll
    for (int i = 0; i < kUpItems; ++i) {
      const int p = i * kUpThreads + (int)threadIdx.x;
      rt[i] = (IdxT)__builtin_nontemporal_load(keys + base + (p < tile_n ? p : tile_n - 1));
      rs[i] = 0;
    }
  }
  bool any_bad = false;
#pragma unroll
  for (int i = 0; i < kUpItems; ++i) {
    const int p = i * kUpThreads + (int)threadIdx.x;
    int k = (int)rt[i];
    if constexpr (FIRST) {
      int sv;
      bool bad;
      decode_edge(m, p, d, rs[i], rt[i], sb != nullptr, &sv, &k, &bad);
      any_bad |= bad && p < tile_n;
    }
    // (a logical shift: packed words use the sign bit)
    if (p < tile_n) atomicAdd(&h[wave][(int)((unsigned)k >> shift) & (radix - 1)], 1);
  }
  if (FIRST && any_bad) atomicOr(err, kErrIndex);
  __syncthreads();
  for (int d = threadIdx.x; d < radix; d += kUpThreads) {
    int c = 0;
#pragma unroll
    for (int w = 0; w < kUpThreads / kWave; ++w) c += h[w][d];
    hist[(int64_t)d * gridDim.x + blockIdx.x] = c;
  }
}

// Tables of at most this many tiles are not scanned by a launch of their own:
// every scatter block adds up the counts it needs from the raw table.
constexpr int kInBlockTiles = 64;

// Output offset of digit d's run in this tile. scanned: hist holds the
// exclusive scan of the digit-major table (the offset itself); otherwise the
// raw counts, and the offset is the total of the digits below d plus the
// counts of d in the tiles before this one. Every thread of the block calls
// it (a block scan inside when !scanned); threads d >= radix get 0.
__device__ __forceinline__ int tile_offset(const int* __restrict__ hist, int d, int radix,
                                           int ntiles, int tile, int scanned, int* tmp) {
  if (scanned) return d < radix ? hist[(int64_t)d * ntiles + tile] : 0;
  int pre = 0, tot = 0;
  if (d < radix)
    for (int t = 0; t < ntiles; ++t) {
      const int h = hist[d * ntiles + t];
      tot += h;
      pre += t < tile ? h : 0;
    }
  return block_excl_scan<kSortWaves>(d < radix ? tot : 0, tmp, nullptr) + (d < radix ? pre : 0);
}

// Stable scatter of one tile by one digit. Wave w owns tile positions
// [w*512, (w+1)*512), visited in rounds of 64 consecutive positions, so the
// (wave, round, lane) order is the input order. Within a round, lanes with the
// same digit find each other with one ballot per digit bit; their rank is the
// number of such lanes below them plus the wave's running count of the digit.
// The tile is then staged in LDS in digit order in two rounds (keys with edge
// ids in two buffers, then source ids) and written out so that consecutive
// threads write consecutive addresses of a digit's run.
//   FIRST: keys and payloads come from edge_index (payload: edge id, source)
// (16-wave blocks; at most 64 VGPRs so that two blocks fit on a CU)
template <bool FIRST, typename IdxT>
__global__ __launch_bounds__(kSortThreads, 8) void scatter(
    const IdxT* __restrict__ src, const IdxT* __restrict__ tgt, KeyMap m,
    const int* __restrict__ kin, const int* __restrict__ ein, const int* __restrict__ sin,
    int64_t E, int shift, int dbits, const int* __restrict__ hist, int ntiles, int scanned,
    int* __restrict__ kout, int* __restrict__ eout, int* __restrict__ sout) {
  __shared__ unsigned short wcnt[kSortWaves][kMaxRadix];
  __shared__ int loff[kMaxRadix];
  __shared__ int goff[kMaxRadix];
  __shared__ int stage[2][kSortTile];
  __shared__ int tmp[kSortWaves];

  const int radix = 1 << dbits;
  const int lane = lane_id();
  const int wave = uniform((int)threadIdx.x / kWave);
  const int tile = tile_of((int)blockIdx.x, ntiles);
  const int64_t base = (int64_t)tile * kSortTile;
  const int tile_n = (int)min<int64_t>(kSortTile, E - base);

  for (int d = lane; d < kMaxRadix; d += kWave) wcnt[wave][d] = 0;
  // the tile's output offset of digit threadIdx.x, first, while few registers
  // are live (placed in LDS with the local offsets, after the ranking)
  const int go = tile_offset(hist, (int)threadIdx.x, radix, ntiles, tile, scanned, tmp);
  __syncthreads();

  // Keys and payloads are loaded together up front (one round of memory
  // latency per tile). In the first pass the edge id is the position itself
  // and the source id comes out of the key's decoding.
  int key[kSortItems], lpos[kSortItems], pe[FIRST ? 1 : kSortItems], ps[kSortItems];
  const int d = input_edges_before(m.E_in, base);
  const IdxT* sb = src ? src + base : nullptr;
  const IdxT* tb = tgt + base;
  const int p0 = wave * (kWave * kSortItems) + lane;  // position of item i: p0 + i * 64
  if constexpr (FIRST) {
    // (items past the tile decode garbage that is never used)
    IdxT rs[kSortItems], rt[kSortItems];
    load_raw_all(sb, tb, p0, kWave, tile_n, d, rs, rt);
#pragma unroll
    for (int i = 0; i < kSortItems; ++i) {
      bool bad;
      decode_edge(m, p0 + i * kWave, d, rs[i], rt[i], sb != nullptr, &ps[i], &key[i], &bad);
    }
  } else {
#pragma unroll
    for (int i = 0; i < kSortItems; ++i) {
      const int c = min(p0 + i * kWave, tile_n - 1);  // clamped to the tile's last
      key[i] = kin[base + c];
      pe[i] = ein[base + c];
      ps[i] = sin[base + c];
    }
  }
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    const int p = wave * (kWave * kSortItems) + i * kWave + lane;
    const bool valid = p < tile_n;
    const int d = (key[i] >> shift) & (radix - 1);
    unsigned long long peers = __ballot(valid);
    for (int b = 0; b < dbits; ++b) {
      const int bit = (d >> b) & 1;
      const unsigned long long bb = __ballot(bit);
      peers &= bit ? bb : ~bb;
    }
    const int below = lanes_below(peers);
    const int run = valid ? (int)wcnt[wave][d] : 0;
    lpos[i] = run + below;  // rank within the wave for now
    if (valid && below == 0) wcnt[wave][d] = (unsigned short)(run + __popcll(peers));
  }
  __syncthreads();

  // Per digit: exclusive offsets of the waves, the tile's start in LDS (scan
  // over digits) and its start in the output.
  {
    const int d = threadIdx.x;
    int tot = 0;
    if (d < radix) {
#pragma unroll
      for (int w = 0; w < kSortWaves; ++w) {
        const int c = wcnt[w][d];
        wcnt[w][d] = (unsigned short)tot;
        tot += c;
      }
    }
    const int ex = block_excl_scan<kSortWaves>(d < radix ? tot : 0, tmp, nullptr);
    if (d < radix) {
      loff[d] = ex;
      goff[d] = go;
    }
  }
  __syncthreads();

#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    const int p = wave * (kWave * kSortItems) + i * kWave + lane;
    const int d = (key[i] >> shift) & (radix - 1);
    // -1 marks positions past the end of the tile
    lpos[i] = p < tile_n ? lpos[i] + loff[d] + (int)wcnt[wave][d] : -1;
  }

  // keys and edge ids: stage both, then every thread writes positions
  // threadIdx.x + i * 1024 of each
  int gpos[kSortItems];
#pragma unroll
  for (int i = 0; i < kSortItems; ++i)
    if (lpos[i] >= 0) {
      stage[0][lpos[i]] = key[i];
      if constexpr (FIRST)
        stage[1][lpos[i]] = (int)(base + wave * (kWave * kSortItems) + i * kWave + lane);
      else
        stage[1][lpos[i]] = pe[i];
    }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    const int p = i * kSortThreads + threadIdx.x;
    gpos[i] = -1;
    if (p < tile_n) {
      const int k = stage[0][p];
      const int d = (k >> shift) & (radix - 1);
      const int64_t gp = (int64_t)goff[d] + (p - loff[d]);
      if (gp >= 0 && gp < E) {  // always true for a consistent histogram
        gpos[i] = (int)gp;
        kout[gp] = k;
        eout[gp] = stage[1][p];
      }
    }
  }
  __syncthreads();
  // source ids
#pragma unroll
  for (int i = 0; i < kSortItems; ++i)
    if (lpos[i] >= 0) stage[0][lpos[i]] = ps[i];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kSortItems; ++i)
    if (gpos[i] >= 0) sout[gpos[i]] = stage[0][i * kSortThreads + threadIdx.x];
}

// Packed payloads. When P is a power of two (key = target << log2 P | source
// part) and the ids and positions fit in 64 bits, an edge travels between
// the passes as two words instead of three,
//   A = target << (32 - bt) | source >> sl,
//   B = (source mod 2^sl) << be | edge id,
// with bt, bs, be the bit widths of target, source and position and
// sl = max(0, bs - (32 - bt)) (so sl + be <= 32). The key's digits above the
// source part are bits of A; the first pass's digit and the last pass's key
// are recomputed from the unpacked ids. The middle passes then move 8 bytes
// per edge instead of 12 and stage two words in LDS instead of three.
struct PackMap {
  int bt, sl, be, lp;  // target bits, source bits kept in B, position bits, log2 P
};

__device__ __forceinline__ unsigned pack_a(int t, int sv, const PackMap& q) {
  return ((unsigned)t << (32 - q.bt)) | ((unsigned)sv >> q.sl);
}
__device__ __forceinline__ unsigned pack_b(int sv, int e, const PackMap& q) {
  return (q.sl > 0 ? ((unsigned)sv & ((1u << q.sl) - 1u)) << q.be : 0u) | (unsigned)e;
}
__device__ __forceinline__ int unpack_t(unsigned a, const PackMap& q) {
  return (int)(a >> (32 - q.bt));
}
__device__ __forceinline__ int unpack_s(unsigned a, unsigned b, const PackMap& q) {
  const unsigned hi = (a & ((1u << (32 - q.bt)) - 1u)) << q.sl;
  return (int)(q.sl > 0 ? hi | (b >> q.be) : hi);
}
__device__ __forceinline__ int unpack_e(unsigned b, const PackMap& q) {
  return (int)(b & ((1u << q.be) - 1u));
}
__device__ __forceinline__ int packed_key(unsigned a, unsigned b, const KeyMap& m,
                                          const PackMap& q) {
  return (unpack_t(a, q) << q.lp) | source_part(unpack_s(a, b, q), m);
}

// The first pass's digit: the low bits of target << log2 P | source part.
__device__ __forceinline__ int first_digit(unsigned a, unsigned b, const KeyMap& m,
                                           const PackMap& q, int radix) {
  const int part = q.lp == 0 ? 0 : source_part(unpack_s(a, b, q), m);
  return ((unpack_t(a, q) << q.lp) | part) & (radix - 1);
}

// The scatter of one pass over packed payloads; the ranking and staging are
// those of scatter() above. MODE 0: the first pass (reads edge_index, writes
// A and B); 1: a middle pass (A and B to A and B); 2: the last pass (A and B
// to the sorted key, edge id and source). `shift` is the digit's position in
// the key (first pass) or in A (the other passes).
template <int MODE, typename IdxT>
__global__ __launch_bounds__(kSortThreads, 8) void scatter_packed(
    const IdxT* __restrict__ src, const IdxT* __restrict__ tgt, KeyMap m, PackMap q,
    const unsigned* __restrict__ ain, const unsigned* __restrict__ bin, int64_t E, int shift,
    int dbits, const int* __restrict__ hist, int ntiles, int scanned, int* __restrict__ o0,
    int* __restrict__ o1, int* __restrict__ o2) {
  __shared__ unsigned short wcnt[kSortWaves][kMaxRadix];
  __shared__ int loff[kMaxRadix];
  __shared__ int goff[kMaxRadix];
  __shared__ uint2 stage[kSortTile];  // (A, B) per staged position: one 8-byte access each
  __shared__ int tmp[kSortWaves];

  const int radix = 1 << dbits;
  const int lane = lane_id();
  const int wave = uniform((int)threadIdx.x / kWave);
  const int tile = tile_of((int)blockIdx.x, ntiles);
  const int64_t base = (int64_t)tile * kSortTile;
  const int tile_n = (int)min<int64_t>(kSortTile, E - base);

  for (int d = lane; d < kMaxRadix; d += kWave) wcnt[wave][d] = 0;
  // the tile's output offset of digit threadIdx.x, first, while few registers
  // are live (placed in LDS with the local offsets, after the ranking)
  const int go = tile_offset(hist, (int)threadIdx.x, radix, ntiles, tile, scanned, tmp);
  __syncthreads();

  // pk: the digit in the upper half, below it first the rank within the
  // wave, then the position in the tile (0xFFFF: past the end of the tile)
  unsigned va[kSortItems], vb[kSortItems];
  int pk[kSortItems];
  {
    const int d = input_edges_before(m.E_in, base);
    const IdxT* sb = src ? src + base : nullptr;
    const IdxT* tb = tgt + base;
    const int p0 = wave * (kWave * kSortItems) + lane;  // position of item i: p0 + i * 64
    if constexpr (MODE == 0) {
      // (items past the tile decode garbage that is never used)
      IdxT rs[kSortItems], rt[kSortItems];
      load_raw_all(sb, tb, p0, kWave, tile_n, d, rs, rt);
#pragma unroll
      for (int i = 0; i < kSortItems; ++i) {
        const int p = p0 + i * kWave;
        int sv, tv;
        bool bad;
        decode_ids(m, p, d, rs[i], rt[i], sb != nullptr, &sv, &tv, &bad);
        const int part = q.lp == 0 ? 0 : source_part(sv, m);  // P = 2^lp
        va[i] = pack_a(tv, sv, q);
        vb[i] = pack_b(sv, (int)base + p, q);
        pk[i] = ((tv << q.lp) | part) & (radix - 1);
      }
    } else {
#pragma unroll
      for (int i = 0; i < kSortItems; ++i) {
        const int c = min(p0 + i * kWave, tile_n - 1);  // clamped to the tile's last
        va[i] = ain[base + c];
        vb[i] = bin[base + c];
      }
#pragma unroll
      for (int i = 0; i < kSortItems; ++i) pk[i] = (int)(va[i] >> shift) & (radix - 1);
    }
  }
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    const int p = wave * (kWave * kSortItems) + i * kWave + lane;
    const bool valid = p < tile_n;
    const int d = pk[i];
    unsigned long long peers = __ballot(valid);
    for (int b = 0; b < dbits; ++b) {
      const int bit = (d >> b) & 1;
      const unsigned long long bb = __ballot(bit);
      peers &= bit ? bb : ~bb;
    }
    const int below = lanes_below(peers);
    const int run = valid ? (int)wcnt[wave][d] : 0;
    pk[i] = (d << 16) | (run + below);
    if (valid && below == 0) wcnt[wave][d] = (unsigned short)(run + __popcll(peers));
  }
  __syncthreads();
  {
    const int d = threadIdx.x;
    int tot = 0;
    if (d < radix) {
#pragma unroll
      for (int w = 0; w < kSortWaves; ++w) {
        const int c = wcnt[w][d];
        wcnt[w][d] = (unsigned short)tot;
        tot += c;
      }
    }
    const int ex = block_excl_scan<kSortWaves>(d < radix ? tot : 0, tmp, nullptr);
    if (d < radix) {
      loff[d] = ex;
      goff[d] = go;
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    const int p = wave * (kWave * kSortItems) + i * kWave + lane;
    const int d = pk[i] >> 16;
    const int pos = p < tile_n ? (pk[i] & 0xFFFF) + loff[d] + (int)wcnt[wave][d] : 0xFFFF;
    pk[i] = (d << 16) | pos;
  }
  static_assert(kSortTile < 0xFFFF, "tile positions fit below the 16-bit marker");
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    const int pos = pk[i] & 0xFFFF;
    if (pos != 0xFFFF) {
      stage[pos] = make_uint2(va[i], vb[i]);
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    const int p = i * kSortThreads + threadIdx.x;
    if (p < tile_n) {
      const uint2 ab = stage[p];
      const unsigned a = ab.x, b = ab.y;
      // the first pass's digit is not a field of A: it is recomputed from
      // the unpacked ids, as the decode formed it
      const int d = MODE == 0 ? first_digit(a, b, m, q, radix)
                              : (int)(a >> shift) & (radix - 1);
      const int64_t gp = (int64_t)goff[d] + (p - loff[d]);
      if (gp >= 0 && gp < E) {  // always true for a consistent histogram
        if constexpr (MODE == 2) {
          o0[gp] = packed_key(a, b, m, q);
          o1[gp] = unpack_e(b, q);
          o2[gp] = unpack_s(a, b, q);
        } else {
          o0[gp] = (int)a;
          o1[gp] = (int)b;
        }
      }
    }
  }
}

// bounds[v] = first position whose sorted key is >= v (v = 0..K). Position k
// starts the keys (key[k-1], key[k]]; k = E closes the keys after the last one.
// Each thread takes kKbGroups groups of four positions (a group per 16-byte
// load, consecutive threads on consecutive groups, all loads issued
// together); the key before a group comes from the neighbouring lane.
constexpr int kKbThreads = 256;  // threads per block of key_bounds
constexpr int kKbGroups = 4;     // groups of four positions per thread
__global__ __launch_bounds__(kKbThreads) void key_bounds(const int* __restrict__ keys, int64_t E,
                                                     int64_t K, int* __restrict__ bounds) {
  typedef int i4 __attribute__((ext_vector_type(4)));
  const int lane = lane_id();
  int c[kKbGroups][4], before[kKbGroups];
#pragma unroll
  for (int j = 0; j < kKbGroups; ++j) {
    const int64_t k0 = (((int64_t)blockIdx.x * kKbGroups + j) * kKbThreads + threadIdx.x) * 4;
    if (k0 + 4 <= E) {
      const i4 v = __builtin_nontemporal_load(reinterpret_cast<const i4*>(keys + k0));
      c[j][0] = v.x;
      c[j][1] = v.y;
      c[j][2] = v.z;
      c[j][3] = v.w;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) c[j][i] = k0 + i < E ? keys[k0 + i] : (int)K;
    }
    before[j] = (lane == 0 && k0 > 0 && k0 <= E) ? keys[k0 - 1] : -1;
  }
#pragma unroll
  for (int j = 0; j < kKbGroups; ++j) {
    const int64_t k0 = (((int64_t)blockIdx.x * kKbGroups + j) * kKbThreads + threadIdx.x) * 4;
    // lane l - 1 holds keys[k0 - 1] whenever this lane has positions to close
    int prev = __shfl_up(c[j][3], 1);
    if (lane == 0) prev = before[j];
    if (k0 > E) continue;
    int64_t cur = prev;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (k0 + i > E) break;
      for (int64_t v = cur + 1; v <= c[j][i]; ++v) bounds[v] = (int)(k0 + i);
      cur = c[j][i];
    }
  }
}

__global__ __launch_bounds__(kBlock) void rows_from_segments(const int* __restrict__ segptr,
                                                             int64_t N, int parts,
                                                             int* __restrict__ rowptr) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t <= N) rowptr[t] = segptr[t * parts];
}

// ---------------------------------------------------------------------------
// Aggregation work lists.
// ---------------------------------------------------------------------------

// Row plan: rows with at most `chunk` edges become one light item; longer
// rows are cut into ceil(deg / chunk) heavy items whose partial results the
// fix-up pass combines. The light rows are listed again by length (short:
// at most kShortRow edges; long: the others). Every list is in row order:
// per-block counts, one scan of them, then a fill pass (no atomics).
constexpr int kWlThreads = 1024;  // rows per block of the work-list kernels
constexpr int kLists = 5;         // heavy chunks, light, split, short, long
__constant__ const int kListCounter[kLists] = {0, 1, 2, 5, 6};  // their slots in counters

// Entries of a row of `deg` edges in each list.
__device__ __forceinline__ void row_counts(bool valid, int deg, int chunk, int (&c)[kLists]) {
  const bool split = valid && deg > chunk;
  const bool shrt = valid && deg <= kShortRow;
  c[0] = split ? (deg + chunk - 1) / chunk : 0;
  c[1] = valid && !split;
  c[2] = split;
  c[3] = shrt;
  c[4] = valid && !split && !shrt;
}

__device__ __forceinline__ void row_entries(const int* __restrict__ rowptr, int64_t N, int chunk,
                                            int64_t r, int* beg, int* deg, int (&c)[kLists]) {
  *beg = 0;
  *deg = 0;
  if (r < N) {
    *beg = rowptr[r];
    *deg = rowptr[r + 1] - *beg;
  }
  row_counts(r < N, *deg, chunk, c);
}

// Entries per list of each block of rows: block_sums[list * nb + block].
__global__ __launch_bounds__(kWlThreads) void worklist_count(const int* __restrict__ rowptr,
                                                             int64_t N, int chunk,
                                                             int* __restrict__ block_sums, int nb) {
  __shared__ int tmp[kLists * (kWlThreads / kWave)];
  int beg, deg, c[kLists], ex[kLists], tot[kLists];
  row_entries(rowptr, N, chunk, (int64_t)blockIdx.x * kWlThreads + threadIdx.x, &beg, &deg, c);
  block_excl_scan_lists<kWlThreads / kWave, kLists>(c, ex, tot, tmp);
  if (threadIdx.x == 0)
#pragma unroll
    for (int i = 0; i < kLists; ++i) block_sums[i * nb + blockIdx.x] = tot[i];
}

// One block: exclusive scan of each list's block sums in place; the list
// lengths go to the counters.
__global__ __launch_bounds__(1024) void worklist_offsets(int* __restrict__ block_sums, int nb,
                                                         int* __restrict__ counters) {
  __shared__ int tmp[1024 / kWave];
  for (int i = 0; i < kLists; ++i) {
    int* b = block_sums + (int64_t)i * nb;
    int carry = 0;
    for (int base = 0; base < nb; base += 1024) {
      const int k = base + (int)threadIdx.x;
      const int v = k < nb ? b[k] : 0;
      int total;
      const int ex = block_excl_scan<1024 / kWave>(v, tmp, &total);
      if (k < nb) b[k] = carry + ex;
      carry += total;
    }
    if (threadIdx.x == 0) counters[kListCounter[i]] = carry;
  }
}

// The three steps in one block, for graphs of at most kWlSingle rows: the
// rows go in chunks of kWlThreads, each chunk's entries placed after the
// previous chunks' (the same lists, in the same order).
constexpr int kWlSingle = 4 * kWlThreads;
__global__ __launch_bounds__(kWlThreads) void worklist_single(
    const int* __restrict__ rowptr, int64_t N, int chunk, int* __restrict__ counters,
    WorkItem* __restrict__ heavy, WorkItem* __restrict__ light, SplitRow* __restrict__ split,
    WorkItem* __restrict__ short_rows, WorkItem* __restrict__ long_rows) {
  __shared__ int tmp[kLists * (kWlThreads / kWave)];
  int carry[kLists] = {0, 0, 0, 0, 0};
  // every chunk's row pointers loaded before the first is used
  constexpr int kChunks = kWlSingle / kWlThreads;
  int rp[kChunks], rq[kChunks];
#pragma unroll
  for (int j = 0; j < kChunks; ++j) {
    const int64_t r = (int64_t)j * kWlThreads + threadIdx.x;
    rp[j] = r < N ? rowptr[r] : 0;
    rq[j] = r < N ? rowptr[r + 1] : 0;
  }
#pragma unroll
  for (int j = 0; j < kChunks; ++j) {
    if ((int64_t)j * kWlThreads >= N) break;  // uniform
    const int64_t r = (int64_t)j * kWlThreads + threadIdx.x;
    const int beg = rp[j], deg = rq[j] - rp[j];
    int c[kLists], o[kLists], tot[kLists];
    row_counts(r < N, deg, chunk, c);
    block_excl_scan_lists<kWlThreads / kWave, kLists>(c, o, tot, tmp);
#pragma unroll
    for (int i = 0; i < kLists; ++i) {
      o[i] += carry[i];
      carry[i] += tot[i];
    }
    if (r < N) {
      if (c[3])
        short_rows[o[3]] = WorkItem{(int)r, beg, beg + deg, -1};
      else if (c[4])
        long_rows[o[4]] = WorkItem{(int)r, beg, beg + deg, -1};
      if (c[2]) {
        for (int q = 0; q < c[0]; ++q) {
          const int kb = beg + q * chunk;
          heavy[o[0] + q] = WorkItem{(int)r, kb, min(kb + chunk, beg + deg), o[0] + q};
        }
        split[o[2]] = SplitRow{(int)r, o[0], c[0], deg};
      } else {
        light[o[1]] = WorkItem{(int)r, beg, beg + deg, -1};
      }
    }
  }
  if (threadIdx.x == 0)
#pragma unroll
    for (int i = 0; i < kLists; ++i) counters[kListCounter[i]] = carry[i];
}

__global__ __launch_bounds__(kWlThreads) void worklist_fill(
    const int* __restrict__ rowptr, int64_t N, int chunk, const int* __restrict__ block_sums,
    int nb, WorkItem* __restrict__ heavy, WorkItem* __restrict__ light,
    SplitRow* __restrict__ split, WorkItem* __restrict__ short_rows, WorkItem* __restrict__ long_rows) {
  __shared__ int tmp[kLists * (kWlThreads / kWave)];
  const int64_t r = (int64_t)blockIdx.x * kWlThreads + threadIdx.x;
  int beg, deg, c[kLists], o[kLists], tot[kLists];
  row_entries(rowptr, N, chunk, r, &beg, &deg, c);
  block_excl_scan_lists<kWlThreads / kWave, kLists>(c, o, tot, tmp);
#pragma unroll
  for (int i = 0; i < kLists; ++i) o[i] += block_sums[i * nb + blockIdx.x];
  if (r >= N) return;
  if (c[3])
    short_rows[o[3]] = WorkItem{(int)r, beg, beg + deg, -1};
  else if (c[4])
    long_rows[o[4]] = WorkItem{(int)r, beg, beg + deg, -1};
  if (c[2]) {
    const int h0 = o[0];
    for (int j = 0; j < c[0]; ++j) {
      const int kb = beg + j * chunk;
      heavy[h0 + j] = WorkItem{(int)r, kb, min(kb + chunk, beg + deg), h0 + j};
    }
    split[o[2]] = SplitRow{(int)r, h0, c[0], deg};
  } else {
    light[o[1]] = WorkItem{(int)r, beg, beg + deg, -1};
  }
}

__device__ __forceinline__ int chunks_of(int len, int chunk) { return (len + chunk - 1) / chunk; }

// Part plan, step 1: items per row (all parts) and per (part, row).
__global__ __launch_bounds__(kBlock) void part_counts(const int* __restrict__ segptr, int64_t N,
                                                      int parts, int chunk,
                                                      int* __restrict__ row_items,
                                                      int* __restrict__ seg_items) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= N) return;
  int tot = 0;
  for (int p = 0; p < parts; ++p) {
    const int len = segptr[t * parts + p + 1] - segptr[t * parts + p];
    const int c = chunks_of(len, chunk);
    seg_items[(int64_t)p * N + t] = c;
    tot += c;
  }
  row_items[t] = tot;
}

// Part plan, step 2: items in part-major order (part, row, chunk); the
// partial slots are numbered row-major so that row t's partials are the
// contiguous range [row_slot[t], row_slot[t+1]), in part order.
__global__ __launch_bounds__(kBlock) void part_fill(const int* __restrict__ segptr, int64_t N,
                                                    int parts, int chunk,
                                                    const int* __restrict__ row_slot,
                                                    const int* __restrict__ seg_pos,
                                                    WorkItem* __restrict__ exec,
                                                    SplitRow* __restrict__ rows) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= N) return;
  int slot = row_slot[t];
  const int s0 = slot;
  for (int p = 0; p < parts; ++p) {
    const int kb = segptr[t * parts + p], ke = segptr[t * parts + p + 1];
    int pos = seg_pos[(int64_t)p * N + t];
    for (int k = kb; k < ke; k += chunk) exec[pos++] = WorkItem{(int)t, k, min(k + chunk, ke), slot++};
  }
  rows[t] = SplitRow{(int)t, s0, slot - s0, segptr[(t + 1) * parts] - segptr[t * parts]};
}

int ceil_log2(int64_t n) {
  int b = 0;
  while ((int64_t(1) << b) < n) ++b;
  return b;
}

struct SortPlan {
  int bits, passes, dbits;
  int64_t ntiles, keyspace;
};

SortPlan sort_plan(int64_t E, int64_t N, int parts) {
  SortPlan p;
  p.keyspace = std::max<int64_t>(N * parts, 1);
  p.bits = std::max(1, ceil_log2(std::max<int64_t>(p.keyspace, 2)));
  p.passes = (p.bits + kMaxDigitBits - 1) / kMaxDigitBits;
  p.dbits = (p.bits + p.passes - 1) / p.passes;
  p.ntiles = (E + kSortTile - 1) / kSortTile;
  return p;
}

struct ScratchLayout {
  size_t hist, sums, bufA, bufB, wl_sums, row_items, seg_items, total;
};

ScratchLayout scratch_layout(int64_t E, int64_t N, int parts) {
  SortPlan p = sort_plan(E, N, parts);
  ScratchLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  const int64_t radix = int64_t(1) << p.dbits;
  const int64_t scan_n = std::max<int64_t>({N * parts + 1, N + 1, radix * p.ntiles});
  L.hist = take(sizeof(int) * std::max<int64_t>(radix * p.ntiles, 1));
  L.sums = take(sizeof(int) * std::max<int64_t>(scan_tiles(scan_n), 1));
  L.bufA = take(sizeof(int) * 3 * std::max<int64_t>(E, 1));
  L.bufB = take(p.passes >= 3 ? sizeof(int) * 3 * std::max<int64_t>(E, 1) : 0);
  L.wl_sums = take(sizeof(int) * kLists * std::max<int64_t>((N + kWlThreads - 1) / kWlThreads, 1));
  L.row_items = take(parts > 1 ? sizeof(int) * (N + 1) : 0);
  L.seg_items = take(parts > 1 ? sizeof(int) * (N * parts + 1) : 0);
  L.total = off;
  return L;
}

template <typename IdxT>
int sort_edges(Graph& g, const IdxT* src, const IdxT* tgt, char* scratch, const ScratchLayout& L,
               hipStream_t s) {
  const int64_t E = g.E;
  const SortPlan p = sort_plan(E, g.N, g.parts);
  const KeyMap m{g.E_in, g.N_src, g.N, (int)g.part_rows, g.parts, 1.0 / (double)g.part_rows,
                 0.5 / (double)g.part_rows};
  int* keys = g.key;  // the last pass leaves the sorted keys in the graph
  int* hist = reinterpret_cast<int*>(scratch + L.hist);
  int* sums = reinterpret_cast<int*>(scratch + L.sums);
  int* bufs[2][3];
  for (int b = 0; b < 2; ++b) {
    int* base = reinterpret_cast<int*>(scratch + (b == 0 ? L.bufA : L.bufB));
    for (int j = 0; j < 3; ++j) bufs[b][j] = base + j * E;
  }
  int* err = g.counters + 3;
  const unsigned nt = (unsigned)p.ntiles;
  const int radix = 1 << p.dbits;

  // packed payloads (scatter_packed): P a power of two, ids and positions in 64 bits
  const int lp = ceil_log2(g.parts);
  const int bt = ceil_log2(g.N), bs = ceil_log2(g.N_src), be = ceil_log2(E);
  const int sl = std::max(0, bs - (32 - bt));
  bool packed = p.passes >= 2 && (int64_t(1) << lp) == g.parts && bt >= 1 && bt <= 31 &&
                be <= 31 && sl + be <= 32 && p.dbits >= lp;
  if (const char* v = std::getenv("TFG_SORT_PACKED")) packed = packed && v[0] != '0';
  const PackMap q{bt, sl, be, lp};

  if (E > 0) {
    int cur = 0;  // which scratch buffer holds the current keys
    for (int pass = 0; pass < p.passes; ++pass) {
      const int shift = pass * p.dbits;
      const bool first = pass == 0, last = pass == p.passes - 1;
      // packed passes after the first find their digit in A
      const int dshift = (packed && !first) ? 32 - bt + shift - lp : shift;
      if (first)
        upsweep<true, IdxT><<<nt, kUpThreads, 0, s>>>(src, tgt, m, nullptr, E, shift, p.dbits,
                                                        hist, err);
      else
        upsweep<false, IdxT><<<nt, kUpThreads, 0, s>>>(src, tgt, m, bufs[cur][0], E, dshift,
                                                         p.dbits, hist, err);
      const int scanned = p.ntiles > kInBlockTiles;
      if (scanned) {
        const int rc = exclusive_scan(hist, hist, radix * p.ntiles, sums, s);
        if (rc) return rc;
        TFG_LAUNCHED("radix offsets");
      }
      const int nxt = first ? 0 : 1 - cur;
      int* ko = last ? keys : bufs[nxt][0];
      int* eo = last ? g.perm : bufs[nxt][1];
      int* so = last ? g.col : bufs[nxt][2];
      const int *ki = bufs[cur][0], *ei = bufs[cur][1], *si = bufs[cur][2];
      if (packed) {
        const unsigned* ai = reinterpret_cast<const unsigned*>(ki);
        const unsigned* bi = reinterpret_cast<const unsigned*>(ei);
        if (first)
          scatter_packed<0, IdxT><<<nt, kSortThreads, 0, s>>>(
              src, tgt, m, q, ai, bi, E, dshift, p.dbits, hist, (int)p.ntiles, scanned, ko, eo, so);
        else if (last)
          scatter_packed<2, IdxT><<<nt, kSortThreads, 0, s>>>(
              src, tgt, m, q, ai, bi, E, dshift, p.dbits, hist, (int)p.ntiles, scanned, ko, eo, so);
        else
          scatter_packed<1, IdxT><<<nt, kSortThreads, 0, s>>>(
              src, tgt, m, q, ai, bi, E, dshift, p.dbits, hist, (int)p.ntiles, scanned, ko, eo, so);
      } else if (first) {
        scatter<true, IdxT><<<nt, kSortThreads, 0, s>>>(src, tgt, m, ki, ei, si, E, shift, p.dbits,
                                                        hist, (int)p.ntiles, scanned, ko, eo, so);
      } else {
        scatter<false, IdxT><<<nt, kSortThreads, 0, s>>>(src, tgt, m, ki, ei, si, E, shift,
                                                         p.dbits, hist, (int)p.ntiles, scanned, ko,
                                                         eo, so);
      }
      TFG_LAUNCHED("radix scatter");
      cur = nxt;
    }
  }
  // segment starts from the boundaries of the sorted keys
  const int64_t K = g.N * g.parts;
  const int64_t kb_per_block = (int64_t)kKbThreads * kKbGroups;  // groups of four positions
  key_bounds<<<dim3((unsigned)((E / 4 + 1 + kb_per_block - 1) / kb_per_block)), dim3(kKbThreads), 0, s>>>(
      keys, E, K, g.segptr);
  TFG_LAUNCHED("key_bounds");
  if (g.parts > 1) {
    rows_from_segments<<<dim3((unsigned)((g.N + 1 + kBlock - 1) / kBlock)), dim3(kBlock), 0, s>>>(
        g.segptr, g.N, g.parts, g.rowptr);
    TFG_LAUNCHED("rows_from_segments");
  }
  return TFG_OK;
}

int build_part_plan(Graph& g, char* scratch, const ScratchLayout& L, hipStream_t s) {
  int* row_items = reinterpret_cast<int*>(scratch + L.row_items);
  int* seg_items = reinterpret_cast<int*>(scratch + L.seg_items);
  int* sums = reinterpret_cast<int*>(scratch + L.sums);
  const unsigned nb = (unsigned)((g.N + kBlock - 1) / kBlock);
  const int64_t NP = g.N * g.parts;
  fill_int<<<1, 64, 0, s>>>(row_items + g.N, 1, 0);
  fill_int<<<1, 64, 0, s>>>(seg_items + NP, 1, 0);
  part_counts<<<nb, kBlock, 0, s>>>(g.segptr, g.N, g.parts, g.chunk, row_items, seg_items);
  TFG_LAUNCHED("part_counts");
  int rc = exclusive_scan(row_items, row_items, g.N + 1, sums, s);
  if (rc) return rc;
  rc = exclusive_scan(seg_items, seg_items, NP + 1, sums, s);
  if (rc) return rc;
  part_fill<<<nb, kBlock, 0, s>>>(g.segptr, g.N, g.parts, g.chunk, row_items, seg_items, g.pexec,
                                  g.prows);
  TFG_LAUNCHED("part_fill");
  // the number of items, read back with the other counters
  TFG_HIP(hipMemcpyAsync(g.counters + 4, seg_items + NP, sizeof(int), hipMemcpyDeviceToDevice, s));
  return TFG_OK;
}

}  // namespace

int64_t exclusive_scan_sums(int64_t n) { return std::max<int64_t>(scan_tiles(n), 1); }

int exclusive_scan(const int* in, int* out, int64_t n, int* tile_sums, hipStream_t s) {
  if (n <= 0) return TFG_OK;
  if (in == out && n <= kSmallScan) {
    scan_small<<<1, 1024, 0, s>>>(out, n);
    TFG_LAUNCHED("exclusive scan (one block)");
    return TFG_OK;
  }
  const int64_t nt = scan_tiles(n);
  scan_tile_sums<<<dim3((unsigned)nt), dim3(kScanThreads), 0, s>>>(in, n, tile_sums);
  scan_sums<<<1, 1024, 0, s>>>(tile_sums, nt);
  scan_apply<<<dim3((unsigned)nt), dim3(kScanThreads), 0, s>>>(in, out, n, tile_sums);
  TFG_LAUNCHED("exclusive scan");
  return TFG_OK;
}

// Eight ints of pinned host memory per calling thread (portable: usable with
// any device's stream), allocated on first use and kept for the life of the
// process, for the few counters that the synchronising calls read back: a
// copy into pinned memory goes straight to the host, without the runtime's
// staging copy (a graph build of 13,264 edges: 0.165 -> 0.137 ms). NULL if
// the allocation fails (the caller then reads into pageable memory).
int* readback_buffer() {
  thread_local int* p = [] {
    void* q = nullptr;
    return hipHostMalloc(&q, sizeof(int) * 8, hipHostMallocPortable) == hipSuccess
               ? static_cast<int*>(q)
               : nullptr;
  }();
  return p;
}

int default_chunk() {
  static const int chunk = [] {
    const char* v = std::getenv("TFG_ROW_CHUNK");
    const int c = v ? std::atoi(v) : kDefaultChunk;
    return c >= 64 && c <= kMaxChunk ? c : kDefaultChunk;
  }();
  return chunk;
}

int choose_parts(int64_t E, int64_t N, int64_t N_src, int requested) {
  int P = 1;
  if (requested >= 1) {
    P = std::min(requested, kMaxParts);
  } else {
    // 512-byte rows (128 float32 features) as the nominal gathered row size
    const double table = (double)N_src * 512.0;
    const double avg_deg = N > 0 ? (double)E / (double)N : 0.0;
    if (table >= 32.0 * (1 << 20)) {
      P = (int)std::min<double>(kMaxParts, std::ceil(table / (16.0 * (1 << 20))));
      P = std::min<int>(P, (int)(avg_deg / 16.0));  // keep (row, part) segments long
    }
  }
  P = (int)std::min<int64_t>(P, std::max<int64_t>(N_src, 1));
  if (P < 1 || N * (int64_t)P >= (int64_t(1) << 31) - 1) P = 1;
  return P;
}

GraphLayout graph_layout(int64_t E, int64_t N, int parts, int chunk) {
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
  // part plan: one item per nonempty (row, part) segment, plus one per
  // further chunk of a long segment
  L.cap_pexec = parts > 1 ? std::min<int64_t>(E, N * parts) + E / chunk + 1 : 0;
  L.rowptr = take(sizeof(int) * (N + 1));
  L.segptr = take(parts > 1 ? sizeof(int) * (N * parts + 1) : 0);
  L.col = take(sizeof(int) * std::max<int64_t>(E, 1));
  L.perm = take(sizeof(int) * std::max<int64_t>(E, 1));
  L.key = take(sizeof(int) * std::max<int64_t>(E, 1));
  L.heavy = take(sizeof(WorkItem) * L.cap_heavy);
  L.light = take(sizeof(WorkItem) * std::max<int64_t>(L.cap_light, 1));
  L.split = take(sizeof(SplitRow) * std::max<int64_t>(L.cap_split, 1));
  L.pexec = take(sizeof(WorkItem) * L.cap_pexec);
  L.prows = take(parts > 1 ? sizeof(SplitRow) * N : 0);
  L.short_rows = take(sizeof(WorkItem) * std::max<int64_t>(N, 1));
  L.long_rows = take(sizeof(WorkItem) * std::max<int64_t>(N, 1));
  L.counters = take(sizeof(int) * 8);
  L.total = off;
  return L;
}

size_t graph_scratch_bytes(int64_t E, int64_t N, int parts) {
  return scratch_layout(E, N, parts).total;
}

int build_graph(Graph& g, const void* src, const void* tgt, int index_type, void* scratch,
                size_t scratch_bytes, hipStream_t s) {
  const ScratchLayout L = scratch_layout(g.E, g.N, g.parts);
  if (scratch_bytes < L.total) return fail(TFG_ERR_WORKSPACE, "graph scratch buffer too small");
  char* sc = static_cast<char*>(scratch);
  fill_int<<<1, 64, 0, s>>>(g.counters, 8, 0);
  int rc;
  if (index_type == TFG_I64)
    rc = sort_edges<int64_t>(g, static_cast<const int64_t*>(src), static_cast<const int64_t*>(tgt),
                             sc, L, s);
  else
    rc = sort_edges<int32_t>(g, static_cast<const int32_t*>(src), static_cast<const int32_t*>(tgt),
                             sc, L, s);
  if (rc) return rc;
  if (g.N > 0) {
    const int nb = (int)((g.N + kWlThreads - 1) / kWlThreads);
    int* wl = reinterpret_cast<int*>(sc + L.wl_sums);
    if (g.N <= kWlSingle) {
      worklist_single<<<1, kWlThreads, 0, s>>>(g.rowptr, g.N, g.chunk, g.counters, g.heavy,
                                               g.light, g.split, g.short_rows, g.long_rows);
    } else {
      worklist_count<<<nb, kWlThreads, 0, s>>>(g.rowptr, g.N, g.chunk, wl, nb);
      worklist_offsets<<<1, 1024, 0, s>>>(wl, nb, g.counters);
      worklist_fill<<<nb, kWlThreads, 0, s>>>(g.rowptr, g.N, g.chunk, wl, nb, g.heavy, g.light,
                                              g.split, g.short_rows, g.long_rows);
    }
    TFG_LAUNCHED("work lists");
    if (g.parts > 1) {
      rc = build_part_plan(g, sc, L, s);
      if (rc) return rc;
    }
  }
  int stack_host[8];
  int* pin = readback_buffer();
  int* host = pin ? pin : stack_host;
  TFG_HIP(hipMemcpyAsync(host, g.counters, sizeof(int) * 8, hipMemcpyDeviceToHost, s));
  TFG_HIP(hipStreamSynchronize(s));
  if (host[3] & kErrIndex) return fail(TFG_ERR_INDEX_RANGE, "edge_index holds an id outside [0, N)");
  g.n_heavy = host[0];
  g.n_light = host[1];
  g.n_split = host[2];
  g.n_pexec = host[4];
  g.n_short = host[5];
  g.n_long = host[6];
  return TFG_OK;
}

}  // namespace tfg
