// GCN normalisation on the CSR-by-target graph (gfx950): the propagation
// matrix of GCN (Sec. 2.2), computed once per graph and cached (Sec. 3):
//   deg[t]  = sum of the weights entering t (loops included when appended)
//   dinv[t] = deg > 0 ? 1 / sqrt(deg) : 0         (IEEE sqrt, IEEE divide)
//   w'[e]   = (dinv[src] * w[e]) * dinv[tgt]       (float32, left to right)
// written in the caller's COO order and/or in the graph's CSR order; both
// orders use the same operands in the same order, so they are bit-identical.
#include <algorithm>
#include <cstdlib>

#include "wave.h"

namespace tfg {
namespace {

// Weight of edge id e in the list with appended loops.
__device__ __forceinline__ float edge_w(const float* __restrict__ w, int64_t E_in, int64_t e) {
  return (w == nullptr || e >= E_in) ? 1.0f : w[e];
}

// Unit weights: the degree is the row length (exact in float32 below 2^24,
// and rounded once above it).
__global__ __launch_bounds__(kBlock) void degree_unit(const int* __restrict__ rowptr, int64_t N,
                                                      float* __restrict__ deg,
                                                      float* __restrict__ dinv) {
  int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= N) return;
  float d = (float)(rowptr[t + 1] - rowptr[t]);
  if (deg) deg[t] = d;
  dinv[t] = d > 0.0f ? 1.0f / sqrtf(d) : 0.0f;
}

// General weights: one wavefront per row, each lane summing a strided part of
// the row in double, then a fixed-order tree across the lanes.
__global__ __launch_bounds__(kItemBlock) void degree_weighted(const int* __restrict__ rowptr,
                                                          const int* __restrict__ perm,
                                                          const float* __restrict__ w,
                                                          int64_t E_in, int64_t N,
                                                          float* __restrict__ deg,
                                                          float* __restrict__ dinv) {
  const int64_t t = (int64_t)blockIdx.x * (kItemBlock / kWave) + threadIdx.x / kWave;
  if (t >= N) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int kb = uniform(rowptr[t]), ke = uniform(rowptr[t + 1]);
  double acc = 0.0;
  for (int k = kb + lane; k < ke; k += kWave) acc += (double)edge_w(w, E_in, perm[k]);
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) {
    float d = (float)acc;
    if (deg) deg[t] = d;
    dinv[t] = d > 0.0f ? 1.0f / sqrtf(d) : 0.0f;
  }
}

// CSR order, one position per thread (four per thread, strided by the block):
// the target comes from the stored sort key (target * parts + part), so the
// source's and the target's dinv are gathered side by side, with no work list.
template <bool HAS_W>
__global__ __launch_bounds__(kBlock) void weights_csr(const int* __restrict__ key, int parts,
                                                      const int* __restrict__ col,
                                                      const int* __restrict__ perm,
                                                      const float* __restrict__ w, int64_t E_in,
                                                      int64_t E, const float* __restrict__ dinv,
                                                      float* __restrict__ out) {
  const int64_t b = (int64_t)blockIdx.x * (4 * kBlock) + threadIdx.x;
  int c[4], t[4], e[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t k = b + j * kBlock;
    const bool ok = k < E;
    c[j] = ok ? col[k] : 0;
    t[j] = ok ? key[k] : 0;
    e[j] = (HAS_W && ok) ? perm[k] : 0;
  }
  float we[4], ds[4], dt[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    we[j] = HAS_W ? edge_w(w, E_in, e[j]) : 1.0f;
    ds[j] = dinv[c[j]];
    dt[j] = dinv[parts == 1 ? t[j] : t[j] / parts];
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t k = b + j * kBlock;
    if (k < E) out[k] = (ds[j] * we[j]) * dt[j];  // (dinv[s] * w) * dinv[t]
  }
}

// COO order (input edges, then loops), optionally writing the edge list; four
// edges per thread, strided by the block size, loads issued together.
template <typename IdxT>
__global__ __launch_bounds__(kBlock) void weights_coo(const IdxT* __restrict__ src,
                                                      const IdxT* __restrict__ tgt, int64_t E_in,
                                                      int64_t E, int64_t N,
                                                      const float* __restrict__ w,
                                                      const float* __restrict__ dinv,
                                                      int32_t* __restrict__ out_ei,
                                                      float* __restrict__ out_w) {
  const int64_t base = (int64_t)blockIdx.x * (4 * kBlock) + threadIdx.x;
  int s[4], t[4];
  float we[4], ds[4], dt[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t e = base + j * kBlock;
    const int64_t ec = e < E_in ? e : (E_in > 0 ? E_in - 1 : 0);
    const int64_t sv = E_in > 0 ? (int64_t)__builtin_nontemporal_load(src + ec) : 0;
    const int64_t tv = E_in > 0 ? (int64_t)__builtin_nontemporal_load(tgt + ec) : 0;
    const bool in = e < E_in;
    // ids were validated when the graph was built; clamped here all the same
    s[j] = in ? ((sv < 0 || sv >= N) ? 0 : (int)sv) : (int)(e - E_in);
    t[j] = in ? ((tv < 0 || tv >= N) ? 0 : (int)tv) : (int)(e - E_in);
    we[j] = (w != nullptr && in) ? w[ec] : 1.0f;
  }
  if (out_w) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool ok = base + j * kBlock < E;
      ds[j] = ok ? dinv[s[j]] : 0.0f;
      dt[j] = ok ? dinv[t[j]] : 0.0f;
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t e = base + j * kBlock;
    if (e >= E) break;
    if (out_ei) {
      __builtin_nontemporal_store(s[j], out_ei + e);
      __builtin_nontemporal_store(t[j], out_ei + E + e);
    }
    if (out_w) {
      const float a = ds[j] * we[j];
      __builtin_nontemporal_store(a * dt[j], out_w + e);
    }
  }
}

// dinv from LDS instead of L2. Gathering one float per endpoint from L2 moves
// a whole cache line per lane, and that line traffic, not HBM, bounds the two
// kernels above. Here a block keeps the node ids of its edges in registers and
// walks dinv in slices that fit in LDS; each endpoint picks up its value in
// the slice that holds it. Every block reads all of dinv once (4 N bytes from
// L2 in full lines, copied straight into LDS) in exchange for one or two
// random line reads per edge, so the tile per block is made as large as the
// registers allow: one register per endpoint, holding the node id until the
// endpoint's slice is seen and then its dinv value. The products are the same
// ones, in the same order, as in weights_coo / weights_csr, so the kernels
// agree bit for bit.
constexpr int kSlThreads = 1024;                  // 16 waves, one block per CU
constexpr int kSlPiece = kWave * 4;               // floats per wave-wide 16-byte copy
constexpr int kSlice = 159 * kSlPiece;            // floats per LDS slice (159 KB)
constexpr int kSlLds = kSlice + kSlPiece;         // the slice, then the sentinel word
// edges per thread in COO order (2 registers each; 64-bit ids and weights
// need registers of their own)
template <typename IdxT, bool HAS_W>
constexpr int coo_items() { return sizeof(IdxT) == 4 && !HAS_W ? 28 : 24; }
constexpr int kCooTile = kSlThreads * coo_items<int32_t, false>();  // 28672 edges per block
// positions per thread in graph order (1 register each; general weights need
// registers for their edge ids and weights)
template <bool HAS_W>
constexpr int csr_items() { return HAS_W ? 24 : 32; }

typedef __attribute__((address_space(3))) void* lds_ptr;

// Starts copying d[0, len) (16-byte aligned) into slice: whole 1 KB pieces as
// direct memory-to-LDS loads (lane l of a wave moves bytes 16 l .. 16 l + 15
// of a piece), the remainder through registers. The caller waits for the
// copies (wait_slice) before the barrier that publishes the slice.
__device__ __forceinline__ void fill_slice(float* slice, const float* __restrict__ d, int len) {
  const int lane = lane_id();
  const int wave = uniform((int)threadIdx.x / kWave);
  const int pieces = len / kSlPiece;
  for (int c = wave; c < pieces; c += kSlThreads / kWave)
    __builtin_amdgcn_global_load_lds(d + c * kSlPiece + lane * 4, (lds_ptr)(slice + c * kSlPiece),
                                     16, 0, 0);
  for (int i = pieces * kSlPiece + (int)threadIdx.x; i < len; i += kSlThreads) slice[i] = d[i];
}

// All of this wave's memory operations done (the LDS copies included).
__device__ __forceinline__ void wait_slice() { __builtin_amdgcn_s_waitcnt(0); }

// An endpoint register, as unsigned: 0x80000000 | (4 * node id) until it is
// resolved (0xFFFFFFFC for no edge, which no slice holds), then the bits of
// its dinv value, which are below 0x80000000 (dinv >= 0). The word after the
// slice holds the sentinel 0xFFFFFFFF. For the slice of nodes [lo, lo + len)
// a register's offset is u = r - (0x80000000 + 4 lo): below 4 len for an id
// in the slice, and at least 4 kSlice for every other register (a later id,
// a resolved value, no edge; earlier ids were resolved by earlier slices;
// N <= 2^28). So min(u, 4 kSlice) addresses either the value or the sentinel,
// and min(r, word read) resolves the register or leaves it as it was: three
// ALU operations and one LDS read per register and slice, with no branch.
__device__ __forceinline__ unsigned unresolved(int id) { return 0x80000000u | (4u * (unsigned)id); }
__device__ __forceinline__ float value_of(unsigned r) { return __uint_as_float(r); }
__device__ __forceinline__ void put_sentinel(float* slice) {
  if (threadIdx.x == 0) reinterpret_cast<unsigned*>(slice)[kSlice] = 0xFFFFFFFFu;
}

template <int ITEMS>
__device__ __forceinline__ void resolve(unsigned (&r)[ITEMS], const float* slice, int64_t lo) {
  const char* sb = reinterpret_cast<const char*>(slice);
  const unsigned b = 0x80000000u + 4u * (unsigned)lo;
#pragma unroll
  for (int j = 0; j < ITEMS; ++j) {
    const unsigned a = min(r[j] - b, 4u * (unsigned)kSlice);
    r[j] = min(r[j], *reinterpret_cast<const unsigned*>(sb + a));
  }
}

// Walks dinv[0, N) slice by slice, resolving every register of the block.
// The first slice and the sentinel were started (fill_slice, put_sentinel) by
// the caller.
template <int ITEMS>
__device__ __forceinline__ void walk_slices(unsigned (&r)[ITEMS], float* slice,
                                            const float* __restrict__ dinv, int64_t N) {
  for (int64_t lo = 0; lo < N; lo += kSlice) {
    const int len = (int)min<int64_t>(kSlice, N - lo);
    if (lo > 0) {
      __syncthreads();  // the previous slice is no longer read
      fill_slice(slice, dinv + lo, len);
    }
    wait_slice();
    __syncthreads();
    resolve(r, slice, lo);
  }
}

// (Block-relative pointers with 32-bit offsets keep one address register per
// thread for all items. The weights are a template choice: a run-time branch
// on them costs the unweighted kernel 13% in spilled scalar registers.)
template <typename IdxT, bool HAS_W>
__global__ __launch_bounds__(kSlThreads, 4) void weights_coo_sliced(
    const IdxT* __restrict__ src, const IdxT* __restrict__ tgt, int64_t E_in, int64_t E, int64_t N,
    const float* __restrict__ w, const float* __restrict__ dinv, int32_t* __restrict__ out_ei,
    float* __restrict__ out_w) {
  constexpr int kCooItems = coo_items<IdxT, HAS_W>();
  constexpr int kTile = kSlThreads * kCooItems;
  __shared__ float slice[kSlLds];
  fill_slice(slice, dinv, (int)min<int64_t>(kSlice, N));  // overlaps the edge loads
  put_sentinel(slice);
  const int64_t b0 = (int64_t)blockIdx.x * kTile;
  const int n_in = (int)max<int64_t>(0, min<int64_t>(kTile, E_in - b0));  // input edges here
  const int n_all = (int)min<int64_t>(kTile, E - b0);                     // with the loops
  // [0, ITEMS): sources, [ITEMS, 2 ITEMS): targets. 32-bit ids are loaded
  // straight into these registers (every load issued before the first use);
  // 64-bit ids go through groups of 8 edges.
  unsigned st[2 * kCooItems];
  const IdxT* sb = src + b0;
  const IdxT* tb = tgt + b0;
  constexpr int G = sizeof(IdxT) == 4 ? kCooItems : 8;
#pragma unroll
  for (int j0 = 0; j0 < kCooItems; j0 += G) {
    IdxT rs[sizeof(IdxT) == 4 ? 1 : G], rt[sizeof(IdxT) == 4 ? 1 : G];
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const int p = (j0 + j) * kSlThreads + (int)threadIdx.x;
      const IdxT a = p < n_in ? __builtin_nontemporal_load(sb + p) : IdxT(0);
      const IdxT b = p < n_in ? __builtin_nontemporal_load(tb + p) : IdxT(0);
      if constexpr (sizeof(IdxT) == 4) {
        st[j0 + j] = (unsigned)a;
        st[kCooItems + j0 + j] = (unsigned)b;
      } else {
        rs[j] = a;
        rt[j] = b;
      }
    }
    if constexpr (sizeof(IdxT) != 4) {
      // ids out of the 32-bit range become N (clamped below)
#pragma unroll
      for (int j = 0; j < G; ++j) {
        st[j0 + j] = (rs[j] < 0 || rs[j] >= N) ? (unsigned)N : (unsigned)rs[j];
        st[kCooItems + j0 + j] = (rt[j] < 0 || rt[j] >= N) ? (unsigned)N : (unsigned)rt[j];
      }
    }
  }
  int32_t* os = out_ei == nullptr ? nullptr : out_ei + b0;
  int32_t* ot = out_ei == nullptr ? nullptr : out_ei + E + b0;
#pragma unroll
  for (int j = 0; j < kCooItems; ++j) {
    // ids were validated when the graph was built; clamped here all the same
    // (as unsigned, so that negative ids are caught too). Loops (i, i) follow
    // the input edges; positions past E get no edge.
    const int p = j * kSlThreads + (int)threadIdx.x;
    const bool in = p < n_in;
    const int loop = (int)(b0 + p - E_in);
    const int sv = in ? (st[j] >= (unsigned)N ? 0 : (int)st[j]) : loop;
    const int tv = in ? (st[kCooItems + j] >= (unsigned)N ? 0 : (int)st[kCooItems + j]) : loop;
    if (os != nullptr && p < n_all) {
      __builtin_nontemporal_store(sv, os + p);
      __builtin_nontemporal_store(tv, ot + p);
    }
    st[j] = p < n_all ? unresolved(sv) : unresolved(-1);
    st[kCooItems + j] = p < n_all ? unresolved(tv) : unresolved(-1);
  }
  walk_slices(st, slice, dinv, N);
  // all loads (the weights) before the first store: a wait for a load also
  // waits for the stores issued before it
  float* ow = out_w + b0;
  float o[kCooItems];
  if constexpr (HAS_W) {
    const float* wb = w + b0;
#pragma unroll
    for (int j = 0; j < kCooItems; ++j)  // loops weigh 1
      o[j] = j * kSlThreads + (int)threadIdx.x < n_in ? wb[j * kSlThreads + threadIdx.x] : 1.0f;
  } else {
#pragma unroll
    for (int j = 0; j < kCooItems; ++j) o[j] = 1.0f;
  }
#pragma unroll
  for (int j = 0; j < kCooItems; ++j)
    o[j] = (value_of(st[j]) * o[j]) * value_of(st[kCooItems + j]);  // (dinv[s] * w) * dinv[t]
#pragma unroll
  for (int j = 0; j < kCooItems; ++j) {
    const int p = j * kSlThreads + (int)threadIdx.x;
    if (p < n_all) __builtin_nontemporal_store(o[j], ow + p);
  }
}

// CSR order: blocks take kCsrTile consecutive positions and only the source
// side goes through the slices; the target of a position comes from its sort
// key (target * parts + part) at the end, and neighbouring positions share it,
// so dinv[target] is read directly, as are the weights.
template <bool HAS_W>
__global__ __launch_bounds__(kSlThreads, 4) void weights_csr_sliced(
    const int* __restrict__ key, int parts, const int* __restrict__ col,
    const int* __restrict__ perm, const float* __restrict__ w, int64_t E_in, int64_t E, int64_t N,
    const float* __restrict__ dinv, float* __restrict__ out) {
  constexpr int kCsrItems = csr_items<HAS_W>();
  constexpr int kCsrTile = kSlThreads * kCsrItems;
  __shared__ float slice[kSlLds];
  fill_slice(slice, dinv, (int)min<int64_t>(kSlice, N));
  put_sentinel(slice);
  const int64_t b0 = (int64_t)blockIdx.x * kCsrTile;
  const int n = (int)min<int64_t>(kCsrTile, E - b0);
  unsigned c[kCsrItems];
  {
    const int* cb = col + b0;
#pragma unroll
    for (int j = 0; j < kCsrItems; ++j) {
      const int p = j * kSlThreads + (int)threadIdx.x;
      c[j] = unresolved(p < n ? cb[p] : -1);
    }
  }
  walk_slices(c, slice, dinv, N);
  // The sources' values replace their registers; then the weights (edge ids
  // first, in groups), the keys and the targets' dinv: all loads before the
  // first store, since a wait for a load also waits for the stores issued
  // before it.
  float o[kCsrItems];
#pragma unroll
  for (int j = 0; j < kCsrItems; ++j) o[j] = value_of(c[j]);
  if constexpr (HAS_W) {  // dinv[col] * w (loops weigh 1)
    const int* pb = perm + b0;
#pragma unroll
    for (int j0 = 0; j0 < kCsrItems; j0 += 8) {
      int pe[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int p = (j0 + j) * kSlThreads + (int)threadIdx.x;
        pe[j] = p < n ? pb[p] : (int)E_in;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j0 + j] = o[j0 + j] * (pe[j] < E_in ? w[pe[j]] : 1.0f);
    }
  }
  // (unit weights: dinv[col] * 1 is dinv[col] itself)
  const int* kb = key + b0;
  float* ob = out + b0;
  int kv[kCsrItems];
#pragma unroll
  for (int j = 0; j < kCsrItems; ++j)
    kv[j] = j * kSlThreads + (int)threadIdx.x < n ? kb[j * kSlThreads + threadIdx.x] : 0;
  float dt[kCsrItems];
#pragma unroll
  for (int j = 0; j < kCsrItems; ++j) dt[j] = dinv[parts == 1 ? kv[j] : kv[j] / parts];
#pragma unroll
  for (int j = 0; j < kCsrItems; ++j) {
    const int p = j * kSlThreads + (int)threadIdx.x;
    if (p < n) ob[p] = o[j] * dt[j];  // (dinv[col] * w) * dinv[row]
  }
}

// Graph order over the part plan's items (unit weights). The items come part
// by part and the sources of a (row, part) item all lie in that part's node
// range. A block takes a contiguous run of items (one block per CU, in chunks
// of kPartItems), copies a part's range of dinv into LDS when its items reach
// that part (once, or twice where the run straddles two parts) and every
// position reads its source's value there: one copy of a part per block
// instead of a walk over all of dinv.
// A position is written in the round of its source's part only, so exactly
// once. Same products as weights_coo, in the same order.
constexpr int kPartItems = 512;             // items per chunk (descriptors in LDS)
constexpr int kPartU = 8;                   // items in flight per wavefront
constexpr int kPartSlice = 36864;           // floats of LDS for one part (144 KB)
constexpr int kPartBlocks = 256;            // blocks: one per CU

__global__ __launch_bounds__(kSlThreads) void weights_csr_parts(
    const WorkItem* __restrict__ items, int n_items, int per_block, int part_rows,
    const int* __restrict__ col, int64_t N, const float* __restrict__ dinv,
    float* __restrict__ out) {
  __shared__ float slice[kPartSlice];
  __shared__ int4 it[kPartItems];  // (row, kbeg, kend, -) of the current chunk of items
  __shared__ int prange[2];
  const int ib = blockIdx.x * per_block;
  const int ie = min(ib + per_block, n_items);
  const int wave = uniform((int)threadIdx.x / kWave), lane = lane_id();
  int loaded = -1;  // the part whose range the slice holds (the same in every thread)
  for (int c0 = ib; c0 < ie; c0 += kPartItems) {
    const int ni = min(kPartItems, ie - c0);
    __syncthreads();  // the previous chunk's items and part range are no longer read
    for (int j = threadIdx.x; j < ni; j += kSlThreads) {
      const WorkItem w = items[c0 + j];
      it[j] = make_int4(w.row, w.kbeg, w.kend, 0);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      // parts of the chunk's first and last item (items are part-major)
      prange[0] = col[it[0].y] / part_rows;
      prange[1] = col[it[ni - 1].y] / part_rows;
    }
    __syncthreads();
    const int p0 = prange[0], p1 = prange[1];
    for (int p = p0; p <= p1; ++p) {
      // part p holds sources [base, base + cnt); the copy starts 16-byte aligned
      const int64_t base = (int64_t)p * part_rows;
      const int cnt = (int)min<int64_t>(part_rows, N - base);
      const int64_t lo = base & ~int64_t(3);
      const int off = (int)(base - lo);
      if (p != loaded) {
        __syncthreads();  // the previous range is no longer read
        fill_slice(slice, dinv + lo, cnt + off);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        loaded = p;
      }
      for (int jb = wave * kPartU; jb < ni; jb += (kSlThreads / kWave) * kPartU) {
        int kb[kPartU], ke[kPartU], c[kPartU][2];
        float dt[kPartU];
#pragma unroll
        for (int u = 0; u < kPartU; ++u) {
          const bool ok = jb + u < ni;
          const int4 d = it[ok ? jb + u : 0];
          kb[u] = ok ? d.y : 0;
          ke[u] = ok ? d.z : 0;
          dt[u] = ok ? dinv[d.x] : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < kPartU; ++u)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int k = kb[u] + h * kWave + lane;
            c[u][h] = k < ke[u] ? col[k] : -1;
          }
#pragma unroll
        for (int u = 0; u < kPartU; ++u) {
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int k = kb[u] + h * kWave + lane;
            const unsigned q = (unsigned)(c[u][h] - (int)base);
            if (k < ke[u] && q < (unsigned)cnt) out[k] = (slice[off + q] * 1.0f) * dt[u];
          }
          // items longer than two rounds of lanes (a row-chunk setting above 128)
          for (int k = kb[u] + 2 * kWave + lane; k < ke[u]; k += kWave) {
            const unsigned q = (unsigned)(col[k] - (int)base);
            if (q < (unsigned)cnt) out[k] = (slice[off + q] * 1.0f) * dt[u];
          }
        }
      }
    }
  }
}

// The sliced kernels pay 4 N bytes of L2 reads per block against one or two
// gathered lines per edge; they are chosen while that fill stays below one
// line per edge and the grid still covers the chip.
bool use_sliced(int64_t E, int64_t N) {
  if (N > (int64_t(1) << 28)) return false;  // see resolved()
  if (const char* v = std::getenv("TFG_NORM_SLICED")) return v[0] == '1';
  return N * 4 <= (int64_t)kCooTile * 128 && E >= (int64_t)256 * kCooTile;
}

// Graph order by source part: a part plan whose items cover the graph and a
// part range that fits the LDS copy (with its alignment slack).
bool use_part_ranges(const Graph& g) {
  if (g.parts <= 1 || g.n_pexec <= 0 || g.part_rows + 3 > kPartSlice) return false;
  if (const char* v = std::getenv("TFG_NORM_PARTS")) return v[0] == '1';
  return use_sliced(g.E, g.N);
}

}  // namespace

int launch_gcn_norm(const Graph& g, const void* edge_index, int index_type,
                    const float* edge_weight, int32_t* out_edge_index, float* out_w,
                    float* out_w_csr, float* out_deg, float* dinv, hipStream_t s) {
  if (g.N == 0) return TFG_OK;
  const unsigned nb_rows = (unsigned)((g.N + kBlock - 1) / kBlock);
  if (edge_weight == nullptr) {
    degree_unit<<<nb_rows, kBlock, 0, s>>>(g.rowptr, g.N, out_deg, dinv);
  } else {
    degree_weighted<<<(unsigned)((g.N + (kItemBlock / kWave) - 1) / (kItemBlock / kWave)), kItemBlock, 0, s>>>(
        g.rowptr, g.perm, edge_weight, g.E_in, g.N, out_deg, dinv);
  }
  TFG_LAUNCHED("gcn degree");
  if (out_w_csr && g.E > 0 && edge_weight == nullptr && use_part_ranges(g)) {
    // one block per CU, each over a contiguous run of items (at most two part
    // ranges to copy), or blocks of kPartItems items on small graphs
    const int per_block = std::max(kPartItems, (g.n_pexec + kPartBlocks - 1) / kPartBlocks);
    weights_csr_parts<<<(unsigned)((g.n_pexec + per_block - 1) / per_block), kSlThreads, 0, s>>>(
        g.pexec, g.n_pexec, per_block, (int)g.part_rows, g.col, g.N, dinv, out_w_csr);
    TFG_LAUNCHED("gcn weights (graph order, by source part)");
  } else if (out_w_csr && g.E > 0 && use_sliced(g.E, g.N)) {
    if (edge_weight) {
      constexpr int64_t tile = kSlThreads * csr_items<true>();
      weights_csr_sliced<true><<<(unsigned)((g.E + tile - 1) / tile), kSlThreads, 0, s>>>(
          g.key, g.parts, g.col, g.perm, edge_weight, g.E_in, g.E, g.N, dinv, out_w_csr);
    } else {
      constexpr int64_t tile = kSlThreads * csr_items<false>();
      weights_csr_sliced<false><<<(unsigned)((g.E + tile - 1) / tile), kSlThreads, 0, s>>>(
          g.key, g.parts, g.col, g.perm, nullptr, g.E_in, g.E, g.N, dinv, out_w_csr);
    }
    TFG_LAUNCHED("gcn weights (CSR order, sliced)");
  } else if (out_w_csr && g.E > 0) {
    const unsigned nb = (unsigned)((g.E + 4 * kBlock - 1) / (4 * kBlock));
    if (edge_weight)
      weights_csr<true><<<nb, kBlock, 0, s>>>(g.key, g.parts, g.col, g.perm, edge_weight, g.E_in,
                                              g.E, dinv, out_w_csr);
    else
      weights_csr<false><<<nb, kBlock, 0, s>>>(g.key, g.parts, g.col, g.perm, nullptr, g.E_in,
                                               g.E, dinv, out_w_csr);
    TFG_LAUNCHED("gcn weights (CSR order)");
  }
  if ((out_w || out_edge_index) && g.E > 0) {
    if (out_w && use_sliced(g.E, g.N)) {
      auto blocks = [&](int items) { return (unsigned)((g.E + kSlThreads * items - 1) / (kSlThreads * items)); };
      if (index_type == TFG_I64) {
        const int64_t* ei = static_cast<const int64_t*>(edge_index);
        if (edge_weight)
          weights_coo_sliced<int64_t, true><<<blocks(coo_items<int64_t, true>()), kSlThreads, 0, s>>>(
              ei, ei + g.E_in, g.E_in, g.E, g.N, edge_weight, dinv, out_edge_index, out_w);
        else
          weights_coo_sliced<int64_t, false><<<blocks(coo_items<int64_t, false>()), kSlThreads, 0, s>>>(
              ei, ei + g.E_in, g.E_in, g.E, g.N, nullptr, dinv, out_edge_index, out_w);
      } else {
        const int32_t* ei = static_cast<const int32_t*>(edge_index);
        if (edge_weight)
          weights_coo_sliced<int32_t, true><<<blocks(coo_items<int32_t, true>()), kSlThreads, 0, s>>>(
              ei, ei + g.E_in, g.E_in, g.E, g.N, edge_weight, dinv, out_edge_index, out_w);
        else
          weights_coo_sliced<int32_t, false><<<blocks(coo_items<int32_t, false>()), kSlThreads, 0, s>>>(
              ei, ei + g.E_in, g.E_in, g.E, g.N, nullptr, dinv, out_edge_index, out_w);
      }
      TFG_LAUNCHED("gcn weights (COO order, sliced)");
      return TFG_OK;
    }
    const unsigned nb = (unsigned)((g.E + 4 * kBlock - 1) / (4 * kBlock));
    if (index_type == TFG_I64) {
      const int64_t* ei = static_cast<const int64_t*>(edge_index);
      weights_coo<int64_t><<<nb, kBlock, 0, s>>>(ei, ei + g.E_in, g.E_in, g.E, g.N, edge_weight,
                                                  dinv, out_edge_index, out_w);
    } else {
      const int32_t* ei = static_cast<const int32_t*>(edge_index);
      weights_coo<int32_t><<<nb, kBlock, 0, s>>>(ei, ei + g.E_in, g.E_in, g.E, g.N, edge_weight,
                                                  dinv, out_edge_index, out_w);
    }
    TFG_LAUNCHED("gcn weights (COO order)");
  }
  return TFG_OK;
}

}  // namespace tfg
