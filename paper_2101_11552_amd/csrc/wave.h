// Wavefront helpers shared by the device sources.
#pragma once

#include "tfg_internal.h"

namespace tfg {

// A value the compiler cannot prove wave-uniform, made scalar.
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

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

// K exclusive scans at once (one value per list per thread) over a block of
// NW waves: the lists share the barriers (two in all). tmp: NW * K ints.
template <int NW, int K>
__device__ __forceinline__ void block_excl_scan_lists(const int (&v)[K], int (&ex)[K],
                                                      int (&total)[K], int* tmp) {
  const int wave = threadIdx.x / kWave;
  int incl[K];
#pragma unroll
  for (int i = 0; i < K; ++i) {
    incl[i] = wave_incl_scan(v[i]);
    if (lane_id() == kWave - 1) tmp[i * NW + wave] = incl[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < K; ++i) {
    int off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const int t = tmp[i * NW + w];
      if (w < wave) off += t;
      tot += t;
    }
    ex[i] = off + incl[i] - v[i];
    total[i] = tot;
  }
  __syncthreads();
}

}  // namespace tfg
