// Softmax statistics merged online (device code): a pair (m, d) stands for a
// set of scores with maximum m and d = sum of exp(s - m) (in double). Adding
// a score or merging two pairs rescales d to the larger maximum, so a
// segment's maximum and denominator come out of one sweep, in any grouping;
// an empty set is (-inf, 0). Both operations are symmetric in their operands
// (IEEE addition and multiplication commute), so xor butterflies leave every
// lane with the same pair.
#pragma once

#include "wave.h"

namespace tfg {

__device__ __forceinline__ void stat_merge(float& m, double& d, float m2, double d2) {
#pragma clang fp contract(off)
  if (m2 == -__builtin_huge_valf()) return;
  if (m == -__builtin_huge_valf()) {
    m = m2;
    d = d2;
    return;
  }
  const float mn = m2 > m ? m2 : m;
  d = d * (double)expf(m - mn) + d2 * (double)expf(m2 - mn);
  m = mn;
}

// One exponential per score: t = exp(-|v - m|) is the new term when the
// maximum stays and the rescale factor of d when it grows (from m = -inf the
// factor is 0).
__device__ __forceinline__ void stat_add(float& m, double& d, float v) {
#pragma clang fp contract(off)
  const float dlt = v - m;
  const float t = expf(-__builtin_fabsf(dlt));
  const bool up = dlt > 0.0f;
  d = up ? d * (double)t + 1.0 : d + (double)t;
  m = up ? v : m;
}

// Register sweeps of the row plan's items (softmax and its gradient): lanes
// are (slot, head) pairs, SL = 64 / HP slots; slot step u of an item
// starting at kb is position kb + slot + u * SL.
// Edge ids of NST steps of [kb, ke) (-1 past ke).
// Where the per-edge values of graph position k live: at the caller's edge id
// perm[k], or (perm NULL: arrays kept in the graph order) at k itself.
__device__ __forceinline__ int edge_at(const int* __restrict__ perm, int k) {
  return perm != nullptr ? perm[k] : k;
}

template <int NST>
__device__ __forceinline__ void load_ids(const int* __restrict__ perm, int kb, int ke, int slot,
                                         int SL, int (&e)[NST]) {
#pragma unroll
  for (int u = 0; u < NST; ++u) {
    const int k = kb + slot + u * SL;
    e[u] = k < ke ? edge_at(perm, k) : -1;
  }
}

// Sum over the slots of a head (lanes l, l ^ HP, l ^ 2 HP, ...). IEEE
// addition commutes, so every lane of a head ends with the same sum.
__device__ __forceinline__ double slots_sum(double d, int HP) {
  for (int off = HP; off < kWave; off <<= 1) d += __shfl_xor(d, off);
  return d;
}

}  // namespace tfg
