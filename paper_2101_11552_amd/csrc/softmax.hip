// Attention map -> reduce -> map (gfx950):
//   gat scores: per node and head, the dot products with a_src / a_dst; per
//               edge, LeakyReLU of their sum (the first map);
//   segment softmax: per target row and head, the maximum, the sum of the
//               shifted exponentials (the reduce) and the division (the last
//               map), one wavefront per row.
#include "tfg_internal.h"

namespace tfg {
namespace {

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

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

// One wavefront per target row. Lanes are (slot, head) pairs: HP heads (a
// power of two) per pass and 64 / HP edge slots; reductions across the slots
// of a head use xor butterflies (all lanes end with the same value). The
// denominator is accumulated in double.
__global__ __launch_bounds__(kBlock) void softmax_rows(const int* __restrict__ rowptr,
                                                       const int* __restrict__ perm, int64_t N,
                                                       const float* __restrict__ s, int H, int HP,
                                                       float* __restrict__ out,
                                                       float* __restrict__ out_csr) {
  const int64_t t = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
  if (t >= N) return;
  const int kb = uniform(rowptr[t]), ke = uniform(rowptr[t + 1]);
  if (kb == ke) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int SL = kWave / HP;
  const int slot = lane / HP, hh = lane % HP;
  for (int hb = 0; hb < H; hb += HP) {
    const int h = hb + hh;
    const bool act = h < H;
    float m = -__builtin_huge_valf();
    for (int k = kb + slot; k < ke; k += SL)
      if (act) {
        const float v = s[(int64_t)perm[k] * H + h];
        m = v > m ? v : m;
      }
    for (int off = HP; off < kWave; off <<= 1) {
      const float o = __shfl_xor(m, off);
      m = o > m ? o : m;
    }
    double den = 0.0;
    for (int k = kb + slot; k < ke; k += SL)
      if (act) den += (double)expf(s[(int64_t)perm[k] * H + h] - m);
    for (int off = HP; off < kWave; off <<= 1) den += __shfl_xor(den, off);
    for (int k = kb + slot; k < ke; k += SL)
      if (act) {
        const int64_t e = perm[k];
        const float a = (float)((double)expf(s[e * H + h] - m) / den);
        out[e * H + h] = a;
        if (out_csr) out_csr[(int64_t)k * H + h] = a;
      }
  }
}

}  // namespace

int launch_node_projections(const float* h, int64_t N, int H, int D, const float* a_src,
                            const float* a_dst, float* as, float* ad, hipStream_t s) {
  if (N * H == 0) return TFG_OK;
  node_projections<<<(unsigned)((N * H + kBlock - 1) / kBlock), kBlock, 0, s>>>(h, N, H, D, a_src,
                                                                               a_dst, as, ad);
  TFG_LAUNCHED("node_projections");
  return TFG_OK;
}

int launch_gat_scores(const void* edge_index, int index_type, int64_t E, const float* h, int64_t N,
                      int H, int D, const float* a_src, const float* a_dst, float slope,
                      float* out, float* proj, int* err, hipStream_t s) {
  float* as = proj;
  float* ad = proj + N * H;
  if (N * H > 0) {
    node_projections<<<(unsigned)((N * H + kBlock - 1) / kBlock), kBlock, 0, s>>>(h, N, H, D, a_src,
                                                                                 a_dst, as, ad);
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

int launch_segment_softmax(const Graph& g, const float* scores, int H, float* out, float* out_csr,
                           hipStream_t s) {
  if (g.N == 0 || g.E == 0 || H == 0) return TFG_OK;
  int hp = 1;
  while (hp * 2 <= std::min(H, kWave)) hp *= 2;
  softmax_rows<<<(unsigned)((g.N + 3) / 4), kBlock, 0, s>>>(g.rowptr, g.perm, g.N, scores, H, hp,
                                                            out, out_csr);
  TFG_LAUNCHED("softmax_rows");
  return TFG_OK;
}

}  // namespace tfg
