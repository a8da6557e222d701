// Fused attention aggregation (gfx950): for every target row, the score map,
// the per-head segment softmax and the weighted per-head sum of Fig. 5(a) in
// one pass over the row's edges. Nothing per edge is written to memory unless
// the attention coefficients are requested.
//
// One wavefront per target row:
//   pass 1  lanes = (edge slot, head): per-head maximum of the scores;
//   pass 2  lanes = (edge slot, features) as in the aggregation kernel: every
//           lane gathers its V features of the source row and weights them with
//           exp(score - max) of its own head; the denominator is summed in
//           double next to the float32 numerators;
//   pass 3  (optional) lanes = (edge slot, head): alpha = exp(score - max) / den
//           written in the caller's edge order.
// The node projections a_s = a_src . h and a_d = a_dst . h come from
// node_projections() (softmax.hip) and sit in the workspace.
#include "tfg_internal.h"

namespace tfg {
namespace {

typedef float f2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kMaxHeads = 64;

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

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

__device__ __forceinline__ float leaky(float z, float slope) { return z >= 0.0f ? z : slope * z; }

template <int V, int SLOTS>
__global__ __launch_bounds__(kBlock) void gat_rows(const int* __restrict__ rowptr,
                                                   const int* __restrict__ col,
                                                   const int* __restrict__ perm, int64_t N, int H,
                                                   int D, int HP, const float* __restrict__ as,
                                                   const float* __restrict__ ad, float slope,
                                                   const float* __restrict__ h,
                                                   float* __restrict__ out,
                                                   float* __restrict__ alpha_out) {
  constexpr int LPS = kWave / SLOTS;
  constexpr int FC = LPS * V;
  constexpr int U = SLOTS * 4 <= kWave ? 4 : kWave / SLOTS;
  __shared__ float s_max[kBlock / kWave][kMaxHeads];
  __shared__ double s_den[kBlock / kWave][kMaxHeads];
  const int wv = threadIdx.x / kWave;
  const int64_t t = (int64_t)blockIdx.x * (kBlock / kWave) + wv;
  if (t >= N) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int F = H * D;
  const int kb = uniform(rowptr[t]), ke = uniform(rowptr[t + 1]);
  if (kb == ke) {  // a target without edges: zero output
    for (int f = lane; f < F; f += kWave) out[t * F + f] = 0.0f;
    return;
  }

  // pass 1: per-head maximum
  {
    const int SL = kWave / HP;
    const int slot = lane / HP, hh = lane % HP;
    const bool act = hh < H;
    const float adt = act ? ad[t * H + hh] : 0.0f;
    float m = -__builtin_huge_valf();
    for (int k = kb + slot; k < ke; k += SL)
      if (act) {
        const float s = leaky(as[(int64_t)col[k] * H + hh] + adt, slope);
        m = s > m ? s : m;
      }
    for (int off = HP; off < kWave; off <<= 1) {
      const float o = __shfl_xor(m, off);
      m = o > m ? o : m;
    }
    if (slot == 0 && act) s_max[wv][hh] = m;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  // pass 2: weighted per-head sums
  const int slot = lane / LPS, sl = lane % LPS;
  for (int f0 = 0; f0 < F; f0 += FC) {
    const int f = f0 + sl * V;
    const bool fok = f < F;
    const int head = fok ? f / D : 0;
    const float mh = s_max[wv][head];
    const float adt = ad[t * H + head];
    float acc[U][V];
    double den[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      den[u] = 0.0;
#pragma unroll
      for (int v = 0; v < V; ++v) acc[u][v] = 0.0f;
    }
    for (int k0 = kb; k0 < ke; k0 += SLOTS * U) {
      float xv[U][V];
      float wgt[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int k = k0 + u * SLOTS + slot;
        const bool ok = k < ke;
        const int c = ok ? col[k] : 0;
        wgt[u] = ok ? expf(leaky(as[(int64_t)c * H + head] + adt, slope) - mh) : 0.0f;
        if (ok && fok) {
          load_row<V>(h + (int64_t)c * F + f, xv[u]);
        } else {
#pragma unroll
          for (int v = 0; v < V; ++v) xv[u][v] = 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        den[u] += (double)wgt[u];
#pragma unroll
        for (int v = 0; v < V; ++v) acc[u][v] = __builtin_fmaf(wgt[u], xv[u][v], acc[u][v]);
      }
    }
#pragma unroll
    for (int step = 1; step < U; step <<= 1)
#pragma unroll
      for (int u = 0; u + step < U; u += 2 * step) {
        den[u] += den[u + step];
#pragma unroll
        for (int v = 0; v < V; ++v) acc[u][v] += acc[u + step][v];
      }
#pragma unroll
    for (int off = LPS; off < kWave; off <<= 1) {
      den[0] += __shfl_xor(den[0], off);
#pragma unroll
      for (int v = 0; v < V; ++v) acc[0][v] += __shfl_xor(acc[0][v], off);
    }
    if (slot == 0 && fok) {
#pragma unroll
      for (int v = 0; v < V; ++v) out[t * F + f + v] = (float)((double)acc[0][v] / den[0]);
      if (alpha_out != nullptr && f % D == 0) s_den[wv][head] = den[0];
    }
  }
  if (alpha_out == nullptr) return;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  // pass 3: attention coefficients in the caller's edge order
  {
    const int SL = kWave / HP;
    const int slot3 = lane / HP, hh = lane % HP;
    if (hh < H) {
      const float adt = ad[t * H + hh];
      const float mh = s_max[wv][hh];
      const double dn = s_den[wv][hh];
      for (int k = kb + slot3; k < ke; k += SL) {
        const float w = expf(leaky(as[(int64_t)col[k] * H + hh] + adt, slope) - mh);
        alpha_out[(int64_t)perm[k] * H + hh] = (float)((double)w / dn);
      }
    }
  }
}

template <int V>
void launch_slots(int slots, dim3 grid, hipStream_t s, const Graph& g, int H, int D, int HP,
                  const float* as, const float* ad, float slope, const float* h, float* out,
                  float* alpha_out) {
#define TFG_GAT(SL)                                                                               \
  gat_rows<V, SL><<<grid, kBlock, 0, s>>>(g.rowptr, g.col, g.perm, g.N, H, D, HP, as, ad, slope, \
                                          h, out, alpha_out)
  switch (slots) {
    case 1: TFG_GAT(1); break;
    case 2: TFG_GAT(2); break;
    case 4: TFG_GAT(4); break;
    case 8: TFG_GAT(8); break;
    default: TFG_GAT(16); break;
  }
#undef TFG_GAT
}

}  // namespace

size_t gat_aggregate_ws_bytes(int64_t N, int64_t H) {
  return align_up(sizeof(float) * (size_t)std::max<int64_t>(2 * N * H, 1), 256) + 256;
}

int max_fused_heads() { return kMaxHeads; }

int launch_gat_aggregate(const Graph& g, const float* h, int H, int D, const float* a_src,
                         const float* a_dst, float slope, float* out, float* alpha_out, void* ws,
                         hipStream_t s) {
  if (g.N == 0 || H == 0 || D == 0) return TFG_OK;
  float* as = static_cast<float*>(ws);
  float* ad = as + g.N * H;
  int rc = launch_node_projections(h, g.N, H, D, a_src, a_dst, as, ad, s);
  if (rc) return rc;
  const int64_t F = (int64_t)H * D;
  auto fits = [&](int v) {
    return D % v == 0 && reinterpret_cast<uintptr_t>(h) % (4 * v) == 0 &&
           reinterpret_cast<uintptr_t>(out) % (4 * v) == 0;
  };
  const int vec = fits(4) ? 4 : fits(2) ? 2 : 1;
  const int lanes = (int)std::min<int64_t>((F + vec - 1) / vec, kWave);
  int p2 = 1;
  while (p2 < lanes) p2 <<= 1;
  const int slots = std::min(kWave / p2, 16);
  int hp = 1;
  while (hp < H) hp <<= 1;  // heads per pass (a power of two, at most 64)
  dim3 grid((unsigned)((g.N + kBlock / kWave - 1) / (kBlock / kWave)));
  if (vec == 4)
    launch_slots<4>(slots, grid, s, g, H, D, hp, as, ad, slope, h, out, alpha_out);
  else if (vec == 2)
    launch_slots<2>(slots, grid, s, g, H, D, hp, as, ad, slope, h, out, alpha_out);
  else
    launch_slots<1>(slots, grid, s, g, H, D, hp, as, ad, slope, h, out, alpha_out);
  TFG_LAUNCHED("gat_rows");
  return TFG_OK;
}

}  // namespace tfg
