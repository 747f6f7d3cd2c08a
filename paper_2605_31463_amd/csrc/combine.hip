// Gather-side kernels of the layer: weighted combine, its backward (with the
// first step of the router backward fused in), and the unpermute-reduce of
// the data gradient (with the router's dx fused in).
//
// All three run one wavefront per token over 16-byte chunks of the hidden
// dimension, keep the k slot rows' loads in flight together, accumulate in
// float32 in fixed slot order (deterministic), and touch every byte of their
// HBM operands once.
#include "common.h"
#include "kernels.h"

namespace moe {

namespace {

constexpr int KMAX = 16;
constexpr int CPL = 4;  // 16-byte chunks per lane per step

__device__ __forceinline__ int64_t uniform_token(int64_t t) {
  return (int64_t)__builtin_amdgcn_readfirstlane((int)t);
}

template <class XT, int KT>
__global__ __launch_bounds__(256) void combine_fwd_kernel(CombineFwdArgs a) {
  constexpr int V = Vec16<XT>::N;
  constexpr int KM = KT > 0 ? KT : KMAX;
  const int lane = threadIdx.x & 63;
  const int64_t t = uniform_token((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
  if (t >= a.T) return;
  const int k = KT > 0 ? KT : a.k;
  const int nch = a.d / V;
  const XT* o = reinterpret_cast<const XT*>(a.o);
  const XT* sh = reinterpret_cast<const XT*>(a.shared_o);
  XT* y = reinterpret_cast<XT*>(a.y);
  const int64_t R = a.T * a.k;
  int64_t rows[KM];
  float w[KM];
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    rows[s] = s < k ? a.row_of[t * a.k + s] : 0;
    w[s] = s < k ? a.topk_w[t * a.k + s] : 0.f;
    if ((uint64_t)rows[s] >= (uint64_t)R) {  // a dropped slot contributes nothing
      rows[s] = 0;
      w[s] = 0.f;
    }
  }
  for (int c0 = 0; c0 < nch; c0 += 64 * CPL) {
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c = c0 + j * 64 + lane;
      if (c >= nch) break;
      uint4 raw[KM];
#pragma unroll
      for (int s = 0; s < KM; ++s)
        raw[s] = s < k ? *reinterpret_cast<const uint4*>(o + rows[s] * a.d + (int64_t)c * V) : make_uint4(0, 0, 0, 0);
      uint4 rs = make_uint4(0, 0, 0, 0);
      if (sh) rs = *reinterpret_cast<const uint4*>(sh + t * a.d + (int64_t)c * V);
      float acc[V];
#pragma unroll
      for (int v = 0; v < V; ++v) acc[v] = 0.f;
#pragma unroll
      for (int s = 0; s < KM; ++s) {
        if (s >= k) break;
        float vv[V];
        Vec16<XT>::load(reinterpret_cast<const XT*>(&raw[s]), vv);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[v] = __builtin_fmaf(w[s], vv[v], acc[v]);
      }
      if (sh) {
        float vv[V];
        Vec16<XT>::load(reinterpret_cast<const XT*>(&rs), vv);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[v] += vv[v];
      }
      Vec16<XT>::store(y + t * a.d + (int64_t)c * V, acc);
    }
  }
}

template <class XT, int KT>
__global__ __launch_bounds__(256) void combine_bwd_kernel(CombineBwdArgs a) {
  constexpr int V = Vec16<XT>::N;
  constexpr int KM = KT > 0 ? KT : KMAX;
  const int lane = threadIdx.x & 63;
  const int64_t t = uniform_token((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
  if (t >= a.T) return;
  const int k = KT > 0 ? KT : a.k;
  const int nch = a.d / V;
  const XT* dy = reinterpret_cast<const XT*>(a.dy);
  const XT* o = reinterpret_cast<const XT*>(a.o);
  XT* d_o = reinterpret_cast<XT*>(a.d_o);
  const int64_t R = a.T * a.k;
  int64_t rows[KM];
  float w[KM], om[KM];
  bool ok[KM];
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    rows[s] = s < k ? a.row_of[t * a.k + s] : 0;
    w[s] = s < k ? a.topk_w[t * a.k + s] : 0.f;
    om[s] = 0.f;
    ok[s] = s < k && (uint64_t)rows[s] < (uint64_t)R;
    if (!ok[s]) rows[s] = 0;
  }
  for (int c0 = 0; c0 < nch; c0 += 64 * CPL) {
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c = c0 + j * 64 + lane;
      if (c >= nch) break;
      const uint4 graw = *reinterpret_cast<const uint4*>(dy + t * a.d + (int64_t)c * V);
      uint4 raw[KM];
#pragma unroll
      for (int s = 0; s < KM; ++s)
        raw[s] = ok[s] ? *reinterpret_cast<const uint4*>(o + rows[s] * a.d + (int64_t)c * V) : make_uint4(0, 0, 0, 0);
      float g[V];
      Vec16<XT>::load(reinterpret_cast<const XT*>(&graw), g);
#pragma unroll
      for (int s = 0; s < KM; ++s) {
        if (!ok[s]) continue;
        float vv[V], out[V];
        Vec16<XT>::load(reinterpret_cast<const XT*>(&raw[s]), vv);
#pragma unroll
        for (int v = 0; v < V; ++v) {
          om[s] = __builtin_fmaf(g[v], vv[v], om[s]);
          out[v] = w[s] * g[v];
        }
        Vec16<XT>::store(d_o + rows[s] * a.d + (int64_t)c * V, out);
      }
    }
  }
  // omega_s = <dy_t, o_s>; every lane ends with the sums
  float wo = 0.f, z = 0.f;
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    if (s >= k) break;
    om[s] = wave_sum(om[s]);
    wo += w[s] * om[s];
  }
  if (lane == 0 && a.d_topk_w) {
#pragma unroll
    for (int s = 0; s < KM; ++s)
      if (s < k) a.d_topk_w[t * a.k + s] = om[s];
  }
  if (a.dl && lane == 0) {
    const float c = a.route_scale;
    if (a.router == MOE_ROUTER_SIGMOID_GROUPED) {
#pragma unroll
      for (int s = 0; s < KM; ++s)
        if (s < k) z += a.s_sel[t * a.k + s];
#pragma unroll
      for (int s = 0; s < KM; ++s)
        if (s < k) {
          const float sv = a.s_sel[t * a.k + s];
          a.dl[t * a.k + s] = (c * om[s] - wo) / z * sv * (1.f - sv);
        }
    } else {
#pragma unroll
      for (int s = 0; s < KM; ++s)
        if (s < k) a.dl[t * a.k + s] = w[s] * (om[s] - wo / c);
    }
  }
}

// The fused router dx gathers rows of W_r^T stored in the activation type
// (bf16 rows for bf16 layers: a 16-byte chunk of a row lines up with the
// activation chunk).  KT > 0: the slot count as a constant.
template <class XT, int KT>
__global__ __launch_bounds__(256) void unpermute_kernel(UnpermuteArgs a) {
  constexpr int V = Vec16<XT>::N;
  constexpr int KM = KT > 0 ? KT : KMAX;
  const int lane = threadIdx.x & 63;
  const int64_t t = uniform_token((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
  if (t >= a.T) return;
  const int k = KT > 0 ? KT : a.k;
  const int nch = a.d / V;
  const XT* dxp = reinterpret_cast<const XT*>(a.dx_perm);
  const XT* dxs = reinterpret_cast<const XT*>(a.dx_shared);
  const XT* dxa = reinterpret_cast<const XT*>(a.dx_aux);
  const XT* wrt = reinterpret_cast<const XT*>(a.w_rt);
  XT* dx = reinterpret_cast<XT*>(a.dx);
  const int64_t R = a.T * a.k;
  int64_t rows[KM], ex[KM];
  float dl[KM];
  bool ok[KM];
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    rows[s] = s < k ? a.row_of[t * a.k + s] : 0;
    ok[s] = s < k && (uint64_t)rows[s] < (uint64_t)R;
    if (!ok[s]) rows[s] = 0;
    dl[s] = (s < k && a.dl) ? a.dl[t * a.k + s] : 0.f;
    ex[s] = (s < k && a.dl) ? a.topk_idx[t * a.k + s] : 0;
  }
  for (int c0 = 0; c0 < nch; c0 += 64 * CPL) {
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c = c0 + j * 64 + lane;
      if (c >= nch) break;
      // every load of this chunk first, then the sums in slot order
      uint4 raw[KM], rw[KM];
#pragma unroll
      for (int s = 0; s < KM; ++s) {
        raw[s] = make_uint4(0, 0, 0, 0);
        rw[s] = make_uint4(0, 0, 0, 0);
        if (s < k && ok[s]) raw[s] = *reinterpret_cast<const uint4*>(dxp + rows[s] * a.d + (int64_t)c * V);
        // (a slot the permutation dropped, row -1, has no valid expert id)
        if (s < k && a.dl && ok[s]) rw[s] = *reinterpret_cast<const uint4*>(wrt + ex[s] * a.d + (int64_t)c * V);
      }
      float acc[V], r[V];
#pragma unroll
      for (int v = 0; v < V; ++v) {
        acc[v] = 0.f;
        r[v] = 0.f;
      }
#pragma unroll
      for (int s = 0; s < KM; ++s) {
        if (s >= k) break;
        float vv[V], ww[V];
        Vec16<XT>::load(reinterpret_cast<const XT*>(&raw[s]), vv);
        Vec16<XT>::load(reinterpret_cast<const XT*>(&rw[s]), ww);
#pragma unroll
        for (int v = 0; v < V; ++v) {
          acc[v] += vv[v];
          r[v] = __builtin_fmaf(dl[s], ww[v], r[v]);
        }
      }
#pragma unroll
      for (int v = 0; v < V; ++v) acc[v] += r[v];
      if (a.dx_router) {
#pragma unroll
        for (int v = 0; v < V; ++v) acc[v] += a.dx_router[t * a.d + (int64_t)c * V + v];
      }
      if (dxs) {
        float vv[V];
        Vec16<XT>::load(dxs + t * a.d + (int64_t)c * V, vv);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[v] += vv[v];
      }
      if (dxa) {
        float vv[V];
        Vec16<XT>::load(dxa + t * a.d + (int64_t)c * V, vv);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[v] += vv[v];
      }
      Vec16<XT>::store(dx + t * a.d + (int64_t)c * V, acc);
    }
  }
}

}  // namespace

#define MOE_BY_K(NAME, KID, KERNEL, XT)                                                   \
  switch (a.k) {                                                                          \
    case 8: return launch(KID, s, NAME, [&] { KERNEL<XT, 8><<<nb, 256, 0, s>>>(a); });     \
    case 4: return launch(KID, s, NAME, [&] { KERNEL<XT, 4><<<nb, 256, 0, s>>>(a); });     \
    case 2: return launch(KID, s, NAME, [&] { KERNEL<XT, 2><<<nb, 256, 0, s>>>(a); });     \
    default: return launch(KID, s, NAME, [&] { KERNEL<XT, 0><<<nb, 256, 0, s>>>(a); });    \
  }

int launch_combine_fwd(const CombineFwdArgs& a, hipStream_t s) {
  if (a.T == 0) return MOE_OK;
  const int nb = (int)((a.T + 3) / 4);
  if (a.bf16) { MOE_BY_K("combine_fwd", K_COMBINE_FWD, combine_fwd_kernel, bf16_t) }
  MOE_BY_K("combine_fwd", K_COMBINE_FWD, combine_fwd_kernel, float)
}

int launch_combine_bwd(const CombineBwdArgs& a, hipStream_t s) {
  if (a.T == 0) return MOE_OK;
  const int nb = (int)((a.T + 3) / 4);
  if (a.bf16) { MOE_BY_K("combine_bwd", K_COMBINE_BWD, combine_bwd_kernel, bf16_t) }
  MOE_BY_K("combine_bwd", K_COMBINE_BWD, combine_bwd_kernel, float)
}

template <class XT>
int launch_unpermute_t(const UnpermuteArgs& a, hipStream_t s) {
  const int nb = (int)((a.T + 3) / 4);
#define MOE_UNP(KT_) \
  return launch(K_UNPERMUTE, s, "unpermute", [&] { unpermute_kernel<XT, KT_><<<nb, 256, 0, s>>>(a); });
  switch (a.k) {
    case 8: MOE_UNP(8)
    case 4: MOE_UNP(4)
    case 2: MOE_UNP(2)
    default: MOE_UNP(0)
  }
#undef MOE_UNP
}

int launch_unpermute(const UnpermuteArgs& a, hipStream_t s) {
  if (a.T == 0) return MOE_OK;
  return a.bf16 ? launch_unpermute_t<bf16_t>(a, s) : launch_unpermute_t<float>(a, s);
}

}  // namespace moe
