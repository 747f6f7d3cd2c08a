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
constexpr int CPL = 2;  // 16-byte chunks per lane per step

__device__ __forceinline__ int64_t uniform_token(int64_t t) {
  return (int64_t)__builtin_amdgcn_readfirstlane((int)t);
}

template <class XT>
__global__ __launch_bounds__(256) void combine_fwd_kernel(CombineFwdArgs a) {
  constexpr int V = Vec16<XT>::N;
  const int lane = threadIdx.x & 63;
  const int64_t t = uniform_token((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
  if (t >= a.T) return;
  const int k = a.k;
  const int nch = a.d / V;
  const XT* o = reinterpret_cast<const XT*>(a.o);
  const XT* sh = reinterpret_cast<const XT*>(a.shared_o);
  XT* y = reinterpret_cast<XT*>(a.y);
  const int64_t R = a.T * k;
  int64_t rows[KMAX];
  float w[KMAX];
#pragma unroll
  for (int s = 0; s < KMAX; ++s) {
    rows[s] = s < k ? a.row_of[t * k + s] : 0;
    w[s] = s < k ? a.topk_w[t * k + s] : 0.f;
    if ((uint64_t)rows[s] >= (uint64_t)R) {  // a dropped slot contributes nothing
      rows[s] = 0;
      w[s] = 0.f;
    }
  }
  for (int c0 = 0; c0 < nch; c0 += 64 * CPL) {
    float acc[CPL][V];
#pragma unroll
    for (int j = 0; j < CPL; ++j)
#pragma unroll
      for (int v = 0; v < V; ++v) acc[j][v] = 0.f;
#pragma unroll
    for (int s = 0; s < KMAX; ++s) {
      if (s >= k) break;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c = c0 + j * 64 + lane;
        if (c < nch) {
          float vv[V];
          Vec16<XT>::load(o + rows[s] * a.d + (int64_t)c * V, vv);
#pragma unroll
          for (int v = 0; v < V; ++v) acc[j][v] = __builtin_fmaf(w[s], vv[v], acc[j][v]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c = c0 + j * 64 + lane;
      if (c < nch) {
        if (sh) {
          float vv[V];
          Vec16<XT>::load(sh + t * a.d + (int64_t)c * V, vv);
#pragma unroll
          for (int v = 0; v < V; ++v) acc[j][v] += vv[v];
        }
        Vec16<XT>::store(y + t * a.d + (int64_t)c * V, acc[j]);
      }
    }
  }
}

template <class XT>
__global__ __launch_bounds__(256) void combine_bwd_kernel(CombineBwdArgs a) {
  constexpr int V = Vec16<XT>::N;
  const int lane = threadIdx.x & 63;
  const int64_t t = uniform_token((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
  if (t >= a.T) return;
  const int k = a.k;
  const int nch = a.d / V;
  const XT* dy = reinterpret_cast<const XT*>(a.dy);
  const XT* o = reinterpret_cast<const XT*>(a.o);
  XT* d_o = reinterpret_cast<XT*>(a.d_o);
  const int64_t R = a.T * k;
  int64_t rows[KMAX];
  float w[KMAX];
  float om[KMAX];
  bool ok[KMAX];
#pragma unroll
  for (int s = 0; s < KMAX; ++s) {
    rows[s] = s < k ? a.row_of[t * k + s] : 0;
    w[s] = s < k ? a.topk_w[t * k + s] : 0.f;
    om[s] = 0.f;
    ok[s] = (uint64_t)rows[s] < (uint64_t)R;
    if (!ok[s]) rows[s] = 0;
  }
  for (int c0 = 0; c0 < nch; c0 += 64 * CPL) {
    float g[CPL][V];
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c = c0 + j * 64 + lane;
      if (c < nch) Vec16<XT>::load(dy + t * a.d + (int64_t)c * V, g[j]);
    }
#pragma unroll
    for (int s = 0; s < KMAX; ++s) {
      if (s >= k) break;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c = c0 + j * 64 + lane;
        if (c < nch && ok[s]) {
          float vv[V], out[V];
          Vec16<XT>::load(o + rows[s] * a.d + (int64_t)c * V, vv);
#pragma unroll
          for (int v = 0; v < V; ++v) {
            om[s] = __builtin_fmaf(g[j][v], vv[v], om[s]);
            out[v] = w[s] * g[j][v];
          }
          Vec16<XT>::store(d_o + rows[s] * a.d + (int64_t)c * V, out);
        }
      }
    }
  }
  // omega_s = <dy_t, o_s>; every lane ends with the sums
  float wo = 0.f, z = 0.f;
#pragma unroll
  for (int s = 0; s < KMAX; ++s) {
    if (s >= k) break;
    om[s] = wave_sum(om[s]);
    wo += w[s] * om[s];
  }
  if (lane == 0 && a.d_topk_w) {
#pragma unroll
    for (int s = 0; s < KMAX; ++s)
      if (s < k) a.d_topk_w[t * k + s] = om[s];
  }
  if (a.dl && lane == 0) {
    const float c = a.route_scale;
    if (a.router == MOE_ROUTER_SIGMOID_GROUPED) {
#pragma unroll
      for (int s = 0; s < KMAX; ++s)
        if (s < k) z += a.s_sel[t * k + s];
#pragma unroll
      for (int s = 0; s < KMAX; ++s)
        if (s < k) {
          const float sv = a.s_sel[t * k + s];
          a.dl[t * k + s] = (c * om[s] - wo) / z * sv * (1.f - sv);
        }
    } else {
#pragma unroll
      for (int s = 0; s < KMAX; ++s)
        if (s < k) a.dl[t * k + s] = w[s] * (om[s] - wo / c);
    }
  }
}

template <class XT>
__global__ __launch_bounds__(256) void unpermute_kernel(UnpermuteArgs a) {
  constexpr int V = Vec16<XT>::N;
  const int lane = threadIdx.x & 63;
  const int64_t t = uniform_token((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
  if (t >= a.T) return;
  const int k = a.k;
  const int nch = a.d / V;
  const XT* dxp = reinterpret_cast<const XT*>(a.dx_perm);
  const XT* dxs = reinterpret_cast<const XT*>(a.dx_shared);
  XT* dx = reinterpret_cast<XT*>(a.dx);
  const int64_t R = a.T * k;
  int64_t rows[KMAX];
  float dl[KMAX];
  int64_t ex[KMAX];
  bool ok[KMAX];
#pragma unroll
  for (int s = 0; s < KMAX; ++s) {
    rows[s] = s < k ? a.row_of[t * k + s] : 0;
    ok[s] = (uint64_t)rows[s] < (uint64_t)R;
    if (!ok[s]) rows[s] = 0;
    dl[s] = (s < k && a.dl) ? a.dl[t * k + s] : 0.f;
    ex[s] = (s < k && a.dl) ? a.topk_idx[t * k + s] : 0;
  }
  for (int c0 = 0; c0 < nch; c0 += 64 * CPL) {
    float acc[CPL][V];
#pragma unroll
    for (int j = 0; j < CPL; ++j)
#pragma unroll
      for (int v = 0; v < V; ++v) acc[j][v] = 0.f;
#pragma unroll
    for (int s = 0; s < KMAX; ++s) {
      if (s >= k) break;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c = c0 + j * 64 + lane;
        if (c < nch && ok[s]) {
          float vv[V];
          Vec16<XT>::load(dxp + rows[s] * a.d + (int64_t)c * V, vv);
#pragma unroll
          for (int v = 0; v < V; ++v) acc[j][v] += vv[v];
        }
      }
    }
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c = c0 + j * 64 + lane;
      if (c >= nch) continue;
      if (a.dx_router) {
#pragma unroll
        for (int v = 0; v < V; ++v) acc[j][v] += a.dx_router[t * a.d + (int64_t)c * V + v];
      }
      if (a.dl) {
        float r[V];
#pragma unroll
        for (int v = 0; v < V; ++v) r[v] = 0.f;
#pragma unroll
        for (int s = 0; s < KMAX; ++s) {
          if (s >= k) break;
#pragma unroll
          for (int v = 0; v < V; ++v)
            r[v] = __builtin_fmaf(dl[s], a.w_rt[ex[s] * a.d + (int64_t)c * V + v], r[v]);
        }
#pragma unroll
        for (int v = 0; v < V; ++v) acc[j][v] += r[v];
      }
      if (dxs) {
        float vv[V];
        Vec16<XT>::load(dxs + t * a.d + (int64_t)c * V, vv);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[j][v] += vv[v];
      }
      Vec16<XT>::store(dx + t * a.d + (int64_t)c * V, acc[j]);
    }
  }
}

}  // namespace

int launch_combine_fwd(const CombineFwdArgs& a, hipStream_t s) {
  if (a.T == 0) return MOE_OK;
  const int nb = (int)((a.T + 3) / 4);
  if (a.bf16)
    return launch(K_COMBINE_FWD, s, "combine_fwd", [&] { combine_fwd_kernel<bf16_t><<<nb, 256, 0, s>>>(a); });
  return launch(K_COMBINE_FWD, s, "combine_fwd", [&] { combine_fwd_kernel<float><<<nb, 256, 0, s>>>(a); });
}

int launch_combine_bwd(const CombineBwdArgs& a, hipStream_t s) {
  if (a.T == 0) return MOE_OK;
  const int nb = (int)((a.T + 3) / 4);
  if (a.bf16)
    return launch(K_COMBINE_BWD, s, "combine_bwd", [&] { combine_bwd_kernel<bf16_t><<<nb, 256, 0, s>>>(a); });
  return launch(K_COMBINE_BWD, s, "combine_bwd", [&] { combine_bwd_kernel<float><<<nb, 256, 0, s>>>(a); });
}

int launch_unpermute(const UnpermuteArgs& a, hipStream_t s) {
  if (a.T == 0) return MOE_OK;
  const int nb = (int)((a.T + 3) / 4);
  if (a.bf16)
    return launch(K_UNPERMUTE, s, "unpermute", [&] { unpermute_kernel<bf16_t><<<nb, 256, 0, s>>>(a); });
  return launch(K_UNPERMUTE, s, "unpermute", [&] { unpermute_kernel<float><<<nb, 256, 0, s>>>(a); });
}

}  // namespace moe
