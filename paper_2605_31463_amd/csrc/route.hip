// Router forward: logits, top-k selection, gating weights, expert counts.
//
// One fused kernel per block of 32 tokens:
//   1. logits l = x W_r for the block's tokens and every expert.  Products
//      run in float32 FMA chains of 16 terms; each chain is folded into a
//      float64 total, so a logit carries about 1e-7 absolute error at the
//      workloads' scale and the float64 selection keys order experts the
//      way an exact evaluation does outside sub-1e-6 near-ties.
//   2. one wavefront per token selects the top-k over float64 keys with
//      64-lane butterfly reductions (the framework's top-k routing kernel,
//      section 3.2 / appendix B.3), optionally restricted to the best
//      expert groups (group score = sum of the group's two largest keys);
//   3. gating weights over the selected experts: softmax of the selected
//      (biased) logits, or route_scale * sigmoid / sum of sigmoids; weights
//      are non-negative and sum to route_scale (appendix B.2.2 rules);
//   4. per-block expert histogram added into the expert counts.
#include <float.h>
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace moe {

namespace {

constexpr int TB = 32;   // tokens per block
constexpr int KS = 32;   // hidden elements per LDS stage
constexpr int CH = 16;   // float32 chain length before folding into float64

struct Cand {
  double key;
  int idx;
};

__device__ __forceinline__ bool better(double ka, int ia, double kb, int ib) {
  return ka > kb || (ka == kb && ia < ib);
}

// Butterfly over `width` lanes (power of two) keeping the better candidate.
__device__ __forceinline__ Cand wave_best(Cand c, int width) {
  for (int m = 1; m < width; m <<= 1) {
    double ok = __shfl_xor(c.key, m, 64);
    int oi = __shfl_xor(c.idx, m, 64);
    if (better(ok, oi, c.key, c.idx)) {
      c.key = ok;
      c.idx = oi;
    }
  }
  return c;
}

__device__ __forceinline__ double wave_sum_d(double v, int width) {
  for (int m = 1; m < width; m <<= 1) v += __shfl_xor(v, m, 64);
  return v;
}
__device__ __forceinline__ double wave_max_d(double v, int width) {
  for (int m = 1; m < width; m <<= 1) v = fmax(v, __shfl_xor(v, m, 64));
  return v;
}

template <class XT, int EPT>
__global__ __launch_bounds__(256) void route_kernel(RouteArgs a) {
  constexpr int EPAD = 16 * EPT;
  constexpr int STAGE_BYTES = (KS * TB + KS * EPAD) * 4;
  constexpr int TABLE_BYTES = TB * EPAD * 8;
  constexpr int SMEM = STAGE_BYTES > TABLE_BYTES ? STAGE_BYTES : TABLE_BYTES;
  __shared__ __align__(16) unsigned char smem[SMEM];
  __shared__ int hist[EPAD];

  const int tid = threadIdx.x;
  const int tx = tid & 15;
  const int ty = tid >> 4;
  const int E = a.E;
  const int d = a.d;
  const int64_t t0 = (int64_t)blockIdx.x * TB;
  const XT* x = reinterpret_cast<const XT*>(a.x);

  for (int e = tid; e < EPAD; e += 256) hist[e] = 0;

  float* xs = reinterpret_cast<float*>(smem);   // [KS][TB]
  float* wsm = xs + KS * TB;                     // [KS][EPAD]

  double acc[2][EPT];
  float part[2][EPT];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      acc[i][j] = 0.0;
      part[i][j] = 0.f;
    }

  for (int k0 = 0; k0 < d; k0 += KS) {
    // stage x: token tid/8, elements (tid%8)*4 .. +3
    {
      const int tl = tid >> 3;
      const int c = (tid & 7) * 4;
      const int64_t t = t0 + tl;
      float v[4] = {0.f, 0.f, 0.f, 0.f};
      if (t < a.T) {
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = Elem<XT>::load(x, t * d + k0 + c + q);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) xs[(c + q) * TB + tl] = v[q];
    }
    // stage W_r rows k0..k0+KS-1
    for (int i = tid; i < KS * EPAD; i += 256) {
      const int r = i / EPAD;
      const int e = i - r * EPAD;
      wsm[i] = e < E ? a.w_r[(int64_t)(k0 + r) * E + e] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const float2 xv = *reinterpret_cast<const float2*>(&xs[kk * TB + 2 * ty]);
      float wv[EPT];
#pragma unroll
      for (int j = 0; j < EPT; ++j) wv[j] = wsm[kk * EPAD + tx * EPT + j];
#pragma unroll
      for (int j = 0; j < EPT; ++j) {
        part[0][j] = __builtin_fmaf(xv.x, wv[j], part[0][j]);
        part[1][j] = __builtin_fmaf(xv.y, wv[j], part[1][j]);
      }
      if ((kk % CH) == CH - 1) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < EPT; ++j) {
            acc[i][j] += (double)part[i][j];
            part[i][j] = 0.f;
          }
      }
    }
    __syncthreads();
  }

  // logits -> LDS table [TB][EPAD] (float64)
  double* lg = reinterpret_cast<double*>(smem);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < EPT; ++j) lg[(2 * ty + i) * EPAD + tx * EPT + j] = acc[i][j];
  __syncthreads();

  // selection: one wavefront per token
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int epl = (E + 63) / 64;              // experts per lane, contiguous
  const bool sigm = a.router == MOE_ROUTER_SIGMOID_GROUPED;
  const bool logit_bias = a.bias_mode == MOE_BIAS_LOGIT;
  const bool select_bias = a.bias_mode == MOE_BIAS_SELECT_ONLY;
  const int gsize = E / a.n_groups;           // experts per group
  const int lpg = gsize / epl;                // lanes per group (power of two)
  const int k = a.k;

  for (int tl = wave; tl < TB; tl += 4) {
    const int64_t t = t0 + tl;
    if (t >= a.T) break;
    double key[4];
    bool avail[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane * epl + q;
      avail[q] = q < epl && e < E;
      key[q] = -INFINITY;
      if (avail[q]) {
        double l = lg[tl * EPAD + e];
        if (logit_bias) l += (double)a.bias[e];
        double sc = sigm ? 1.0 / (1.0 + exp(-l)) : l;
        const double kv = select_bias ? sc + (double)a.bias[e] : sc;
        key[q] = isnan(kv) ? -INFINITY : kv;  // NaN orders below every number
      }
    }
    // group limit
    if (a.n_groups > 1) {
      double m1 = -INFINITY, m2 = -INFINITY;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (!avail[q]) continue;
        if (key[q] > m1) {
          m2 = m1;
          m1 = key[q];
        } else if (key[q] > m2) {
          m2 = key[q];
        }
      }
      for (int m = 1; m < lpg; m <<= 1) {
        double o1 = __shfl_xor(m1, m, 64);
        double o2 = __shfl_xor(m2, m, 64);
        double n1 = fmax(m1, o1);
        double n2 = fmax(fmin(m1, o1), fmax(m2, o2));
        m1 = n1;
        m2 = n2;
      }
      const bool lane_live = lane * epl < E;
      const int g = lane_live ? (lane * epl) / gsize : 0x7fffffff;
      double gscore = !lane_live ? -INFINITY : (gsize >= 2 ? m1 + m2 : m1);
      if (isnan(gscore)) gscore = -INFINITY;
      bool kept = false;
      bool gtaken = false;
      for (int r = 0; r < a.topk_groups; ++r) {
        Cand c{(lane_live && !gtaken) ? gscore : -INFINITY, (lane_live && !gtaken) ? g : 0x7fffffff};
        c = wave_best(c, 64);
        if (c.idx == g) {
          kept = true;
          gtaken = true;
        }
      }
      if (!kept) {
#pragma unroll
        for (int q = 0; q < 4; ++q) avail[q] = false;
      }
    }
    // top-k
    int my_idx = -1;
    for (int s = 0; s < k; ++s) {
      Cand c{-INFINITY, 0x7fffffff};  // any available expert beats the empty slot (lower index)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = lane * epl + q;
        if (avail[q] && better(key[q], e, c.key, c.idx)) {
          c.key = key[q];
          c.idx = e;
        }
      }
      c = wave_best(c, 64);
      if (c.idx / epl == lane) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (lane * epl + q == c.idx) avail[q] = false;
      }
      if (lane == s) my_idx = c.idx;
    }
    // weights over the k selected (lanes 0..k-1 hold one slot each)
    const bool holds = lane < k;
    double sc = 0.0;
    if (holds) {
      double l = lg[tl * EPAD + my_idx];
      if (logit_bias) l += (double)a.bias[my_idx];
      sc = sigm ? 1.0 / (1.0 + exp(-l)) : l;
    }
    double w;
    if (sigm) {
      const double z = wave_sum_d(holds ? sc : 0.0, 64);
      w = (double)a.route_scale * sc / z;
    } else {
      const double m = wave_max_d(holds ? sc : -INFINITY, 64);
      const double p = holds ? exp(sc - m) : 0.0;
      const double z = wave_sum_d(p, 64);
      w = (double)a.route_scale * p / z;
    }
    if (holds) {
      a.topk_idx[t * k + lane] = my_idx;
      a.topk_w[t * k + lane] = (float)w;
      if (sigm && a.s_sel) a.s_sel[t * k + lane] = (float)sc;
      atomicAdd(&hist[my_idx], 1);
    }
  }
  __syncthreads();
  if (a.counts) {
    for (int e = tid; e < E; e += 256)
      if (hist[e]) atomicAdd(&a.counts[e], hist[e]);
  }
}

__global__ void zero_i32_kernel(int32_t* p, int64_t n) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

template <class XT>
int launch_route_t(const RouteArgs& a, hipStream_t s) {
  const int nblk = (int)((a.T + TB - 1) / TB);
  const dim3 grid(nblk), block(256);
#define MOE_ROUTE_CASE(EPT_)                                                                      \
  if (a.E <= 16 * EPT_)                                                                           \
    return launch(K_ROUTE, s, "route", [&] { route_kernel<XT, EPT_><<<grid, block, 0, s>>>(a); });
  MOE_ROUTE_CASE(1)
  MOE_ROUTE_CASE(2)
  MOE_ROUTE_CASE(4)
  MOE_ROUTE_CASE(8)
  MOE_ROUTE_CASE(16)
#undef MOE_ROUTE_CASE
  return moe_set_error(MOE_ERR_UNSUPPORTED, "route: E=%d above 256", a.E);
}

}  // namespace

int zero_i32(int32_t* p, int64_t n, hipStream_t s) {
  if (n <= 0) return MOE_OK;
  const int nb = (int)((n + 255) / 256);
  return launch(K_COUNT_ZERO, s, "zero", [&] { zero_i32_kernel<<<nb, 256, 0, s>>>(p, n); });
}

int launch_route(const RouteArgs& a, hipStream_t s) {
  if (a.counts) {
    int st = zero_i32(a.counts, a.E, s);
    if (st) return st;
  }
  if (a.T == 0) return MOE_OK;
  return a.bf16 ? launch_route_t<bf16_t>(a, s) : launch_route_t<float>(a, s);
}

}  // namespace moe
