// Global-level load-balancing loss of the router (the paper pretrains with
// one of coefficient 1e-3, appendix A.1 training configuration):
//   L = coef * E * sum_e eta_e f_e P_e,  P_e = mean over tokens of p[t][e],
// p the softmax over all E logits of the pool (written by the route kernels),
// f_e the fraction of the T*k routed slots that chose e (or fractions of the
// whole batch given by the caller), eta_e = 1 for FFN experts and the given
// weight for zero-computation experts (appendix B.3, MoE++: the loss treats
// them explicitly).  f carries no gradient, so with q = eta f
//   dL/dl[t][j] = coef * E / T * p[t][j] * (q_j - sum_e q_e p[t][e]),
// a dense [T][E] term added to the router's logit gradient; its products
// with x (dW_r) and W_r^T (dx) run on the grouped GEMM kernels.
// Deterministic: every sum has a fixed order, no floating-point atomics.
#include "common.h"
#include "kernels.h"

namespace moe {
namespace {

// eta_e f_e: zero-computation experts (e >= E_ffn) weigh zc_weight.  The
// threshold router fills a variable number of slots: f is the share of the
// filled ones.
__device__ __forceinline__ double aux_frac(const AuxArgs& a, int e) {
  const double n = a.thr ? (double)max(a.offsets[a.E], 1) : (double)a.T * (double)a.k;
  const double f = a.aux_f ? (double)a.aux_f[e] : (double)(a.offsets[e + 1] - a.offsets[e]) / n;
  return e >= a.E_ffn ? (double)a.zc_weight * f : f;
}

// Column sums of p over each block of 256 tokens: 64 experts (blockIdx.y
// picks which) by 4 quarters of 64 tokens, 16 loads in flight per thread, the
// quarters added in order.
__global__ __launch_bounds__(256) void aux_partial_kernel(AuxArgs a) {
  const int el = threadIdx.x & 63, tq = threadIdx.x >> 6;
  const int e = blockIdx.y * 64 + el;
  __shared__ double red[4][64];
  double acc = 0.0;
  if (e < a.E) {
    // indices clamped to the last token and the values masked, so that the
    // 16 loads of a batch are issued together (no branch between them)
    const int64_t tb = (int64_t)blockIdx.x * 256 + tq * 64;
    for (int j0 = 0; j0 < 64; j0 += 16) {
      float v[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int64_t t = tb + j0 + j;
        v[j] = a.probs[(t < a.T ? t : a.T - 1) * a.E + e];
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) acc += tb + j0 + j < a.T ? (double)v[j] : 0.0;
    }
  }
  red[tq][el] = acc;
  __syncthreads();
  if (tq == 0 && e < a.E)
    a.part[(int64_t)blockIdx.x * a.E + e] = ((red[0][el] + red[1][el]) + red[2][el]) + red[3][el];
}

// One block: P_e from the partials in block order, then the loss by a fixed
// tree over the experts.
__global__ __launch_bounds__(256) void aux_loss_kernel(AuxArgs a, int nb) {
  __shared__ double red[256];
  const int e = threadIdx.x;
  double term = 0.0;
  if (e < a.E && a.T > 0) {
    // eight running sums (eight loads in flight), added in a fixed order
    double Ps[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int b0 = 0; b0 < nb; b0 += 8) {
      double v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = a.part[(int64_t)(b0 + j < nb ? b0 + j : nb - 1) * a.E + e];
#pragma unroll
      for (int j = 0; j < 8; ++j) Ps[j] += b0 + j < nb ? v[j] : 0.0;
    }
    const double P = ((Ps[0] + Ps[1]) + (Ps[2] + Ps[3])) + ((Ps[4] + Ps[5]) + (Ps[6] + Ps[7]));
    term = aux_frac(a, e) * (P / (double)a.T);
  }
  red[e] = term;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (e < w) red[e] += red[e + w];
    __syncthreads();
  }
  if (e == 0) *a.loss = (float)((double)a.coef * (double)a.E * red[0]);
}

__device__ __forceinline__ double wave_sum(double v) {
  for (int m = 1; m < 64; m <<= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// Threshold router: column sums of p = s / sum_e s (s the sigmoid scores in
// probs) over blocks of 256 tokens; each wavefront takes 64 tokens in order
// (the per-token sum over experts is a wave sum), expert e = lane + 64 q, and
// the four wavefronts' sums are added in order.
__global__ __launch_bounds__(256) void aux_partial_rows_kernel(AuxArgs a) {
  __shared__ double red[4][256];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  const int64_t tb = (int64_t)blockIdx.x * 256 + w * 64;
  for (int j = 0; j < 64; ++j) {
    const int64_t t = tb + j;
    if (t >= a.T) break;
    double sv[4], S = 0.0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane + 64 * q;
      sv[q] = e < a.E ? (double)a.probs[t * a.E + e] : 0.0;
      S += sv[q];
    }
    S = wave_sum(S);
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] += sv[q] / S;
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) red[w][lane + 64 * q] = acc[q];
  __syncthreads();
  for (int e = threadIdx.x; e < a.E; e += 256)
    a.part[(int64_t)blockIdx.x * a.E + e] = ((red[0][e] + red[1][e]) + red[2][e]) + red[3][e];
}

// One wavefront per token, expert e = lane + 64 q.  Block 0 also writes the
// token-chunk offsets [G+1] of the grouped dW_r product.
template <class OT>
__global__ __launch_bounds__(256) void aux_grad_kernel(AuxArgs a, OT* __restrict__ dl, int E_pad, int32_t* off,
                                                       int G, int64_t chunk) {
  if (blockIdx.x == 0)
    for (int g = threadIdx.x; g <= G; g += blockDim.x) {
      const int64_t r = (int64_t)g * chunk;
      off[g] = (int32_t)(r < a.T ? r : a.T);
    }
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= a.T) return;
  double p[4], fe[4], sg[4];
  double F = 0.0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = lane + 64 * q;
    p[q] = 0.0;
    fe[q] = 0.0;
    sg[q] = 0.0;
    if (e < a.E) {
      p[q] = (double)a.probs[t * a.E + e];
      fe[q] = aux_frac(a, e);
    }
  }
  if (a.thr) {
    // p = s / sum s; dp/dl carries the factor (1 - s)
    double S = 0.0;
#pragma unroll
    for (int q = 0; q < 4; ++q) S += p[q];
    S = wave_sum(S);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      sg[q] = p[q];
      p[q] = p[q] / S;
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) F += p[q] * fe[q];
  F = wave_sum(F);
  const double c = (double)a.coef * (double)a.E / (double)a.T;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = lane + 64 * q;
    const double g = c * p[q] * (fe[q] - F) * (a.thr ? 1.0 - sg[q] : 1.0);
    if (e < E_pad) Elem<OT>::store(dl, t * E_pad + e, e < a.E ? (float)g : 0.f);
  }
}

// dw_r[i][e] += sum_g part[g][i][e], chunks in order.
template <class IT>
__global__ __launch_bounds__(256) void aux_dwr_kernel(const IT* __restrict__ part, int G, int d, int E, int E_pad,
                                                      float* __restrict__ dw_r) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)d * E) return;
  const int i = (int)(idx / E), e = (int)(idx - (int64_t)i * E);
  float acc = 0.f;
  for (int g0 = 0; g0 < G; g0 += 8) {
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = Elem<IT>::load(part, ((int64_t)(g0 + j < G ? g0 + j : G - 1) * d + i) * E_pad + e);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc += g0 + j < G ? v[j] : 0.f;
  }
  dw_r[idx] += acc;
}

}  // namespace

int launch_aux_stats(const AuxArgs& a, hipStream_t s) {
  const int nb = (int)aux_blocks(a.T);
  if (nb > 0 && a.thr) {
    const int st =
        launch(K_AUX_PARTIAL_ROWS, s, "aux_partial_rows", [&] { aux_partial_rows_kernel<<<nb, 256, 0, s>>>(a); });
    if (st) return st;
  } else if (nb > 0) {
    const dim3 grid(nb, (a.E + 63) / 64);
    const int st = launch(K_AUX_STATS, s, "aux_stats", [&] { aux_partial_kernel<<<grid, 256, 0, s>>>(a); });
    if (st) return st;
  }
  return launch(K_AUX_STATS, s, "aux_stats", [&] { aux_loss_kernel<<<1, 256, 0, s>>>(a, nb); });
}

int launch_aux_grad(const AuxArgs& a, void* dl, int E_pad, int32_t* chunk_off, int G, int64_t chunk, bool bf16,
                    hipStream_t s) {
  if (a.T == 0) return MOE_OK;
  const int nb = (int)((a.T + 3) / 4);
  if (bf16)
    return launch(K_AUX_GRAD, s, "aux_grad", [&] {
      aux_grad_kernel<bf16_t><<<nb, 256, 0, s>>>(a, reinterpret_cast<bf16_t*>(dl), E_pad, chunk_off, G, chunk);
    });
  return launch(K_AUX_GRAD, s, "aux_grad", [&] {
    aux_grad_kernel<float><<<nb, 256, 0, s>>>(a, reinterpret_cast<float*>(dl), E_pad, chunk_off, G, chunk);
  });
}

int launch_aux_dwr(const void* part, int G, int d, int E, int E_pad, bool bf16, float* dw_r, hipStream_t s) {
  const int nb = (int)(((int64_t)d * E + 255) / 256);
  if (bf16)
    return launch(K_AUX_DWR, s, "aux_dwr", [&] {
      aux_dwr_kernel<bf16_t><<<nb, 256, 0, s>>>(reinterpret_cast<const bf16_t*>(part), G, d, E, E_pad, dw_r);
    });
  return launch(K_AUX_DWR, s, "aux_dwr", [&] {
    aux_dwr_kernel<float><<<nb, 256, 0, s>>>(reinterpret_cast<const float*>(part), G, d, E, E_pad, dw_r);
  });
}

}  // namespace moe
