// Parameter gradients of the constant zero-computation experts (MoE++,
// appendix B.3).  A constant expert c returns a0 x + a1 v_c with
// (a0, a1) = softmax(W_c x); the combine backward leaves per slot
// (dz0, dz1, w a1) with dz the gradient at W_c x.  Summed over the slots that
// chose c:
//   dW_c[c][j] = sum dz_j x_t,    dv[c] = sum (w a1) dy_t.
// The permutation lists the tokens of every pool expert in its rows, so the
// sums run over the rows of each constant expert: tasks of up to DWR_ROWS
// rows of one expert write float32 partials [3][d], and a second kernel adds
// each expert's partials in task order.  No atomics: bitwise reproducible.
#include "common.h"
#include "kernels.h"

namespace moe {

namespace {

// LDS prefix over the constant experts of ceil(rows / DWR_ROWS); pre[c] =
// first task of c, pre[n] = number of tasks.  blockDim.x = 256, n <= 256.
__device__ void zc_task_prefix(const ZcParamArgs& a, int* pre, int* buf) {
  const int tid = threadIdx.x;
  int c = 0;
  if (tid < a.n_const) {
    const int e = a.e0 + tid;
    c = (a.offsets[e + 1] - a.offsets[e] + DWR_ROWS - 1) / DWR_ROWS;
  }
  __shared__ int total;
  const int ex = block_scan_256(c, buf, &total);
  if (tid < a.n_const) pre[tid] = ex;
  if (tid == 0) pre[a.n_const] = total;
  __syncthreads();
}

template <class XT>
__global__ __launch_bounds__(256) void zc_param_partial_kernel(ZcParamArgs a) {
  __shared__ int pre[257];
  __shared__ int sbuf[256];
  __shared__ int tok[DWR_ROWS];
  __shared__ float4 cf[DWR_ROWS];
  zc_task_prefix(a, pre, sbuf);
  const int task = blockIdx.x;
  if (task >= pre[a.n_const]) return;
  int lo = 0, hi = a.n_const - 1;  // last c with pre[c] <= task
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pre[mid] <= task) lo = mid; else hi = mid - 1;
  }
  const int e = a.e0 + lo;
  const int r0 = a.offsets[e] + (task - pre[lo]) * DWR_ROWS;
  const int r1 = min(a.offsets[e + 1], r0 + DWR_ROWS);
  const int n = r1 - r0;
  for (int i = threadIdx.x; i < n; i += 256) {
    const int ts = a.token_of[r0 + i];
    tok[i] = ts / a.k;
    cf[i] = a.coef[ts];
  }
  __syncthreads();
  constexpr int V = Vec16<XT>::N;
  const XT* x = reinterpret_cast<const XT*>(a.x);
  const XT* dy = reinterpret_cast<const XT*>(a.dy);
  const int nch = a.d / V;
  for (int c = threadIdx.x; c < nch; c += 256) {
    float s0[V], s1[V], s2[V];
#pragma unroll
    for (int v = 0; v < V; ++v) s0[v] = s1[v] = s2[v] = 0.f;
#pragma unroll 2
    for (int i = 0; i < n; ++i) {
      float xv[V], gv[V];
      const int64_t off = (int64_t)tok[i] * a.d + (int64_t)c * V;
      Vec16<XT>::load(x + off, xv);
      Vec16<XT>::load(dy + off, gv);
      const float4 q = cf[i];
#pragma unroll
      for (int v = 0; v < V; ++v) {
        s0[v] = __builtin_fmaf(q.x, xv[v], s0[v]);
        s1[v] = __builtin_fmaf(q.y, xv[v], s1[v]);
        s2[v] = __builtin_fmaf(q.z, gv[v], s2[v]);
      }
    }
    float* out = a.partial + (int64_t)task * 3 * a.d + (int64_t)c * V;
#pragma unroll
    for (int v = 0; v < V; ++v) {
      out[v] = s0[v];
      out[a.d + v] = s1[v];
      out[2 * a.d + v] = s2[v];
    }
  }
}

// grid (n_const, ceil(d / 256)): each constant expert's partials in task order
__global__ __launch_bounds__(256) void zc_param_reduce_kernel(ZcParamArgs a) {
  __shared__ int pre[257];
  __shared__ int sbuf[256];
  zc_task_prefix(a, pre, sbuf);
  const int c = blockIdx.x;
  const int i = blockIdx.y * 256 + threadIdx.x;
  if (i >= a.d) return;
  float s0 = 0.f, s1 = 0.f, s2 = 0.f;
  for (int q = pre[c]; q < pre[c + 1]; ++q) {
    const float* p = a.partial + (int64_t)q * 3 * a.d + i;
    s0 += p[0];
    s1 += p[a.d];
    s2 += p[2 * a.d];
  }
  float* w0 = a.dwc + (int64_t)c * 2 * a.d + i;
  float* w1 = w0 + a.d;
  float* dv = a.dv + (int64_t)c * a.d + i;
  *w0 = a.accumulate ? *w0 + s0 : s0;
  *w1 = a.accumulate ? *w1 + s1 : s1;
  *dv = a.accumulate ? *dv + s2 : s2;
}

}  // namespace

int launch_zc_param_grads(const ZcParamArgs& a, hipStream_t s) {
  if (a.n_const <= 0) return MOE_OK;
  const int64_t tasks = route_dwr_tasks(a.T * a.k, a.n_const);
  if (a.T > 0 && tasks > 0) {
    const int st = a.bf16 ? launch(K_ZC_PARAM_PARTIAL, s, "zc_param_partial",
                                   [&] { zc_param_partial_kernel<bf16_t><<<(int)tasks, 256, 0, s>>>(a); })
                          : launch(K_ZC_PARAM_PARTIAL, s, "zc_param_partial",
                                   [&] { zc_param_partial_kernel<float><<<(int)tasks, 256, 0, s>>>(a); });
    if (st) return st;
  }
  const dim3 grid(a.n_const, (a.d + 255) / 256);
  return launch(K_ZC_PARAM_REDUCE, s, "zc_param_reduce", [&] { zc_param_reduce_kernel<<<grid, 256, 0, s>>>(a); });
}

}  // namespace moe
