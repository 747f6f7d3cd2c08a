// Router backward.
//
//   dl      dL/dlogit on the k selected experts of each token from
//           omega = dL/dw (softmax families: w_j (omega_j - sum w omega / c);
//           sigmoid router: (c omega_j - sum w omega) / sum s * s_j (1 - s_j));
//   dW_r    dW_r[:, e] = sum over the rows of expert e of x[token] * dl, using
//           the permutation's expert-contiguous rows: each task sums up to 256
//           rows of one expert in row order into a float32 partial, then a
//           second kernel adds the partials of each expert in task order.
//           No atomics, so dW_r is reproducible bit for bit; the gather reads x
//           (T x d) instead of the k-times larger permuted copy;
//   dx      dx_router[t] = sum_s dl[t][s] * W_r[:, e_s], from a transposed copy
//           of W_r so that the rows are contiguous.
#include "common.h"
#include "kernels.h"

namespace moe {

namespace {

// LDS prefix over experts of ceil(rows_e / DWR_ROWS); pre[e] = first task of
// e, pre[E] = number of tasks.  blockDim.x must be 256 and E <= 256.
__device__ void task_prefix(const int32_t* offsets, int E, int* pre, int* buf) {
  const int tid = threadIdx.x;
  int c = 0;
  if (tid < E) c = (offsets[tid + 1] - offsets[tid] + DWR_ROWS - 1) / DWR_ROWS;
  __shared__ int total;
  const int ex = block_scan_256(c, buf, &total);
  if (tid < E) pre[tid] = ex;
  if (tid == 0) pre[E] = total;
  __syncthreads();
}

__global__ void dl_kernel(RouteBwdArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= a.T) return;
  const int k = a.k;
  const float c = a.route_scale;
  float wo = 0.f;
  for (int s = 0; s < k; ++s) wo += a.topk_w[t * k + s] * a.d_topk_w[t * k + s];
  if (a.router == MOE_ROUTER_SIGMOID_GROUPED || a.router == MOE_ROUTER_SIGMOID_THRESHOLD) {
    float z = 0.f;
    for (int s = 0; s < k; ++s) z += a.s_sel[t * k + s];
    for (int s = 0; s < k; ++s) {
      const float sv = a.s_sel[t * k + s];
      a.dl[t * k + s] = (c * a.d_topk_w[t * k + s] - wo) / z * sv * (1.f - sv);
    }
  } else {
    for (int s = 0; s < k; ++s)
      a.dl[t * k + s] = a.topk_w[t * k + s] * (a.d_topk_w[t * k + s] - wo / c);
  }
}

template <class XT>
__global__ __launch_bounds__(256) void dwr_partial_kernel(RouteBwdArgs a, const float* __restrict__ dl) {
  __shared__ int pre[257];
  __shared__ int sbuf[256];
  __shared__ int tok[DWR_ROWS];
  __shared__ float g[DWR_ROWS];
  task_prefix(a.offsets, a.E, pre, sbuf);
  const int task = blockIdx.x;
  if (task >= pre[a.E]) return;
  int lo = 0, hi = a.E - 1;  // last e with pre[e] <= task
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pre[mid] <= task) lo = mid; else hi = mid - 1;
  }
  const int e = lo;
  const int r0 = a.offsets[e] + (task - pre[e]) * DWR_ROWS;
  const int r1 = min(a.offsets[e + 1], r0 + DWR_ROWS);
  const int n = r1 - r0;
  for (int i = threadIdx.x; i < n; i += 256) {
    const int ts = a.token_of[r0 + i];
    tok[i] = ts / a.k;
    g[i] = dl[ts];
  }
  __syncthreads();
  constexpr int V = Vec16<XT>::N;
  const XT* x = reinterpret_cast<const XT*>(a.x);
  const int nch = a.d / V;
  for (int c = threadIdx.x; c < nch; c += 256) {
    float acc[V];
#pragma unroll
    for (int v = 0; v < V; ++v) acc[v] = 0.f;
    // eight rows' loads in flight per thread (unrolled by 4: DeepSeek-V3
    // shape 154 us, by 16: 197 us; by 8: 141 us, Qwen3 48 -> 38)
#pragma unroll 8
    for (int i = 0; i < n; ++i) {
      float xv[V];
      Vec16<XT>::load(x + (int64_t)tok[i] * a.d + (int64_t)c * V, xv);
#pragma unroll
      for (int v = 0; v < V; ++v) acc[v] = __builtin_fmaf(xv[v], g[i], acc[v]);
    }
    float* out = a.partial + (int64_t)task * a.d + (int64_t)c * V;
#pragma unroll
    for (int v = 0; v < V; ++v) out[v] = acc[v];
  }
}

// dW_r[i][e] = sum of the partials of expert e (task order); grid (E, d/256)
__global__ __launch_bounds__(256) void dwr_reduce_kernel(RouteBwdArgs a) {
  __shared__ int pre[257];
  __shared__ int sbuf[256];
  task_prefix(a.offsets, a.E, pre, sbuf);
  const int e = blockIdx.x;
  const int i = blockIdx.y * 256 + threadIdx.x;
  if (i >= a.d) return;
  float acc = 0.f;
  for (int q = pre[e]; q < pre[e + 1]; ++q) acc += a.partial[(int64_t)q * a.d + i];
  float* o = a.dw_r + (int64_t)i * a.E + e;
  *o = a.accumulate ? *o + acc : acc;
}

// wt [Eo][d] = w^T for rows e < E, zero for E <= e < Eo.
template <class OT>
__global__ void transpose_kernel(const float* __restrict__ w, OT* __restrict__ wt, int d, int E, int Eo) {
  __shared__ float tile[32][33];
  const int e0 = blockIdx.x * 32, i0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 256 threads: 32 x 8
  for (int r = ty; r < 32; r += 8) {
    const int i = i0 + r, e = e0 + tx;
    tile[r][tx] = (i < d && e < E) ? w[(int64_t)i * E + e] : 0.f;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int e = e0 + r, i = i0 + tx;
    if (e < Eo && i < d) Elem<OT>::store(wt, (int64_t)e * d + i, tile[tx][r]);
  }
}

__global__ __launch_bounds__(256) void dx_router_kernel(RouteBwdArgs a, const float* __restrict__ dl) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= a.T) return;
  const int k = a.k;
  for (int i = lane * 4; i < a.d; i += 256) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s = 0; s < k; ++s) {
      const int e = a.topk_idx[t * k + s];
      if ((unsigned)e >= (unsigned)a.E) continue;  // an empty slot (threshold router)
      const float g = dl[t * k + s];
      const float4 w = *reinterpret_cast<const float4*>(a.w_rt + (int64_t)e * a.d + i);
      acc.x = __builtin_fmaf(g, w.x, acc.x);
      acc.y = __builtin_fmaf(g, w.y, acc.y);
      acc.z = __builtin_fmaf(g, w.z, acc.z);
      acc.w = __builtin_fmaf(g, w.w, acc.w);
    }
    *reinterpret_cast<float4*>(a.dx_router + t * a.d + i) = acc;
  }
}

// dtheta[e] (+)= sum over the rows of expert e of g[token_of[row]], each
// expert's rows summed by one block in a fixed order (strided per thread,
// then a fixed tree).
__global__ __launch_bounds__(256) void threshold_reduce_kernel(const int32_t* __restrict__ offsets,
                                                              const int32_t* __restrict__ token_of,
                                                              const float* __restrict__ g, float* dtheta,
                                                              bool accumulate) {
  __shared__ float red[256];
  const int e = blockIdx.x;
  const int r0 = offsets[e], r1 = offsets[e + 1];
  float acc = 0.f;
  for (int r = r0 + (int)threadIdx.x; r < r1; r += 256) acc += g[token_of[r]];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) dtheta[e] = accumulate ? dtheta[e] + red[0] : red[0];
}

}  // namespace

int launch_wr_transpose(const float* w_r, float* w_rt, int d, int E, hipStream_t s) {
  dim3 grid((E + 31) / 32, (d + 31) / 32);
  return launch(K_WR_TRANSPOSE, s, "wr_transpose",
                [&] { transpose_kernel<float><<<grid, 256, 0, s>>>(w_r, w_rt, d, E, E); });
}

int launch_wr_transpose_act(const float* w_r, void* w_rt, int d, int E, int Eo, bool bf16, hipStream_t s) {
  dim3 grid((Eo + 31) / 32, (d + 31) / 32);
  if (!bf16) {
    float* o = reinterpret_cast<float*>(w_rt);
    return launch(K_WR_TRANSPOSE, s, "wr_transpose",
                  [&] { transpose_kernel<float><<<grid, 256, 0, s>>>(w_r, o, d, E, Eo); });
  }
  bf16_t* o = reinterpret_cast<bf16_t*>(w_rt);
  return launch(K_WR_TRANSPOSE, s, "wr_transpose",
                [&] { transpose_kernel<bf16_t><<<grid, 256, 0, s>>>(w_r, o, d, E, Eo); });
}

int launch_threshold_grad(const int32_t* offsets, const int32_t* token_of, const float* g, int E, float* dtheta,
                          bool accumulate, hipStream_t s) {
  return launch(K_THRESHOLD_GRAD, s, "threshold_grad", [&] {
    threshold_reduce_kernel<<<E, 256, 0, s>>>(offsets, token_of, g, dtheta, accumulate);
  });
}

int launch_route_bwd(const RouteBwdArgs& a, hipStream_t s) {
  int st;
  const float* dl = a.dl_in;
  if (!dl) {
    if (a.T > 0) {
      st = launch(K_ROUTE_DL, s, "route_dl", [&] { dl_kernel<<<(int)((a.T + 255) / 256), 256, 0, s>>>(a); });
      if (st) return st;
    }
    dl = a.dl;
  }
  const int64_t tasks = route_dwr_tasks(a.T * a.k, a.E);
  if (tasks > 0 && a.T > 0) {
    if (a.bf16)
      st = launch(K_ROUTE_DWR_PARTIAL, s, "dwr_partial",
                  [&] { dwr_partial_kernel<bf16_t><<<(int)tasks, 256, 0, s>>>(a, dl); });
    else
      st = launch(K_ROUTE_DWR_PARTIAL, s, "dwr_partial",
                  [&] { dwr_partial_kernel<float><<<(int)tasks, 256, 0, s>>>(a, dl); });
    if (st) return st;
  }
  dim3 rg(a.E, (a.d + 255) / 256);
  st = launch(K_ROUTE_DWR_REDUCE, s, "dwr_reduce", [&] { dwr_reduce_kernel<<<rg, 256, 0, s>>>(a); });
  if (st) return st;
  if (a.dx_router && a.T > 0) {
    st = launch_wr_transpose(a.w_r, a.w_rt, a.d, a.E, s);
    if (st) return st;
    st = launch(K_ROUTE_DX, s, "dx_router",
                [&] { dx_router_kernel<<<(int)((a.T + 3) / 4), 256, 0, s>>>(a, dl); });
    if (st) return st;
  }
  return MOE_OK;
}

}  // namespace moe
