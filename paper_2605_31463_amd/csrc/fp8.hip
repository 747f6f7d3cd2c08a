// FP8 (OCP E4M3) operands of the expert GEMMs.
//
//   quant_rows     E4M3 rows with one scale per row (the row's largest
//                  magnitude / 448), one wavefront per row.  A row is the
//                  concatenation of a row of s0 (w0 values) and a row of s1
//                  (w1 values, possibly none): activation rows of h, d_o or
//                  [dg | du] (only the rows of the FFN experts, below
//                  offsets[E]) and, for the data-gradient GEMMs, the weight
//                  rows of W_down and of [W_gate | W_up] (one scale over both);
//   weight quant   the forward's weight cache: per expert, the largest
//                  magnitude of every output column of W [K][N] (one thread per
//                  column, rows read in order), then the codes of W^T [N][K]
//                  (64 x 64 tiles through LDS, so that both the bf16 reads and
//                  the code writes are contiguous).  The GEMMs read both
//                  operands K-contiguous.
// A value v of a row (column) with largest magnitude amax is stored as the
// E4M3 code nearest to clamp(v * (448 / amax)), the product in float32.
#include "common.h"
#include "kernels.h"

namespace moe {

namespace {

struct QuantRowsArgs {
  const bf16_t* s0;
  const bf16_t* s1;
  int w0, w1;
  const int32_t* offsets;  // non-null: rows at or past offsets[E] are skipped
  int E;
  int64_t rows;
  uint8_t* q;  // [rows][w0 + w1]
  float* scale;  // [rows]
};

__global__ __launch_bounds__(256) void quant_rows_kernel(QuantRowsArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  if (r >= a.rows || (a.offsets && r >= a.offsets[a.E])) return;
  const int n0 = a.w0 / 8, nch = (a.w0 + a.w1) / 8;
  auto src = [&](int c) {
    return c < n0 ? a.s0 + r * a.w0 + (int64_t)c * 8 : a.s1 + r * a.w1 + (int64_t)(c - n0) * 8;
  };
  auto put = [&](int c, const float* v, float inv) {
    *reinterpret_cast<uint2*>(a.q + r * (a.w0 + a.w1) + (int64_t)c * 8) =
        make_uint2(e4m3x4(v[0] * inv, v[1] * inv, v[2] * inv, v[3] * inv),
                   e4m3x4(v[4] * inv, v[5] * inv, v[6] * inv, v[7] * inv));
  };
  float m = 0.f;
  constexpr int HOLD = 4;  // rows of up to 64 * HOLD chunks stay in registers between the passes
  if (nch <= 64 * HOLD) {
    float v[HOLD][8];
#pragma unroll
    for (int j = 0; j < HOLD; ++j) {
      const int c = lane + 64 * j;
      if (c < nch) {
        Vec16<bf16_t>::load(src(c), v[j]);
#pragma unroll
        for (int q = 0; q < 8; ++q) m = fmaxf(m, fabsf(v[j][q]));
      }
    }
    m = wave_max(m);
    const float inv = e4m3_inv(m);
#pragma unroll
    for (int j = 0; j < HOLD; ++j)
      if (lane + 64 * j < nch) put(lane + 64 * j, v[j], inv);
  } else {
    for (int c = lane; c < nch; c += 64) {
      float v[8];
      Vec16<bf16_t>::load(src(c), v);
#pragma unroll
      for (int q = 0; q < 8; ++q) m = fmaxf(m, fabsf(v[q]));
    }
    m = wave_max(m);
    const float inv = e4m3_inv(m);
    for (int c = lane; c < nch; c += 64) {
      float v[8];
      Vec16<bf16_t>::load(src(c), v);
      put(c, v, inv);
    }
  }
  if (lane == 0) a.scale[r] = e4m3_scale(m);
}

// grid (ceil(N / 256), E): column maxima over the K rows of W[e]
__global__ __launch_bounds__(256) void col_amax_kernel(const bf16_t* __restrict__ w, int K, int N,
                                                       float* __restrict__ amax, float* __restrict__ scale) {
  const int n = blockIdx.x * 256 + threadIdx.x;
  const int e = blockIdx.y;
  if (n >= N) return;
  const bf16_t* p = w + (int64_t)e * K * N + n;
  float m = 0.f;
  for (int k = 0; k < K; ++k) m = fmaxf(m, fabsf(bf2f(p[(int64_t)k * N])));
  amax[(int64_t)e * N + n] = m;
  scale[(int64_t)e * N + n] = e4m3_scale(m);
}

// grid (K / 64, N / 64, E): Q[e][n][k] = code(W[e][k][n] * 448 / amax[e][n])
__global__ __launch_bounds__(256) void quant_transpose_kernel(const bf16_t* __restrict__ w, int K, int N,
                                                              const float* __restrict__ amax,
                                                              uint8_t* __restrict__ q) {
  __shared__ float tile[64][65];
  const int k0 = blockIdx.x * 64, n0 = blockIdx.y * 64, e = blockIdx.z;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;  // 64 x 4
  const bf16_t* src = w + (int64_t)e * K * N;
  for (int r = ty; r < 64; r += 4) tile[r][tx] = bf2f(src[(int64_t)(k0 + r) * N + n0 + tx]);
  __syncthreads();
  // thread: one column n (row of Q) and 16 consecutive k
  const int n = threadIdx.x >> 2, kq = (threadIdx.x & 3) * 16;
  const float inv = e4m3_inv(amax[(int64_t)e * N + n0 + n]);
  uint32_t c[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    c[j] = e4m3x4(tile[kq + 4 * j][n] * inv, tile[kq + 4 * j + 1][n] * inv, tile[kq + 4 * j + 2][n] * inv,
                  tile[kq + 4 * j + 3][n] * inv);
  *reinterpret_cast<uint4*>(q + ((int64_t)e * N + n0 + n) * K + k0 + kq) = make_uint4(c[0], c[1], c[2], c[3]);
}

}  // namespace

int launch_quant_rows(const void* s0, const void* s1, int w0, int w1, const int32_t* offsets, int E, int64_t rows,
                      uint8_t* q, float* scale, hipStream_t s) {
  if (rows <= 0) return MOE_OK;
  QuantRowsArgs a{reinterpret_cast<const bf16_t*>(s0), reinterpret_cast<const bf16_t*>(s1), w0, w1, offsets, E,
                  rows, q, scale};
  const int64_t nb = (rows + 3) / 4;
  return launch(K_QUANT_ROWS, s, "quant_rows", [&] { quant_rows_kernel<<<(unsigned)nb, 256, 0, s>>>(a); });
}

int launch_weight_quant(const void* w, int E, int K, int N, float* amax, float* scale, uint8_t* q, hipStream_t s) {
  const bf16_t* wb = reinterpret_cast<const bf16_t*>(w);
  const dim3 g1((N + 255) / 256, E);
  int st = launch(K_WEIGHT_QUANT, s, "weight_quant", [&] { col_amax_kernel<<<g1, 256, 0, s>>>(wb, K, N, amax, scale); });
  if (st) return st;
  const dim3 g2(K / 64, N / 64, E);
  return launch(K_WEIGHT_QUANT, s, "weight_quant",
                [&] { quant_transpose_kernel<<<g2, 256, 0, s>>>(wb, K, N, amax, q); });
}

}  // namespace moe
