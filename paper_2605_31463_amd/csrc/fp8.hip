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
//                  magnitude of every output column of W [K][N] (blocks of 256
//                  rows, combined by an atomic max), then the codes of W^T [N][K]
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

// Column maxima of W[e] [K][N] (N a multiple of 4): grid (ceil(N / 256),
// ceil(K / 256), E), each lane 4 adjacent columns over 64 rows, the block's
// four wavefronts combined in LDS, the blocks of a column by an integer
// atomic max on the float bits (the values are non-negative), into amax
// cleared by amax_clear_kernel.
__global__ __launch_bounds__(256) void amax_clear_kernel(float* amax, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) amax[i] = 0.f;
}

__global__ __launch_bounds__(256) void col_amax_kernel(const bf16_t* __restrict__ w, int K, int N,
                                                       float* __restrict__ amax) {
  __shared__ float4 part[4][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int n = blockIdx.x * 256 + lane * 4;
  const int e = blockIdx.z;
  const int k0 = blockIdx.y * 256 + wv * 64;
  float4 m = make_float4(0.f, 0.f, 0.f, 0.f);
  if (n < N) {
    const bf16_t* p = w + (int64_t)e * K * N + n;
    const int k1 = min(K, k0 + 64);
    for (int k = k0; k < k1; ++k) {
      const uint2 u = *reinterpret_cast<const uint2*>(p + (int64_t)k * N);
      m.x = fmaxf(m.x, fabsf(__uint_as_float(u.x << 16)));
      m.y = fmaxf(m.y, fabsf(__uint_as_float(u.x & 0xffff0000u)));
      m.z = fmaxf(m.z, fabsf(__uint_as_float(u.y << 16)));
      m.w = fmaxf(m.w, fabsf(__uint_as_float(u.y & 0xffff0000u)));
    }
  }
  part[wv][lane] = m;
  __syncthreads();
  if (wv == 0 && n < N) {
#pragma unroll
    for (int j = 1; j < 4; ++j) {
      const float4 o = part[j][lane];
      m.x = fmaxf(m.x, o.x);
      m.y = fmaxf(m.y, o.y);
      m.z = fmaxf(m.z, o.z);
      m.w = fmaxf(m.w, o.w);
    }
    unsigned int* a = reinterpret_cast<unsigned int*>(amax + (int64_t)e * N + n);
    atomicMax(a + 0, __float_as_uint(m.x));
    atomicMax(a + 1, __float_as_uint(m.y));
    atomicMax(a + 2, __float_as_uint(m.z));
    atomicMax(a + 3, __float_as_uint(m.w));
  }
}

// grid (K / 64, N / 64, E): Q[e][n][k] = code(W[e][k][n] * 448 / amax[e][n])
__global__ __launch_bounds__(256) void quant_transpose_kernel(const bf16_t* __restrict__ w, int K, int N,
                                                              const float* __restrict__ amax,
                                                              uint8_t* __restrict__ q, float* __restrict__ scale) {
  __shared__ float tile[64][65];
  const int k0 = blockIdx.x * 64, n0 = blockIdx.y * 64, e = blockIdx.z;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;  // 64 x 4
  const bf16_t* src = w + (int64_t)e * K * N;
  for (int r = ty; r < 64; r += 4) tile[r][tx] = bf2f(src[(int64_t)(k0 + r) * N + n0 + tx]);
  __syncthreads();
  // thread: one column n (row of Q) and 16 consecutive k
  const int n = threadIdx.x >> 2, kq = (threadIdx.x & 3) * 16;
  const float am = amax[(int64_t)e * N + n0 + n];
  const float inv = e4m3_inv(am);
  if (k0 == 0 && (threadIdx.x & 3) == 0) scale[(int64_t)e * N + n0 + n] = e4m3_scale(am);
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
  const int64_t na = (int64_t)E * N;
  int st = launch(K_WEIGHT_QUANT, s, "weight_quant",
                  [&] { amax_clear_kernel<<<(unsigned)((na + 255) / 256), 256, 0, s>>>(amax, na); });
  if (st) return st;
  const dim3 g1((N + 255) / 256, (K + 255) / 256, E);
  st = launch(K_WEIGHT_QUANT, s, "weight_quant", [&] { col_amax_kernel<<<g1, 256, 0, s>>>(wb, K, N, amax); });
  if (st) return st;
  const dim3 g2(K / 64, N / 64, E);
  return launch(K_WEIGHT_QUANT, s, "weight_quant",
                [&] { quant_transpose_kernel<<<g2, 256, 0, s>>>(wb, K, N, amax, q, scale); });
}

}  // namespace moe
