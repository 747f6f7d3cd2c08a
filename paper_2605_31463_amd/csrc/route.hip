// Router forward: logits, top-k selection, gating weights, expert counts.
//
// Three paths, all computing:
//   1. logits l = x W_r for every token and expert, accurate enough (float32
//      partial sums folded into float64) that the float64 selection keys
//      order experts the way an exact evaluation does outside sub-1e-6
//      near-ties;
//   2. top-k over the selection keys with one wavefront per token and 64-lane
//      butterfly reductions (the framework's top-k routing kernel, section
//      3.2 / appendix B.3), optionally restricted to the best expert groups
//      (group score = sum of the group's two largest keys);
//   3. gating weights over the selected experts: softmax of the selected
//      (biased) logits, or route_scale * sigmoid / sum of sigmoids; weights
//      are non-negative and sum to route_scale (appendix B.2.2 rules);
//   4. per-block expert histograms added into the expert counts.
// bf16 activations with E a multiple of 32: a tiled MFMA logits GEMM into a
// float64 workspace, then a selection kernel.  Other bf16 cases: one fused
// MFMA kernel per block of tokens.  float32: one fused kernel of float32 FMA
// chains of 16 terms folded into float64.
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

// Top-k selection and gating weights for `ntok` tokens whose float64 logits
// sit in LDS (lg[token][ld]); one wavefront per token, four wavefronts per
// block.  Adds each selected expert to the block histogram `hist`.
// sel (may be null): [16][16] LDS, the expert of (token tl, slot s) at
// 16 tl + s (-1: none)
__device__ void select_tokens(const RouteArgs& a, const double* lg, int ld, int64_t t0, int ntok, int* hist,
                              int* sel = nullptr) {
  const int tid = threadIdx.x;
  const int E = a.E;
  const int EPAD = ld;
  const int TB = ntok;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int epl = (E + 63) / 64;              // experts per lane, contiguous
  // threshold router: key l - theta_e, weights from sigmoid scores
  const bool thr = a.router == MOE_ROUTER_SIGMOID_THRESHOLD;
  const bool sigm = a.router == MOE_ROUTER_SIGMOID_GROUPED || thr;
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
        double sc = (sigm && !thr) ? 1.0 / (1.0 + exp(-l)) : l;
        const double kv = thr ? l - (double)a.threshold[e] : select_bias ? sc + (double)a.bias[e] : sc;
        key[q] = isnan(kv) ? -INFINITY : kv;  // NaN orders below every number
      }
    }
    if (a.probs && thr) {
      // threshold router: the sigmoid scores of all experts (the auxiliary
      // loss normalises them per token)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = lane * epl + q;
        if (q < epl && e < E) a.probs[t * E + e] = (float)(1.0 / (1.0 + exp(-lg[tl * EPAD + e])));
      }
    } else if (a.probs) {
      // the router's probabilities over all experts (auxiliary loss): softmax
      // of the logits (+ bias when it is added to the logits)
      double v[4];
      double m = -INFINITY;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = lane * epl + q;
        v[q] = -INFINITY;
        if (q < epl && e < E) {
          double l = lg[tl * EPAD + e];
          if (logit_bias) l += (double)a.bias[e];
          v[q] = l;
          m = fmax(m, l);
        }
      }
      m = wave_max_d(m, 64);
      double z = 0.0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = lane * epl + q;
        if (q < epl && e < E) {
          v[q] = exp(v[q] - m);
          z += v[q];
        }
      }
      z = wave_sum_d(z, 64);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = lane * epl + q;
        if (q < epl && e < E) a.probs[t * E + e] = (float)(v[q] / z);
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
    double my_key = -INFINITY;
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
      if (lane == s) {
        my_idx = c.idx;
        my_key = c.key;
      }
    }
    // weights over the k selected (lanes 0..k-1 hold one slot each); the
    // threshold router keeps the slots whose key is positive, and always the
    // first: the rest become empty (-1)
    const bool holds = lane < k;
    const bool active = holds && (!thr || lane == 0 || my_key > 0.0);
    double sc = 0.0;
    if (active) {
      double l = lg[tl * EPAD + my_idx];
      if (logit_bias) l += (double)a.bias[my_idx];
      sc = sigm ? 1.0 / (1.0 + exp(-l)) : l;
    }
    double w;
    if (sigm) {
      const double z = wave_sum_d(active ? sc : 0.0, 64);
      w = (double)a.route_scale * sc / z;
    } else {
      const double m = wave_max_d(holds ? sc : -INFINITY, 64);
      const double p = holds ? exp(sc - m) : 0.0;
      const double z = wave_sum_d(p, 64);
      w = (double)a.route_scale * p / z;
    }
    if (active) {
      a.topk_idx[t * k + lane] = my_idx;
      a.topk_w[t * k + lane] = (float)w;
      if (sigm && a.s_sel) a.s_sel[t * k + lane] = (float)sc;
      atomicAdd(&hist[my_idx], 1);
      if (sel && tl < 16) sel[tl * 16 + lane] = my_idx;
    } else if (holds) {
      a.topk_idx[t * k + lane] = -1;
      a.topk_w[t * k + lane] = 0.f;
      if (a.s_sel) a.s_sel[t * k + lane] = 0.f;
    }
  }
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

  select_tokens(a, lg, EPAD, t0, TB, hist);
  __syncthreads();
  if (a.counts) {
    for (int e = tid; e < E; e += 256)
      if (hist[e]) atomicAdd(&a.counts[e], hist[e]);
  }
}


// ---------------------------------------------------------------------------
// bf16 path: logits on MFMA.
//
// W_r (float32) is split once per call into three bf16 terms,
// w = w1 + w2 + w3 with w1 = bf16(w), w2 = bf16(w - w1), w3 = bf16(w - w1 - w2),
// stored expert-major ([3][E][d]).  x is bf16, so every product x * w_i is exact
// in float32; v_mfma_f32_16x16x32_bf16 sums them, and the float32 partial sums
// are folded into float64 accumulators every 64 hidden elements.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// The launch also clears what the selection then accumulates into: the
// expert counts (nz0), the permutation's per-block counts (nz1) and the
// selection's arrival counter (nz2); pointers may be null.
__global__ void wr_split_kernel(const float* __restrict__ w, bf16_t* __restrict__ ws, int d, int E,
                                int32_t* z0, int nz0, int32_t* z1, int64_t nz1, int32_t* z2, int nz2) {
  {
    const int64_t nth = (int64_t)gridDim.x * gridDim.y * blockDim.x;
    const int64_t g = ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * blockDim.x + threadIdx.x;
    for (int64_t i = g; i < nz0; i += nth) z0[i] = 0;
    for (int64_t i = g; i < nz1; i += nth) z1[i] = 0;
    for (int64_t i = g; i < nz2; i += nth) z2[i] = 0;
  }
  __shared__ float tile[32][33];
  const int e0 = blockIdx.x * 32, i0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int r = ty; r < 32; r += 8) {
    const int i = i0 + r, e = e0 + tx;
    tile[r][tx] = (i < d && e < E) ? w[(int64_t)i * E + e] : 0.f;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int e = e0 + r, i = i0 + tx;
    if (e < E && i < d) {
      const float v = tile[tx][r];
      const bf16_t p1 = f2bf(v);
      const float r1 = v - bf2f(p1);
      const bf16_t p2 = f2bf(r1);
      const float r2 = r1 - bf2f(p2);
      const bf16_t p3 = f2bf(r2);
      const int64_t o = (int64_t)e * d + i;
      ws[o] = p1;
      ws[(int64_t)E * d + o] = p2;
      ws[2 * (int64_t)E * d + o] = p3;
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 path, large expert counts: logits as a tiled GEMM, then a selection
// kernel.  The logits kernel's workgroup tile is TT tokens x TE experts; K = d
// advances in stages of 64 copied global -> LDS without registers (x rows and
// the three bf16 parts of W_r, all K-contiguous 128-byte rows with the 16-byte
// chunk index XOR-swizzled by (row >> 1) & 7).  One wavefront per 16 tokens
// runs v_mfma_f32_16x16x32_bf16 over the three parts into one float32
// accumulator per 16 x 16 block (every product x * w_i is exact in float32)
// and folds it into float64 after every stage, as the fused kernel does.
// The expert tiles of one token tile are consecutive in the XCD-contiguous
// order, so the token rows are fetched from HBM once.
// ---------------------------------------------------------------------------
template <int TT, int TE>
__global__ __launch_bounds__(TT * 4) void route_logits_kernel(RouteArgs a) {
  constexpr int NW = TT / 16;
  constexpr int KC = 64, S = 3;
  constexpr int XROWS = TT, WROWS = 3 * TE;
  constexpr int STAGE = (XROWS + WROWS) * KC;  // bf16 elements
  constexpr int NI = (XROWS + WROWS) / 8;      // 1 KB copies per stage
  static_assert(NI % NW == 0, "every wavefront issues the same number of copies");
  constexpr int NIW = NI / NW;
  constexpr int NJ = TE / 16;
  __shared__ __align__(16) bf16_t st[S][STAGE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int E = a.E, d = a.d;
  const int net = E / TE;
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int tt = lin / net, et = lin - tt * net;
  const int64_t t0 = (int64_t)tt * TT;
  const int e0 = et * TE;
  const bf16_t* x = reinterpret_cast<const bf16_t*>(a.x);
  const bf16_t* wsp = reinterpret_cast<const bf16_t*>(a.wsplit);
  const int32x4_t rx = make_rsrc(x + t0 * d, (a.T - t0) * d * 2);  // rows past T read as zeros
  const int32x4_t rw = make_rsrc(wsp, (int64_t)3 * E * d * 2);
  uint32_t voff[NIW];
  bool isx[NIW];
#pragma unroll
  for (int j = 0; j < NIW; ++j) {
    const int q = (NIW * wave + j) * 64 + lane;
    const int row = q >> 3, c = (q & 7) ^ ((row >> 1) & 7);
    isx[j] = 8 * (NIW * wave + j) < XROWS;  // whole copies fall in one part
    if (row < XROWS) {
      voff[j] = (uint32_t)(((int64_t)row * d + 8 * c) * 2);
    } else {
      const int wr = row - XROWS, p = wr / TE, e = wr - p * TE;
      voff[j] = (uint32_t)((((int64_t)p * E + e0 + e) * d + 8 * c) * 2);
    }
  }
  const uint32_t lds0 = lds_addr(&st[0][0]);
  auto issue = [&](int kt) {
    const uint32_t base = lds0 + (kt % S) * STAGE * 2;
#pragma unroll
    for (int j = 0; j < NIW; ++j)
      dma16(isx[j] ? rx : rw, base + (NIW * wave + j) * 1024, voff[j], (uint32_t)(kt * KC * 2));
  };

  floatx4 acc[NJ];
  double acc64[NJ][4];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int v = 0; v < 4; ++v) acc64[j][v] = 0.0;
  }
  const int nk = d / KC;
#pragma unroll
  for (int p = 0; p < S - 1; ++p)
    if (p < nk) issue(p);
  const int arow = wave * 16 + (lane & 15);
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) wait_vmcnt<(S - 2) * NIW>();
    else wait_vmcnt<0>();
    __syncthreads();
    if (kt + S - 1 < nk) issue(kt + S - 1);
    const bf16_t* sx = st[kt % S];
    const bf16_t* sw = sx + XROWS * KC;
#pragma unroll
    for (int ks = 0; ks < KC / 32; ++ks) {
      const int c = ks * 4 + (lane >> 4);
      const bf16x8 af = *reinterpret_cast<const bf16x8*>(sx + arow * KC + ((c ^ ((arow >> 1) & 7)) << 3));
#pragma unroll
      for (int p = 0; p < 3; ++p)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int br = p * TE + 16 * j + (lane & 15);
          const bf16x8 bfr = *reinterpret_cast<const bf16x8*>(sw + br * KC + ((c ^ ((br >> 1) & 7)) << 3));
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bfr, acc[j], 0, 0, 0);
        }
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
#pragma unroll
      for (int v = 0; v < 4; ++v) acc64[j][v] += (double)acc[j][v];
      acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
  }
  // D block (j): lane holds tokens 4 (lane / 16) + v, expert 16 j + lane % 16
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t t = t0 + wave * 16 + 4 * (lane >> 4) + v;
      if (t < a.T) a.lg[t * E + e0 + 16 * j + (lane & 15)] = acc64[j][v];
    }
}

// ---------------------------------------------------------------------------
// Selection with one DPP row (16 lanes) per token: the same decisions as
// select_tokens (float64 keys, ties to the lower index, NaN below every
// number, group limit by the sum of a group's two best keys), with the
// reductions as DPP moves inside the row instead of 64-lane shuffles through
// LDS, and four tokens per wavefront side by side.
// ---------------------------------------------------------------------------
// DPP controls: quad permutations lane ^ 1 and lane ^ 2, the row half mirror
// (lane i <-> 7 - i within each 8 lanes) and the row mirror (i <-> 15 - i).
// Applied in this order they pair aligned groups of 2, 4, 8, 16 lanes.
constexpr int DPP_QXOR1 = 0xB1, DPP_QXOR2 = 0x4E, DPP_HMIRROR = 0x141, DPP_MIRROR = 0x140;

template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) { return __builtin_amdgcn_mov_dpp(v, CTRL, 0xf, 0xf, false); }
template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = dpp_i<CTRL>((int)(b & 0xffffffffll));
  const int hi = dpp_i<CTRL>((int)(b >> 32));
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}
template <int CTRL>
__device__ __forceinline__ void dpp_best_step(double& k, int& i) {
  const double ok = dpp_d<CTRL>(k);
  const int oi = dpp_i<CTRL>(i);
  if (better(ok, oi, k, i)) {
    k = ok;
    i = oi;
  }
}
// best (key, index) over aligned groups of 2^levels lanes of the row
__device__ __forceinline__ void dpp_best(double& k, int& i, int levels) {
  if (levels > 0) dpp_best_step<DPP_QXOR1>(k, i);
  if (levels > 1) dpp_best_step<DPP_QXOR2>(k, i);
  if (levels > 2) dpp_best_step<DPP_HMIRROR>(k, i);
  if (levels > 3) dpp_best_step<DPP_MIRROR>(k, i);
}
__device__ __forceinline__ double dpp_row_sum(double v) {
  v += dpp_d<DPP_QXOR1>(v);
  v += dpp_d<DPP_QXOR2>(v);
  v += dpp_d<DPP_HMIRROR>(v);
  v += dpp_d<DPP_MIRROR>(v);
  return v;
}
__device__ __forceinline__ double dpp_row_max(double v) {
  v = fmax(v, dpp_d<DPP_QXOR1>(v));
  v = fmax(v, dpp_d<DPP_QXOR2>(v));
  v = fmax(v, dpp_d<DPP_HMIRROR>(v));
  v = fmax(v, dpp_d<DPP_MIRROR>(v));
  return v;
}
// top-2 of (m1, m2) pairs over aligned groups of 2^levels lanes
template <int CTRL>
__device__ __forceinline__ void dpp_top2_step(double& m1, double& m2) {
  const double o1 = dpp_d<CTRL>(m1), o2 = dpp_d<CTRL>(m2);
  const double n1 = fmax(m1, o1);
  m2 = fmax(fmin(m1, o1), fmax(m2, o2));
  m1 = n1;
}

// KPL = E / 16 experts per lane (contiguous); E <= 256.  Needs, with a group
// limit, groups of a whole power-of-two number of lanes.
template <int KPL>
__device__ void select_tokens16(const RouteArgs& a, const double* lg, int ld, int64_t t0, int ntok, int* hist,
                                int* sel = nullptr) {
  const int tid = threadIdx.x;
  const int E = a.E;
  const int lane = tid & 63, sub = lane & 15;
  const int tl = (tid >> 6) * 4 + (lane >> 4);  // this row's token within the block
  const int64_t t = t0 + tl;
  const bool valid = tl < ntok && t < a.T;   // rows past the end compute on -inf keys, store nothing
  const bool sigm = a.router == MOE_ROUTER_SIGMOID_GROUPED;
  const bool logit_bias = a.bias_mode == MOE_BIAS_LOGIT;
  const bool select_bias = a.bias_mode == MOE_BIAS_SELECT_ONLY;
  const int k = a.k;
  const int e0 = sub * KPL;
  double lv[KPL], key[KPL];
  unsigned avail = 0;
#pragma unroll
  for (int q = 0; q < KPL; ++q) {
    double l = valid ? lg[(int64_t)tl * ld + e0 + q] : 0.0;
    if (logit_bias) l += (double)a.bias[e0 + q];
    lv[q] = l;
    const double sc = sigm ? 1.0 / (1.0 + exp(-l)) : l;
    const double kv = select_bias ? sc + (double)a.bias[e0 + q] : sc;
    key[q] = (!valid || isnan(kv)) ? -INFINITY : kv;  // NaN orders below every number
    avail |= 1u << q;
  }
  if (a.probs) {
    // the router's probabilities over all experts (auxiliary loss)
    double m = -INFINITY;
#pragma unroll
    for (int q = 0; q < KPL; ++q) m = fmax(m, lv[q]);
    m = dpp_row_max(m);
    double ex[KPL], z = 0.0;
#pragma unroll
    for (int q = 0; q < KPL; ++q) {
      ex[q] = exp(lv[q] - m);
      z += ex[q];
    }
    z = dpp_row_sum(z);
    if (valid)
#pragma unroll
      for (int q = 0; q < KPL; ++q) a.probs[t * E + e0 + q] = (float)(ex[q] / z);
  }
  // group limit: keep the topk_groups groups with the best sums of two keys
  if (a.n_groups > 1) {
    const int gsize = E / a.n_groups;
    const int lpg = gsize / KPL;
    const int levels = lpg >= 16 ? 4 : lpg >= 8 ? 3 : lpg >= 4 ? 2 : lpg >= 2 ? 1 : 0;
    double m1 = -INFINITY, m2 = -INFINITY;
#pragma unroll
    for (int q = 0; q < KPL; ++q) {
      if (key[q] > m1) {
        m2 = m1;
        m1 = key[q];
      } else if (key[q] > m2) {
        m2 = key[q];
      }
    }
    if (levels > 0) dpp_top2_step<DPP_QXOR1>(m1, m2);
    if (levels > 1) dpp_top2_step<DPP_QXOR2>(m1, m2);
    if (levels > 2) dpp_top2_step<DPP_HMIRROR>(m1, m2);
    if (levels > 3) dpp_top2_step<DPP_MIRROR>(m1, m2);
    const int g = e0 / gsize;
    double gscore = gsize >= 2 ? m1 + m2 : m1;
    if (isnan(gscore)) gscore = -INFINITY;
    bool kept = false;
    for (int r = 0; r < a.topk_groups; ++r) {
      double ck = kept ? -INFINITY : gscore;
      int ci = kept ? 0x7fffffff : g;
      dpp_best(ck, ci, 4);
      if (ci == g) kept = true;
    }
    if (!kept) avail = 0;
  }
  // top-k: k rounds of a row argmax; lane s keeps the expert of slot s
  int my_idx = -1;
  for (int s = 0; s < k; ++s) {
    double ck = -INFINITY;
    int ci = 0x7fffffff;  // any available expert beats the empty slot (lower index)
#pragma unroll
    for (int q = 0; q < KPL; ++q)
      if (((avail >> q) & 1u) && better(key[q], e0 + q, ck, ci)) {
        ck = key[q];
        ci = e0 + q;
      }
    dpp_best(ck, ci, 4);
    if (ci >= e0 && ci < e0 + KPL) avail &= ~(1u << (ci - e0));
    if (sub == s) my_idx = ci;
  }
  // weights over the k selected (lanes 0..k-1 of the row hold one slot each)
  const bool holds = sub < k;
  double sc = 0.0;
  if (holds && valid && my_idx >= 0 && my_idx < E) {
    double l = lg[(int64_t)tl * ld + my_idx];
    if (logit_bias) l += (double)a.bias[my_idx];
    sc = sigm ? 1.0 / (1.0 + exp(-l)) : l;
  }
  double w;
  if (sigm) {
    const double z = dpp_row_sum(holds ? sc : 0.0);
    w = (double)a.route_scale * sc / z;
  } else {
    const double m = dpp_row_max(holds ? sc : -INFINITY);
    const double p = holds ? exp(sc - m) : 0.0;
    const double z = dpp_row_sum(p);
    w = (double)a.route_scale * p / z;
  }
  if (holds && valid) {
    a.topk_idx[t * k + sub] = my_idx;
    a.topk_w[t * k + sub] = (float)w;
    if (sigm && a.s_sel) a.s_sel[t * k + sub] = (float)sc;
    atomicAdd(&hist[my_idx], 1);
    if (sel) sel[tl * 16 + sub] = my_idx;
  }
}

// Selection over the float64 logits in the workspace, 16 tokens per
// workgroup: KPL > 0, one DPP row per token (KPL = E / 16 experts per lane);
// KPL = 0, one wavefront per token.
//
// With a.hist set, the selection also builds the permutation's maps inputs
// (section 3.2's token scatter needs, per expert, the rows before each block
// and the expert offsets): every block adds its counts into the count of its
// PERM_TB-token block (cleared by the preceding W_r split launch), and the
// last block to finish (arrival counter, device-scope fences on both sides)
// turns the block counts into bases inside each expert and writes
// expert_offsets.  Nothing waits: the last arrival does the work.
template <int KPL>
__global__ __launch_bounds__(256) void route_select_kernel(RouteArgs a) {
  constexpr int TPB = 16;
  static_assert(PERM_TB % TPB == 0, "selection blocks tile the permutation's blocks");
  __shared__ int hist[256];
  __shared__ int sel[TPB * 16];
  __shared__ int last;
  for (int e = threadIdx.x; e < 256; e += 256) hist[e] = 0;
  for (int i = threadIdx.x; i < TPB * 16; i += 256) sel[i] = -1;
  __syncthreads();
  const int64_t t0 = (int64_t)blockIdx.x * TPB;
  const int ntok = (int)min((int64_t)TPB, a.T - t0);
  int* sl = a.hist ? sel : nullptr;
  if constexpr (KPL > 0)
    select_tokens16<KPL>(a, a.lg + t0 * a.E, a.E, t0, ntok, hist, sl);
  else
    select_tokens(a, a.lg + t0 * a.E, a.E, t0, ntok, hist, sl);
  __syncthreads();
  const int E = a.E;
  if (a.counts) {
    for (int e = threadIdx.x; e < E; e += 256)
      if (hist[e]) atomicAdd(&a.counts[e], hist[e]);
  }
  if (!a.hist) return;
  // this block's counts, and each slot's rank among the block's earlier
  // tokens of its expert (a token never repeats an expert)
  for (int e = threadIdx.x; e < E; e += 256) a.cnt16[(int64_t)blockIdx.x * E + e] = hist[e];
  {
    const int tl = threadIdx.x >> 4, s = threadIdx.x & 15;
    if (tl < ntok && s < a.k) {
      const int e = sel[tl * 16 + s];
      int r = -1;
      if (e >= 0) {
        r = 0;
        for (int u = 0; u < tl; ++u)
#pragma unroll
          for (int v = 0; v < 16; ++v) r += sel[u * 16 + v] == e;
      }
      a.row_of[(t0 + tl) * a.k + s] = r;
    }
  }
  // the block counts and the arrival counter are device-scope atomics, all
  // performed where every XCD sees them; a block counts its arrival only once
  // its count additions have returned, and the last block reads the counts
  // with device-scope atomic loads
  int32_t* bh = a.hist + (t0 / PERM_TB) * E;
  for (int e = threadIdx.x; e < E; e += 256)
    if (hist[e]) (void)__hip_atomic_fetch_add(&bh[e], hist[e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  wait_vmcnt<0>();
  __syncthreads();
  if (threadIdx.x == 0)
    last = __hip_atomic_fetch_add(a.sync, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (int)gridDim.x - 1;
  __syncthreads();
  if (!last) return;
  // the last block: bases inside each expert, then the expert offsets
  const int64_t nblk = perm_blocks(a.T);
  int tot = 0;
  if ((int)threadIdx.x < E) {
    const int e = threadIdx.x;
    for (int64_t b0 = 0; b0 < nblk; b0 += 16) {
      int v[16];
#pragma unroll
      for (int q = 0; q < 16; ++q)
        v[q] = b0 + q < nblk ? __hip_atomic_load(&a.hist[(b0 + q) * E + e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                             : 0;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        if (b0 + q < nblk) a.hist[(b0 + q) * E + e] = tot;
        tot += v[q];
      }
    }
  }
  __shared__ int sbuf[256];
  __shared__ int total;
  const int ex = block_scan_256(tot, sbuf, &total);
  if ((int)threadIdx.x < E) a.offsets[threadIdx.x] = ex;
  if (threadIdx.x == 0) a.offsets[E] = total;
}

int launch_route_gemm(const RouteArgs& a, hipStream_t s) {
  {
    dim3 grid((a.E + 31) / 32, (a.d + 31) / 32);
    bf16_t* wsp = reinterpret_cast<bf16_t*>(a.wsplit);
    const int64_t nh = a.hist ? perm_blocks(a.T) * a.E : 0;
    const int st = launch(K_WR_SPLIT, s, "wr_split", [&] {
      wr_split_kernel<<<grid, 256, 0, s>>>(a.w_r, wsp, a.d, a.E, a.counts, a.counts ? a.E : 0, a.hist, nh, a.sync,
                                           a.hist ? 1 : 0);
    });
    if (st) return st;
  }
  // a router weight that fits in L2 is re-read per 64-token tile; a larger
  // one (DeepSeek-like d x 256) per 128 tokens
  const bool big_w = (int64_t)3 * a.E * a.d * 2 > ((int64_t)2 << 20);
  int st;
#define MOE_RL(TT_, TE_)                                                                               \
  st = launch(K_ROUTE, s, "route", [&] {                                                               \
    route_logits_kernel<TT_, TE_><<<(int)(((a.T + TT_ - 1) / TT_) * (a.E / TE_)), TT_ * 4, 0, s>>>(a); \
  });
  if (a.E % 64 == 0) {
    if (big_w) { MOE_RL(128, 64) } else { MOE_RL(64, 64) }
  } else {
    MOE_RL(64, 32)
  }
#undef MOE_RL
  if (st) return st;
  // one DPP row per token when E / 16 experts per lane tile the groups into
  // whole power-of-two lane sets (always without a group limit)
  const int kpl = a.E / 16;
  bool rows16 = a.E % 16 == 0 && a.E <= 256 && a.router != MOE_ROUTER_SIGMOID_THRESHOLD;
  if (rows16 && a.n_groups > 1) {
    const int gsize = a.E / a.n_groups, lpg = gsize / kpl;
    rows16 = gsize % kpl == 0 && lpg >= 1 && lpg <= 16 && (lpg & (lpg - 1)) == 0;
  }
  const int nb = (int)((a.T + 15) / 16);
#define MOE_SEL(KPL_) \
  return launch(K_ROUTE_SELECT, s, "route_select", [&] { route_select_kernel<KPL_><<<nb, 256, 0, s>>>(a); });
  if (rows16) switch (kpl) {
      case 2: MOE_SEL(2)
      case 4: MOE_SEL(4)
      case 6: MOE_SEL(6)
      case 8: MOE_SEL(8)
      case 10: MOE_SEL(10)
      case 12: MOE_SEL(12)
      case 14: MOE_SEL(14)
      case 16: MOE_SEL(16)
      default: break;
    }
  MOE_SEL(0)
#undef MOE_SEL
}

// NTW: 16-expert MFMA tiles per wavefront.  Without SPLIT a block is 64 tokens
// x 16*NTW experts (4 wavefronts stacked over tokens); with SPLIT it is 32
// tokens x 32*NTW experts (2 x 2 wavefronts).
template <int NTW, bool SPLIT>
__global__ __launch_bounds__(256) void route_mfma_kernel(RouteArgs a) {
  constexpr int TBM = SPLIT ? 32 : 64;
  constexpr int EW = 16 * NTW;
  constexpr int EB = SPLIT ? 2 * EW : EW;
  constexpr int KC = 32;
  constexpr int STAGE = 3 * EB * KC;  // bf16 elements
  constexpr int NCH = STAGE / 8;               // 16-byte chunks per stage
  constexpr int NB = (NCH + 255) / 256;       // per thread
  constexpr int BYTES_STAGES = 2 * STAGE * 2;
  constexpr int BYTES_TABLE = TBM * EB * 8;
  constexpr int LDS = BYTES_STAGES > BYTES_TABLE ? BYTES_STAGES : BYTES_TABLE;
  __shared__ __align__(16) unsigned char smem[LDS];
  __shared__ int hist[256];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wt = SPLIT ? (wave >> 1) : wave;
  const int we = SPLIT ? (wave & 1) : 0;
  const int E = a.E, d = a.d;
  const int64_t t0 = (int64_t)blockIdx.x * TBM;
  const bf16_t* x = reinterpret_cast<const bf16_t*>(a.x);
  const bf16_t* wsp = reinterpret_cast<const bf16_t*>(a.wsplit);
  bf16_t* stage = reinterpret_cast<bf16_t*>(smem);

  for (int e = tid; e < 256; e += 256) hist[e] = 0;

  // A fragment source: token row (lane % 16) of this wavefront, 8 k at 8*(lane/16)
  const int64_t trow = t0 + wt * 16 + (lane & 15);
  const bool tok_ok = trow < a.T;
  const bf16_t* xrow = x + (tok_ok ? trow : 0) * d + 8 * (lane >> 4);

  // B staging: chunk q = tid + 256*i -> row (q / 4) of [3][EB], 16-byte chunk q % 4
  const bf16_t* bsrc[NB];
  int boff[NB];
  bool bok[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int q0 = tid + 256 * i;
    const bool inr = q0 < NCH;
    const int q = inr ? q0 : 0;
    const int row = q >> 2, c = q & 3;
    const int p = row / EB, e = row - p * EB;
    bok[i] = inr && e < E;
    bsrc[i] = wsp + ((int64_t)p * E + (e < E ? e : 0)) * d + 8 * c;
    boff[i] = inr ? row * KC + ((c ^ ((row >> 2) & 3)) << 3) : -1;
  }
  uint4 breg[NB];
  uint4 areg;
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < NB; ++i)
      breg[i] = bok[i] ? *reinterpret_cast<const uint4*>(bsrc[i] + k0) : make_uint4(0, 0, 0, 0);
    areg = tok_ok ? *reinterpret_cast<const uint4*>(xrow + k0) : make_uint4(0, 0, 0, 0);
  };
  auto store = [&](int buf) {
    bf16_t* st = stage + buf * STAGE;
#pragma unroll
    for (int i = 0; i < NB; ++i)
      if (boff[i] >= 0) *reinterpret_cast<uint4*>(st + boff[i]) = breg[i];
  };

  floatx4 acc[NTW];
  double acc64[NTW][4];
#pragma unroll
  for (int j = 0; j < NTW; ++j) {
    acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int v = 0; v < 4; ++v) acc64[j][v] = 0.0;
  }
  const int nk = d / KC;
  load(0);
  store(0);
  uint4 acur = areg;
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load((kt + 1) * KC);
    const bf16_t* st = stage + cur * STAGE;
    const bf16x8 af = __builtin_bit_cast(bf16x8, acur);
#pragma unroll
    for (int p = 0; p < 3; ++p) {
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        const int row = p * EB + we * EW + 16 * j + (lane & 15);
        const int c = lane >> 4;
        const bf16x8 bfr = *reinterpret_cast<const bf16x8*>(st + row * KC + ((c ^ ((row >> 2) & 3)) << 3));
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bfr, acc[j], 0, 0, 0);
      }
    }
    if ((kt & 1) || kt + 1 == nk) {
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
#pragma unroll
        for (int v = 0; v < 4; ++v) acc64[j][v] += (double)acc[j][v];
        acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
    }
    if (kt + 1 < nk) {
      store(cur ^ 1);
      acur = areg;
    }
    __syncthreads();
  }

  // logits -> LDS table [TBM][EB]
  double* lg = reinterpret_cast<double*>(smem);
#pragma unroll
  for (int j = 0; j < NTW; ++j)
#pragma unroll
    for (int v = 0; v < 4; ++v)
      lg[(wt * 16 + 4 * (lane >> 4) + v) * EB + we * EW + 16 * j + (lane & 15)] = acc64[j][v];
  __syncthreads();

  select_tokens(a, lg, EB, t0, TBM, hist);
  __syncthreads();
  if (a.counts) {
    for (int e = tid; e < E; e += 256)
      if (hist[e]) atomicAdd(&a.counts[e], hist[e]);
  }
}

int launch_route_mfma(const RouteArgs& a, hipStream_t s) {
  {
    dim3 grid((a.E + 31) / 32, (a.d + 31) / 32);
    bf16_t* wsp = reinterpret_cast<bf16_t*>(a.wsplit);
    const int st = launch(K_WR_SPLIT, s, "wr_split", [&] {
      wr_split_kernel<<<grid, 256, 0, s>>>(a.w_r, wsp, a.d, a.E, a.counts, a.counts ? a.E : 0, nullptr, 0, nullptr, 0);
    });
    if (st) return st;
  }
#define MOE_RM(NTW_, SPLIT_, TBM_)                                                                           \
  return launch(K_ROUTE, s, "route", [&] {                                                                   \
    route_mfma_kernel<NTW_, SPLIT_><<<(int)((a.T + TBM_ - 1) / TBM_), 256, 0, s>>>(a);                       \
  });
  if (a.E <= 32) { MOE_RM(2, false, 64) }
  if (a.E <= 64) { MOE_RM(4, false, 64) }
  if (a.E <= 128) { MOE_RM(8, false, 64) }
  MOE_RM(8, true, 32)
#undef MOE_RM
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

int launch_route(const RouteArgs& a, hipStream_t s, bool* maps_built) {
  if (maps_built) *maps_built = false;
  const bool gemm_path = a.T > 0 && a.bf16 && a.wsplit && a.lg && a.E % 32 == 0;
  const bool mfma_path = a.T > 0 && a.bf16 && a.wsplit && a.E % 16 == 0;
  // (the W_r split launch of the MFMA paths clears the counts itself)
  if (a.counts && !gemm_path && !mfma_path) {
    int st = zero_i32(a.counts, a.E, s);
    if (st) return st;
  }
  if (a.T == 0) return MOE_OK;
  if (gemm_path) {
    // the selection builds the permutation's block bases and offsets when
    // the last block's serial pass over the blocks stays short
    RouteArgs b = a;
    const bool maps = a.hist && a.offsets && a.sync && a.cnt16 && a.row_of && a.E <= 256 && a.k <= 16 &&
                      perm_blocks(a.T) <= 512;
    if (!maps) b.hist = nullptr;
    const int st = launch_route_gemm(b, s);
    if (st == MOE_OK && maps_built) *maps_built = maps;
    return st;
  }
  RouteArgs b = a;
  b.hist = nullptr;
  if (mfma_path) return launch_route_mfma(b, s);
  return a.bf16 ? launch_route_t<bf16_t>(b, s) : launch_route_t<float>(b, s);
}

}  // namespace moe
