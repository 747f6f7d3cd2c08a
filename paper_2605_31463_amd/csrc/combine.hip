// Gather-side kernels of the layer: weighted combine, its backward (with the
// first step of the router backward fused in), and the unpermute-reduce of
// the data gradient (with the router's dx fused in); each also in a variant
// for pools with zero-computation experts (MoE++, appendix B.3).
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

// 16 bytes of an expert row that the layer reads exactly once (o rows in the
// combine, dx_perm rows in the unpermute), as a nontemporal load: measured
// in the whole layer, DeepSeek-V3 shape combine forward 253 -> 211 us,
// unpermute 259 -> 246; Qwen3 shape combine forward 61 -> 55, combine backward
// 107 -> 98, unpermute 64 -> 62 (nontemporal stores of d_o and x_perm were
// slower: 107 -> 127 and 48 -> 60 us at the Qwen3 shape)
template <class XT>
__device__ __forceinline__ uint4 load_once(const XT* p) {
  return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const int32x4_t*>(p)));
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
  bool ok[KM];
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    rows[s] = s < k ? a.row_of[t * a.k + s] : 0;
    w[s] = s < k ? a.topk_w[t * a.k + s] : 0.f;
    ok[s] = s < k && (uint64_t)rows[s] < (uint64_t)R;
    if (!ok[s]) {  // an empty or dropped slot contributes nothing (and loads nothing)
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
        raw[s] = ok[s] ? load_once(o + rows[s] * a.d + (int64_t)c * V) : make_uint4(0, 0, 0, 0);
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

// Q8: also the E4M3 rows of d_o (a kernel of its own, so that the bf16 path
// keeps its register count and occupancy)
template <class XT, int KT, bool Q8 = false>
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
  float w[KM], om[KM], qi[KM];
  bool ok[KM];
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    rows[s] = s < k ? a.row_of[t * a.k + s] : 0;
    w[s] = s < k ? a.topk_w[t * a.k + s] : 0.f;
    om[s] = 0.f;
    ok[s] = s < k && (uint64_t)rows[s] < (uint64_t)R;
    if (!ok[s]) rows[s] = 0;
  }
  // FP8 data gradients: E4M3 rows of the stored d_o as well.  Row s is
  // bf16(w_s dy_t); rounding is monotone and sign-symmetric, so its largest
  // magnitude is bf16(|w_s| max|dy_t|), known before any value is written.
  static_assert(!Q8 || sizeof(XT) == 2, "E4M3 rows of bf16 layers only");
  if constexpr (Q8) {
    float m = 0.f;
    for (int c = lane; c < nch; c += 64) {
      float g[V];
      Vec16<XT>::load(dy + t * a.d + (int64_t)c * V, g);
#pragma unroll
      for (int v = 0; v < V; ++v) m = fmaxf(m, fabsf(g[v]));
    }
    m = wave_max(m);
#pragma unroll
    for (int s = 0; s < KM; ++s) {
      const float am = bf2f(f2bf(fabsf(w[s]) * m));
      qi[s] = e4m3_inv(am);
      if (lane == 0 && ok[s]) a.sdo[rows[s]] = e4m3_scale(am);
    }
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
        raw[s] = ok[s] ? load_once(o + rows[s] * a.d + (int64_t)c * V) : make_uint4(0, 0, 0, 0);
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
        if constexpr (Q8) {  // the codes of the stored (bf16) values
          float b[8];
#pragma unroll
          for (int v = 0; v < 8; ++v) b[v] = bf2f(f2bf(out[v])) * qi[s];
          *reinterpret_cast<uint2*>(a.doq + rows[s] * a.d + (int64_t)c * 8) =
              make_uint2(e4m3x4(b[0], b[1], b[2], b[3]), e4m3x4(b[4], b[5], b[6], b[7]));
        }
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
    if (a.router == MOE_ROUTER_SIGMOID_GROUPED || a.router == MOE_ROUTER_SIGMOID_THRESHOLD) {
      // (an empty slot of the threshold router has s = 0 and gets 0)
#pragma unroll
      for (int s = 0; s < KM; ++s)
        if (s < k) z += a.s_sel[t * a.k + s];
#pragma unroll
      for (int s = 0; s < KM; ++s)
        if (s < k) {
          const float sv = a.s_sel[t * a.k + s];
          const float gs = (c * om[s] - wo) / z * sv;
          a.dl[t * a.k + s] = gs * (1.f - sv);
          if (a.dth) a.dth[t * a.k + s] = -gs;  // straight-through threshold gradient
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
  // workgroup b takes column slice b % ns of its four tokens' rows: with 8
  // slices every XCD gathers its own eighth of the W_r^T rows, which then
  // stays in its L2
  const int ns = a.ns, sl = (int)(blockIdx.x % ns);
  const int64_t t = uniform_token((int64_t)(blockIdx.x / ns) * 4 + (threadIdx.x >> 6));
  if (t >= a.T) return;
  const int k = KT > 0 ? KT : a.k;
  const int cs = a.d / V / ns;  // 16-byte chunks per slice
  const int c_lo = sl * cs, c_hi = c_lo + cs;
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
  for (int c0 = c_lo; c0 < c_hi; c0 += 64 * CPL) {
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c = c0 + j * 64 + lane;
      if (c >= c_hi) break;
      // every load of this chunk first, then the sums in slot order
      uint4 raw[KM], rw[KM];
#pragma unroll
      for (int s = 0; s < KM; ++s) {
        raw[s] = make_uint4(0, 0, 0, 0);
        rw[s] = make_uint4(0, 0, 0, 0);
        if (s < k && ok[s]) raw[s] = load_once(dxp + rows[s] * a.d + (int64_t)c * V);
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

// ---------------------------------------------------------------------------
// Zero-computation experts (MoE++).  A slot whose pool id is E_ffn or above
// has no expert row: a zero expert adds nothing, a copy expert w x_t, a
// constant expert w (a0 x_t + a1 v_c) with (a0, a1) = softmax(W_c x_t).  Per
// token the wave first takes the dot products W_c x_t of its constant slots
// (one pass over x_t), then runs the combine with them.
// ---------------------------------------------------------------------------
enum { ZK_FFN = 0, ZK_ZERO = 1, ZK_COPY = 2, ZK_CONST = 3 };

// Kind of pool id e (c: index among the constant experts).  An id outside
// the pool (not produced by the router) is taken as a zero expert, so that
// no load leaves the parameter arrays.
__device__ __forceinline__ int zc_kind(const ZcArgs& z, int e, int& c) {
  c = 0;
  if (e < 0) return ZK_ZERO;
  const int j = e - z.E_ffn;
  if (j < 0) return ZK_FFN;
  if (j < z.n_zero) return ZK_ZERO;
  if (j < z.n_zero + z.n_copy) return ZK_COPY;
  c = j - z.n_zero - z.n_copy;
  return c < z.n_const ? ZK_CONST : ZK_ZERO;
}

__device__ __forceinline__ bool zc_in_pool(const ZcArgs& z, int64_t e) {
  return (uint64_t)e < (uint64_t)(z.E_ffn + z.n_zero + z.n_copy + z.n_const);
}

// (a0, a1) = softmax(z0, z1)
__device__ __forceinline__ void softmax2(float z0, float z1, float& a0, float& a1) {
  const float m = fmaxf(z0, z1);
  const float e0 = __expf(z0 - m), e1 = __expf(z1 - m);
  const float r = 1.0f / (e0 + e1);
  a0 = e0 * r;
  a1 = e1 * r;
}

// Slot kinds of token t, and z = W_c x_t for its constant slots (every lane
// ends with the sums).  Returns whether the token has a constant slot.
template <class XT, int KM>
__device__ __forceinline__ bool zc_slots(const ZcArgs& z, const int32_t* topk_idx, int64_t t, int k, int d,
                                         int lane, int* kind, int* cid, float* z0, float* z1) {
  constexpr int V = Vec16<XT>::N;
  bool any_const = false;
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    kind[s] = ZK_ZERO;
    cid[s] = 0;
    z0[s] = z1[s] = 0.f;
    if (s < k) {
      const int e = __builtin_amdgcn_readfirstlane(topk_idx[t * k + s]);
      kind[s] = zc_kind(z, e, cid[s]);
      any_const |= kind[s] == ZK_CONST;
    }
  }
  if (!any_const) return false;
  const XT* x = reinterpret_cast<const XT*>(z.x) + t * d;
  const int nch = d / V;
  for (int c = lane; c < nch; c += 64) {
    float xv[V];
    Vec16<XT>::load(x + (int64_t)c * V, xv);
#pragma unroll
    for (int s = 0; s < KM; ++s) {
      if (s >= k || kind[s] != ZK_CONST) continue;
      const float* w0 = z.wc + (int64_t)cid[s] * 2 * d + (int64_t)c * V;
      const float* w1 = w0 + d;
#pragma unroll
      for (int v = 0; v < V; ++v) {
        z0[s] = __builtin_fmaf(w0[v], xv[v], z0[s]);
        z1[s] = __builtin_fmaf(w1[v], xv[v], z1[s]);
      }
    }
  }
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    if (s >= k || kind[s] != ZK_CONST) continue;
    z0[s] = wave_sum(z0[s]);
    z1[s] = wave_sum(z1[s]);
  }
  return true;
}

template <class XT, int KT>
__global__ __launch_bounds__(256) void combine_fwd_zc_kernel(CombineFwdArgs a) {
  constexpr int V = Vec16<XT>::N;
  constexpr int KM = KT > 0 ? KT : KMAX;
  const int lane = threadIdx.x & 63;
  const int64_t t = uniform_token((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
  if (t >= a.T) return;
  const int k = KT > 0 ? KT : a.k;
  const int nch = a.d / V;
  const ZcArgs& z = a.zc;
  const XT* o = reinterpret_cast<const XT*>(a.o);
  const XT* sh = reinterpret_cast<const XT*>(a.shared_o);
  const XT* x = reinterpret_cast<const XT*>(z.x) + t * a.d;
  XT* y = reinterpret_cast<XT*>(a.y);
  int kind[KM], cid[KM];
  float z0[KM], z1[KM];
  zc_slots<XT, KM>(z, a.topk_idx, t, a.k, a.d, lane, kind, cid, z0, z1);
  int64_t rows[KM];
  float w[KM], bv[KM];
  float ax = 0.f;  // factor of x_t: copy slots w, constant slots w a0
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    rows[s] = 0;
    w[s] = bv[s] = 0.f;
    if (s >= k) continue;
    const float ws = a.topk_w[t * a.k + s];
    if (kind[s] == ZK_FFN) {
      rows[s] = a.row_of[t * a.k + s];
      w[s] = ws;
      if ((uint64_t)rows[s] >= (uint64_t)(a.T * a.k)) {  // no row: contributes nothing
        kind[s] = ZK_ZERO;
        rows[s] = 0;
      }
    } else if (kind[s] == ZK_COPY) {
      ax += ws;
    } else if (kind[s] == ZK_CONST) {
      float a0, a1;
      softmax2(z0[s], z1[s], a0, a1);
      ax += ws * a0;
      bv[s] = ws * a1;
    }
  }
  const bool use_x = ax != 0.f;
  for (int c0 = 0; c0 < nch; c0 += 64 * CPL) {
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c = c0 + j * 64 + lane;
      if (c >= nch) break;
      uint4 raw[KM];
#pragma unroll
      for (int s = 0; s < KM; ++s)
        raw[s] = (s < k && kind[s] == ZK_FFN) ? load_once(o + rows[s] * a.d + (int64_t)c * V)
                                              : make_uint4(0, 0, 0, 0);
      float acc[V];
#pragma unroll
      for (int v = 0; v < V; ++v) acc[v] = 0.f;
#pragma unroll
      for (int s = 0; s < KM; ++s) {
        if (s >= k) break;
        if (kind[s] == ZK_FFN) {
          float vv[V];
          Vec16<XT>::load(reinterpret_cast<const XT*>(&raw[s]), vv);
#pragma unroll
          for (int v = 0; v < V; ++v) acc[v] = __builtin_fmaf(w[s], vv[v], acc[v]);
        } else if (kind[s] == ZK_CONST) {
          const float* vc = z.v + (int64_t)cid[s] * a.d + (int64_t)c * V;
#pragma unroll
          for (int v = 0; v < V; ++v) acc[v] = __builtin_fmaf(bv[s], vc[v], acc[v]);
        }
      }
      if (use_x) {
        float xv[V];
        Vec16<XT>::load(x + (int64_t)c * V, xv);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[v] = __builtin_fmaf(ax, xv[v], acc[v]);
      }
      if (sh) {
        float vv[V];
        Vec16<XT>::load(sh + t * a.d + (int64_t)c * V, vv);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[v] += vv[v];
      }
      Vec16<XT>::store(y + t * a.d + (int64_t)c * V, acc);
    }
  }
}

// Combine backward with zero-computation slots.  One pass over d takes, per
// slot, omega = <dy, out>: FFN slots from their row (and d_o = w dy), copy
// slots <dy, x>, constant slots a0 <dy, x> + a1 <dy, v_c> (with z = W_c x
// taken in the same pass); then dl as for the FFN-only combine, and per slot
// the coefficients of the zero-computation gradients:
//   constant: da = w (<dy, x>, <dy, v_c>), dz = a * (da - <a, da>),
//             coef = (dz0, dz1, w a1, w a0)
//   copy:     coef = (0, 0, 0, w);  zero and FFN slots: 0.
template <class XT, int KT>
__global__ __launch_bounds__(256) void combine_bwd_zc_kernel(CombineBwdArgs a) {
  constexpr int V = Vec16<XT>::N;
  constexpr int KM = KT > 0 ? KT : KMAX;
  const int lane = threadIdx.x & 63;
  const int64_t t = uniform_token((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
  if (t >= a.T) return;
  const int k = KT > 0 ? KT : a.k;
  const int nch = a.d / V;
  const ZcArgs& z = a.zc;
  const XT* dy = reinterpret_cast<const XT*>(a.dy);
  const XT* o = reinterpret_cast<const XT*>(a.o);
  const XT* x = reinterpret_cast<const XT*>(z.x) + t * a.d;
  XT* d_o = reinterpret_cast<XT*>(a.d_o);
  int kind[KM], cid[KM];
  int64_t rows[KM];
  float w[KM], om[KM], dyv[KM], z0[KM], z1[KM];
  bool need_x = false;
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    kind[s] = ZK_ZERO;
    cid[s] = 0;
    rows[s] = 0;
    w[s] = om[s] = dyv[s] = z0[s] = z1[s] = 0.f;
    if (s < k) {
      const int e = __builtin_amdgcn_readfirstlane(a.topk_idx[t * a.k + s]);
      kind[s] = zc_kind(z, e, cid[s]);
      w[s] = a.topk_w[t * a.k + s];
      if (kind[s] == ZK_FFN) {
        rows[s] = a.row_of[t * a.k + s];
        if ((uint64_t)rows[s] >= (uint64_t)(a.T * a.k)) {
          kind[s] = ZK_ZERO;
          rows[s] = 0;
        }
      }
      need_x |= kind[s] == ZK_COPY || kind[s] == ZK_CONST;
    }
  }
  float dyx = 0.f;
  for (int c0 = 0; c0 < nch; c0 += 64 * CPL) {
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c = c0 + j * 64 + lane;
      if (c >= nch) break;
      const uint4 graw = *reinterpret_cast<const uint4*>(dy + t * a.d + (int64_t)c * V);
      uint4 raw[KM];
#pragma unroll
      for (int s = 0; s < KM; ++s)
        raw[s] = (s < k && kind[s] == ZK_FFN) ? load_once(o + rows[s] * a.d + (int64_t)c * V)
                                              : make_uint4(0, 0, 0, 0);
      float g[V], xv[V];
      Vec16<XT>::load(reinterpret_cast<const XT*>(&graw), g);
#pragma unroll
      for (int v = 0; v < V; ++v) xv[v] = 0.f;
      if (need_x) {
        Vec16<XT>::load(x + (int64_t)c * V, xv);
#pragma unroll
        for (int v = 0; v < V; ++v) dyx = __builtin_fmaf(g[v], xv[v], dyx);
      }
#pragma unroll
      for (int s = 0; s < KM; ++s) {
        if (s >= k) break;
        if (kind[s] == ZK_FFN) {
          float vv[V], out[V];
          Vec16<XT>::load(reinterpret_cast<const XT*>(&raw[s]), vv);
#pragma unroll
          for (int v = 0; v < V; ++v) {
            om[s] = __builtin_fmaf(g[v], vv[v], om[s]);
            out[v] = w[s] * g[v];
          }
          Vec16<XT>::store(d_o + rows[s] * a.d + (int64_t)c * V, out);
        } else if (kind[s] == ZK_CONST) {
          const float* vc = z.v + (int64_t)cid[s] * a.d + (int64_t)c * V;
          const float* w0 = z.wc + (int64_t)cid[s] * 2 * a.d + (int64_t)c * V;
          const float* w1 = w0 + a.d;
#pragma unroll
          for (int v = 0; v < V; ++v) {
            dyv[s] = __builtin_fmaf(g[v], vc[v], dyv[s]);
            z0[s] = __builtin_fmaf(w0[v], xv[v], z0[s]);
            z1[s] = __builtin_fmaf(w1[v], xv[v], z1[s]);
          }
        }
      }
    }
  }
  if (need_x) dyx = wave_sum(dyx);
  float4 cf[KM];
  float wo = 0.f;
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    if (s >= k) break;
    cf[s] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (kind[s] == ZK_FFN) {
      om[s] = wave_sum(om[s]);
    } else if (kind[s] == ZK_COPY) {
      om[s] = dyx;
      cf[s].w = w[s];
    } else if (kind[s] == ZK_CONST) {
      dyv[s] = wave_sum(dyv[s]);
      float a0, a1;
      softmax2(wave_sum(z0[s]), wave_sum(z1[s]), a0, a1);
      om[s] = a0 * dyx + a1 * dyv[s];
      const float da0 = w[s] * dyx, da1 = w[s] * dyv[s];
      const float ad = a0 * da0 + a1 * da1;
      cf[s] = make_float4(a0 * (da0 - ad), a1 * (da1 - ad), w[s] * a1, w[s] * a0);
    }
    wo += w[s] * om[s];
  }
  if (lane == 0) {
#pragma unroll
    for (int s = 0; s < KM; ++s) {
      if (s >= k) break;
      z.coef[t * a.k + s] = cf[s];
      if (a.d_topk_w) a.d_topk_w[t * a.k + s] = om[s];
      // softmax families only (zero-computation experts need a softmax router)
      if (a.dl) a.dl[t * a.k + s] = w[s] * (om[s] - wo / a.route_scale);
    }
  }
}

// Unpermute with zero-computation slots: dx_t = sum over FFN slots of their
// dx_perm rows + sum over all slots of dl W_r[:, e] + (sum of the slots' dy
// factors) dy_t + sum over constant slots of W_c^T dz (+ shared, auxiliary).
template <class XT, int KT>
__global__ __launch_bounds__(256) void unpermute_zc_kernel(UnpermuteArgs a) {
  constexpr int V = Vec16<XT>::N;
  constexpr int KM = KT > 0 ? KT : KMAX;
  const int lane = threadIdx.x & 63;
  const int64_t t = uniform_token((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
  if (t >= a.T) return;
  const int k = KT > 0 ? KT : a.k;
  const int nch = a.d / V;
  const ZcArgs& z = a.zc;
  const XT* dxp = reinterpret_cast<const XT*>(a.dx_perm);
  const XT* dxs = reinterpret_cast<const XT*>(a.dx_shared);
  const XT* dxa = reinterpret_cast<const XT*>(a.dx_aux);
  const XT* wrt = reinterpret_cast<const XT*>(a.w_rt);
  const XT* dyt = reinterpret_cast<const XT*>(z.dy) + t * a.d;
  XT* dx = reinterpret_cast<XT*>(a.dx);
  int64_t rows[KM], ex[KM];
  int kind[KM], cid[KM];
  float dl[KM], dz0[KM], dz1[KM];
  float gdy = 0.f;  // factor of dy_t
#pragma unroll
  for (int s = 0; s < KM; ++s) {
    rows[s] = ex[s] = 0;
    kind[s] = ZK_ZERO;
    cid[s] = 0;
    dl[s] = dz0[s] = dz1[s] = 0.f;
    if (s >= k) continue;
    const int e = __builtin_amdgcn_readfirstlane(a.topk_idx[t * a.k + s]);
    ex[s] = e;
    kind[s] = zc_kind(z, e, cid[s]);
    dl[s] = a.dl ? a.dl[t * a.k + s] : 0.f;
    if (kind[s] == ZK_FFN) {
      rows[s] = a.row_of[t * a.k + s];
      if ((uint64_t)rows[s] >= (uint64_t)(a.T * a.k)) {
        kind[s] = ZK_ZERO;
        rows[s] = 0;
      }
    } else {
      const float4 cf = z.coef[t * a.k + s];
      dz0[s] = cf.x;
      dz1[s] = cf.y;
      gdy += cf.w;
    }
  }
  const bool use_dy = gdy != 0.f;
  for (int c0 = 0; c0 < nch; c0 += 64 * CPL) {
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c = c0 + j * 64 + lane;
      if (c >= nch) break;
      uint4 raw[KM], rw[KM];
#pragma unroll
      for (int s = 0; s < KM; ++s) {
        raw[s] = make_uint4(0, 0, 0, 0);
        rw[s] = make_uint4(0, 0, 0, 0);
        if (s < k && kind[s] == ZK_FFN) raw[s] = load_once(dxp + rows[s] * a.d + (int64_t)c * V);
        if (s < k && a.dl && zc_in_pool(z, ex[s]))
          rw[s] = *reinterpret_cast<const uint4*>(wrt + ex[s] * a.d + (int64_t)c * V);
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
        if (kind[s] == ZK_CONST) {
          const float* w0 = z.wc + (int64_t)cid[s] * 2 * a.d + (int64_t)c * V;
          const float* w1 = w0 + a.d;
#pragma unroll
          for (int v = 0; v < V; ++v) r[v] = __builtin_fmaf(dz0[s], w0[v], __builtin_fmaf(dz1[s], w1[v], r[v]));
        }
      }
      if (use_dy) {
        float g[V];
        Vec16<XT>::load(dyt + (int64_t)c * V, g);
#pragma unroll
        for (int v = 0; v < V; ++v) r[v] = __builtin_fmaf(gdy, g[v], r[v]);
      }
#pragma unroll
      for (int v = 0; v < V; ++v) acc[v] += r[v];
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
  if (a.zc.on) {
    if (a.bf16) { MOE_BY_K("combine_fwd", K_COMBINE_FWD, combine_fwd_zc_kernel, bf16_t) }
    MOE_BY_K("combine_fwd", K_COMBINE_FWD, combine_fwd_zc_kernel, float)
  }
  if (a.bf16) { MOE_BY_K("combine_fwd", K_COMBINE_FWD, combine_fwd_kernel, bf16_t) }
  MOE_BY_K("combine_fwd", K_COMBINE_FWD, combine_fwd_kernel, float)
}

int launch_combine_bwd(const CombineBwdArgs& a, hipStream_t s) {
  if (a.doq && (a.zc.on || !a.bf16 || !a.sdo))
    return moe_set_error(MOE_ERR_UNSUPPORTED, "combine_bwd: E4M3 d_o rows need bf16 without zero-computation experts");
  if (a.T == 0) return MOE_OK;
  const int nb = (int)((a.T + 3) / 4);
  if (a.zc.on) {
    if (a.bf16) { MOE_BY_K("combine_bwd", K_COMBINE_BWD, combine_bwd_zc_kernel, bf16_t) }
    MOE_BY_K("combine_bwd", K_COMBINE_BWD, combine_bwd_zc_kernel, float)
  }
  if (a.doq) {
    switch (a.k) {
      case 8: return launch(K_COMBINE_BWD, s, "combine_bwd", [&] { combine_bwd_kernel<bf16_t, 8, true><<<nb, 256, 0, s>>>(a); });
      case 4: return launch(K_COMBINE_BWD, s, "combine_bwd", [&] { combine_bwd_kernel<bf16_t, 4, true><<<nb, 256, 0, s>>>(a); });
      default: return launch(K_COMBINE_BWD, s, "combine_bwd", [&] { combine_bwd_kernel<bf16_t, 0, true><<<nb, 256, 0, s>>>(a); });
    }
  }
  if (a.bf16) { MOE_BY_K("combine_bwd", K_COMBINE_BWD, combine_bwd_kernel, bf16_t) }
  MOE_BY_K("combine_bwd", K_COMBINE_BWD, combine_bwd_kernel, float)
}

template <class XT>
int launch_unpermute_t(const UnpermuteArgs& a0, hipStream_t s) {
  UnpermuteArgs a = a0;
  a.ns = 1;
  if (a.zc.on) {
    const int nb = (int)((a.T + 3) / 4);
    MOE_BY_K("unpermute", K_UNPERMUTE, unpermute_zc_kernel, XT)
  }
  // the router dx gathers k rows of W_r^T per token: in 8 column slices of
  // at least 64 chunks each (one per XCD) once W_r^T outgrows an XCD's share
  // of L2 (DeepSeek-V3 shape, 3.7 MB: 245 -> 233 us)
  const int nch = a.d / Vec16<XT>::N;
  if (a.dl && nch % 8 == 0 && nch / 8 >= 64) a.ns = 8;
  const int nb = (int)((a.T + 3) / 4) * a.ns;
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
