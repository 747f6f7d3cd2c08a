// libmoe C ABI: argument checks, workspace planning, the component entry
// points and the fused layer forward / backward.  Everything here runs on the
// host and only enqueues kernels on the caller's stream.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <vector>

#include <cstddef>

#include "common.h"
#include "kernels.h"

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------
static thread_local char g_err[512];

int moe_set_error(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return status;
}

namespace moe {

int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return moe_set_error(MOE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return MOE_OK;
}

// ---------------------------------------------------------------------------
// kernel timing (benchmarks)
// ---------------------------------------------------------------------------
namespace {
struct Timing {
  int sel = -1;
  std::vector<hipEvent_t> ev;  // start, stop pairs
  int used = 0;
  bool open = false;
};
thread_local Timing g_timing;
constexpr int kMaxTimed = 4096;
}  // namespace

void timing_before(int id, hipStream_t s) {
  Timing& t = g_timing;
  t.open = false;
  if (t.sel != id || t.used >= kMaxTimed) return;
  if ((int)t.ev.size() < 2 * (t.used + 1)) {
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess) return;
    if (hipEventCreate(&b) != hipSuccess) {
      (void)hipEventDestroy(a);
      return;
    }
    t.ev.push_back(a);
    t.ev.push_back(b);
  }
  if (hipEventRecord(t.ev[2 * t.used], s) == hipSuccess) t.open = true;
}

void timing_after(int id, hipStream_t s) {
  Timing& t = g_timing;
  if (!t.open || t.sel != id) return;
  t.open = false;
  if (hipEventRecord(t.ev[2 * t.used + 1], s) == hipSuccess) ++t.used;
}

const char* kernel_name(int id) {
  static const char* names[K_NUM_KERNELS] = {
      "route", "count_zero", "hist", "scan", "scatter", "gemm_gateup_fwd", "gemm_down_fwd",
      "combine_fwd", "combine_bwd", "route_dl", "route_dwr_partial", "route_dwr_reduce",
      "wr_transpose", "route_dx", "gemm_down_dgrad", "gemm_gateup_dgrad", "gemm_down_wgrad",
      "gemm_gateup_wgrad", "unpermute", "rank", "wr_split", "route_select", "aux_stats", "aux_grad",
      "aux_dwr", "zc_param_partial", "zc_param_reduce", "threshold_grad", "aux_partial_rows", "quant_rows",
      "weight_quant", "gemm_shared_gateup_fwd", "gemm_shared_down_fwd", "gemm_shared_down_dgrad",
      "gemm_shared_gateup_dgrad", "gemm_shared_down_wgrad", "gemm_shared_gateup_wgrad", "gemm_aux_dx",
      "gemm_aux_dwr"};
  if (id < 0 || id >= K_NUM_KERNELS) return nullptr;
  return names[id];
}

// ---------------------------------------------------------------------------
// shape checks and workspace plan
// ---------------------------------------------------------------------------
namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Experts the router chooses from: the E FFN experts and any zero-computation
// experts after them.
inline int64_t epool(const moe_shape& s) { return s.E + s.n_zero + s.n_copy + s.n_const; }
inline bool has_zc(const moe_shape& s) { return s.n_zero + s.n_copy + s.n_const > 0; }
inline bool is_thr(const moe_shape& s) { return s.router == MOE_ROUTER_SIGMOID_THRESHOLD; }
inline bool is_sigm(const moe_shape& s) { return s.router == MOE_ROUTER_SIGMOID_GROUPED || is_thr(s); }

int check_shape(const moe_shape* sh) {
  if (!sh) return moe_set_error(MOE_ERR_INVALID_ARG, "shape is NULL");
  const moe_shape& s = *sh;
  if (s.n_zero < 0 || s.n_copy < 0 || s.n_const < 0)
    return moe_set_error(MOE_ERR_INVALID_ARG, "negative zero-computation expert count");
  if (!(s.zc_aux_weight >= 0.f) || !isfinite(s.zc_aux_weight))
    return moe_set_error(MOE_ERR_INVALID_ARG, "zc_aux_weight must be finite and non-negative");
  if (has_zc(s) && (s.router == MOE_ROUTER_SIGMOID_GROUPED || s.router == MOE_ROUTER_SIGMOID_THRESHOLD))
    return moe_set_error(MOE_ERR_UNSUPPORTED, "zero-computation experts need a softmax router");
  if (s.router == MOE_ROUTER_SIGMOID_THRESHOLD && s.bias_mode != MOE_BIAS_NONE)
    return moe_set_error(MOE_ERR_UNSUPPORTED, "the threshold router takes no router bias");
  if (s.fp8 < 0 || s.fp8 > 2) return moe_set_error(MOE_ERR_INVALID_ARG, "fp8 must be 0, 1 or 2");
  if (s.fp8 && (s.dtype != MOE_BF16 || s.d % 128 || s.f % 128))
    return moe_set_error(MOE_ERR_UNSUPPORTED, "fp8 needs bf16 layers with d and f multiples of 128");
  if (s.act != MOE_ACT_SWIGLU && s.act != MOE_ACT_CLAMPED_GLU)
    return moe_set_error(MOE_ERR_INVALID_ARG, "unknown activation %d", s.act);
  if (s.act == MOE_ACT_CLAMPED_GLU &&
      (!(s.act_alpha > 0.f) || !isfinite(s.act_alpha) || !(s.act_limit > 0.f) || !isfinite(s.act_limit)))
    return moe_set_error(MOE_ERR_INVALID_ARG, "clamped GLU needs finite positive act_alpha and act_limit");
  if (s.T < 0 || s.d <= 0 || s.E <= 0 || s.k <= 0 || s.f <= 0)
    return moe_set_error(MOE_ERR_INVALID_ARG, "sizes must be positive (T >= 0): T=%lld d=%lld E=%lld k=%lld f=%lld",
                         (long long)s.T, (long long)s.d, (long long)s.E, (long long)s.k, (long long)s.f);
  if (s.k > epool(s))
    return moe_set_error(MOE_ERR_INVALID_ARG, "k=%lld exceeds the %lld experts of the pool", (long long)s.k,
                         (long long)epool(s));
  if (s.router < MOE_ROUTER_SOFTMAX_TOPK || s.router > MOE_ROUTER_SIGMOID_THRESHOLD)
    return moe_set_error(MOE_ERR_INVALID_ARG, "unknown router %d", s.router);
  if (s.bias_mode < MOE_BIAS_NONE || s.bias_mode > MOE_BIAS_LOGIT)
    return moe_set_error(MOE_ERR_INVALID_ARG, "unknown bias_mode %d", s.bias_mode);
  if (s.dtype != MOE_F32 && s.dtype != MOE_BF16)
    return moe_set_error(MOE_ERR_INVALID_ARG, "unknown dtype %d", s.dtype);
  if (s.n_groups < 1 || s.topk_groups < 1 || s.topk_groups > s.n_groups)
    return moe_set_error(MOE_ERR_INVALID_ARG, "bad groups: n_groups=%d topk_groups=%d", s.n_groups, s.topk_groups);
  if (s.E % s.n_groups)
    return moe_set_error(MOE_ERR_INVALID_ARG, "E=%lld not a multiple of n_groups=%d", (long long)s.E, s.n_groups);
  if (s.k > (s.E / s.n_groups) * s.topk_groups)
    return moe_set_error(MOE_ERR_INVALID_ARG, "k=%lld exceeds the experts of the kept groups", (long long)s.k);
  if (s.n_groups > 1 && s.router != MOE_ROUTER_SIGMOID_GROUPED)
    return moe_set_error(MOE_ERR_INVALID_ARG, "group-limited routing needs the sigmoid grouped router");
  if (!(s.route_scale > 0.f) || !isfinite(s.route_scale))
    return moe_set_error(MOE_ERR_INVALID_ARG, "route_scale must be positive and finite");
  if (s.n_shared < 0 || s.n_shared > 1)
    return moe_set_error(MOE_ERR_INVALID_ARG, "n_shared must be 0 or 1");
  if (s.n_shared && s.f_shared <= 0)
    return moe_set_error(MOE_ERR_INVALID_ARG, "f_shared must be positive with a shared expert");
  if (s.renorm != 1) return moe_set_error(MOE_ERR_UNSUPPORTED, "only renormalised top-k weights (renorm=1)");
  if (!(s.aux_coef >= 0.f) || !isfinite(s.aux_coef))
    return moe_set_error(MOE_ERR_INVALID_ARG, "aux_coef must be finite and non-negative");
  if (s.aux_coef > 0.f && s.router == MOE_ROUTER_SIGMOID_GROUPED)
    return moe_set_error(MOE_ERR_UNSUPPORTED, "the auxiliary loss is defined for the softmax routers");
  if (epool(s) > 256) return moe_set_error(MOE_ERR_UNSUPPORTED, "E_pool=%lld above 256", (long long)epool(s));
  if (s.k > 16) return moe_set_error(MOE_ERR_UNSUPPORTED, "k=%lld above 16", (long long)s.k);
  if (s.d % 64 || s.f % 64 || (s.n_shared && s.f_shared % 64))
    return moe_set_error(MOE_ERR_UNSUPPORTED, "d, f and f_shared must be multiples of 64");
  if (s.d > 16384) return moe_set_error(MOE_ERR_UNSUPPORTED, "d above 16384");
  if (s.T * s.k >= (int64_t)1 << 31 || s.T * s.d >= (int64_t)1 << 40)
    return moe_set_error(MOE_ERR_UNSUPPORTED, "T too large");
  {
    // operands staged through 32-bit buffer descriptors (the GEMMs' per-expert
    // activations and weights, the router's x, the dense passes) stay below 4 GiB
    const int64_t eb = s.dtype == MOE_BF16 ? 2 : 4;
    const int64_t R = s.T * s.k, lim = (int64_t)1 << 32;
    const int64_t wmax = s.d > 2 * s.f ? s.d : 2 * s.f;
    const int64_t shw = s.n_shared ? (s.d > 2 * s.f_shared ? s.d : 2 * s.f_shared) : 0;
    const int64_t Ep = epool(s), Epad = (Ep + 63) / 64 * 64;
    const int64_t big[4] = {R * wmax * eb, s.T * shw * eb, s.d * 2 * s.f * eb,
                            s.aux_coef > 0.f ? s.T * (Epad > s.d ? Epad : s.d) * eb : 0};
    for (int64_t b : big)
      if (b >= lim)
        return moe_set_error(MOE_ERR_UNSUPPORTED,
                             "an operand of %lld bytes exceeds the 4 GiB reach of the kernels' buffer descriptors",
                             (long long)b);
  }
  if (s.router == MOE_ROUTER_SIGMOID_GROUPED && s.n_groups > 1) {
    const int64_t epl = (s.E + 63) / 64, gs = s.E / s.n_groups;
    const int64_t lpg = gs / epl;
    if (gs % epl || lpg < 1 || (lpg & (lpg - 1)))
      return moe_set_error(MOE_ERR_UNSUPPORTED, "group size %lld does not map onto whole power-of-two lane sets",
                           (long long)gs);
  }
  return MOE_OK;
}

inline size_t act_bytes(const moe_shape& s) { return s.dtype == MOE_BF16 ? 2 : 4; }

struct Plan {
  // forward
  size_t hist, sync, cnt16, wsplit, lg, aux_part, xq, sx, hq, sh;
  size_t fwd_total;
  // backward
  size_t d_o, dgu, dx_perm, dl, partial, w_rt, dgu_sh, dx_sh;
  size_t aux_dl, aux_dx, aux_off, aux_wpart;
  size_t zc_coef, zc_part, dth;
  size_t doq, sdo, dguq, sdgu;
  size_t bwd_total;
  size_t saved_total;
};

// Auxiliary loss: experts padded to a multiple of 64 (the K of the router-dx
// product), tokens in at most 256 chunks of a multiple of 256 rows (the groups
// of the dW_r product).
inline bool has_aux(const moe_shape& s) { return s.aux_coef > 0.f; }
inline int aux_epad(const moe_shape& s) { return (int)((epool(s) + 63) / 64 * 64); }
inline int64_t aux_chunk(const moe_shape& s) { return 256 * ((s.T + 256 * 256 - 1) / (256 * 256)); }
inline int aux_groups(const moe_shape& s) { return s.T > 0 ? (int)((s.T + aux_chunk(s) - 1) / aux_chunk(s)) : 0; }

Plan plan(const moe_shape& s) {
  Plan p{};
  const size_t eb = act_bytes(s);
  const int64_t R = s.T * s.k;
  size_t off = 0;
  const int64_t Ep = epool(s);
  p.hist = off;
  off += align_up((size_t)moe::perm_blocks(s.T) * Ep * 4);
  p.sync = off;
  off += align_up(4);
  p.cnt16 = off;
  off += align_up((size_t)((s.T + 15) / 16) * Ep * 4);
  p.wsplit = off;
  off += s.dtype == MOE_BF16 ? align_up((size_t)3 * Ep * s.d * 2) : 0;
  p.lg = off;
  off += s.dtype == MOE_BF16 ? align_up((size_t)s.T * Ep * 8) : 0;
  p.aux_part = off;
  off += has_aux(s) ? align_up((size_t)aux_blocks(s.T) * Ep * 8) : 0;
  // FP8 forward: E4M3 rows of x_perm and h, and their scales
  p.xq = off; off += s.fp8 ? align_up((size_t)R * s.d) : 0;
  p.sx = off; off += s.fp8 ? align_up((size_t)R * 4) : 0;
  p.hq = off; off += s.fp8 ? align_up((size_t)R * s.f) : 0;
  p.sh = off; off += s.fp8 ? align_up((size_t)R * 4) : 0;
  p.fwd_total = off;
  off = 0;
  p.d_o = off; off += align_up((size_t)R * s.d * eb);
  p.dgu = off; off += align_up((size_t)R * 2 * s.f * eb);
  p.dx_perm = off; off += align_up((size_t)R * s.d * eb);
  p.dl = off; off += align_up((size_t)R * 4);
  p.partial = off; off += align_up((size_t)moe::route_dwr_tasks(R, Ep) * s.d * 4);
  p.w_rt = off; off += align_up((size_t)(has_aux(s) ? aux_epad(s) : Ep) * s.d * 4);
  p.dgu_sh = off; off += s.n_shared ? align_up((size_t)s.T * 2 * s.f_shared * eb) : 0;
  p.dx_sh = off; off += s.n_shared ? align_up((size_t)s.T * s.d * eb) : 0;
  const bool aux = has_aux(s);
  p.aux_dl = off; off += aux ? align_up((size_t)s.T * aux_epad(s) * eb) : 0;
  p.aux_dx = off; off += aux ? align_up((size_t)s.T * s.d * eb) : 0;
  p.aux_off = off; off += aux ? align_up((size_t)(aux_groups(s) + 1) * 4) : 0;
  p.aux_wpart = off; off += aux ? align_up((size_t)aux_groups(s) * s.d * aux_epad(s) * eb) : 0;
  p.zc_coef = off; off += has_zc(s) ? align_up((size_t)R * 16) : 0;
  p.zc_part = off; off += s.n_const > 0 ? align_up((size_t)moe::route_dwr_tasks(R, s.n_const) * 3 * s.d * 4) : 0;
  p.dth = off; off += is_thr(s) ? align_up((size_t)R * 4) : 0;
  // FP8 data-gradient GEMMs: E4M3 rows of d_o and dgu, and their scales
  const bool q2 = s.fp8 == 2;
  p.doq = off; off += q2 ? align_up((size_t)R * s.d) : 0;
  p.sdo = off; off += q2 ? align_up((size_t)R * 4) : 0;
  p.dguq = off; off += q2 ? align_up((size_t)R * 2 * s.f) : 0;
  p.sdgu = off; off += q2 ? align_up((size_t)R * 4) : 0;
  p.bwd_total = off;
  size_t sv = 0;
  sv += (size_t)R * (4 + 4 + 4 + 4 + 4);  // topk_idx, topk_w, s_sel, row_of, token_of
  sv += (size_t)(Ep + 1) * 4;
  sv += (size_t)R * (s.d + 2 * s.f + s.f + s.d) * eb;
  if (s.n_shared) sv += (size_t)s.T * (2 * s.f_shared + s.f_shared + s.d) * eb;
  if (has_aux(s)) sv += (size_t)s.T * Ep * 4 + 4;
  p.saved_total = sv;
  return p;
}

inline char* wsp(void* ws, size_t off) { return static_cast<char*>(ws) + off; }

int check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return MOE_OK;
  if (!ws) return moe_set_error(MOE_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (have < need) return moe_set_error(MOE_ERR_WORKSPACE, "workspace %zu bytes, %zu needed", have, need);
  return MOE_OK;
}

#define MOE_NEED(p, name)                                                        \
  do {                                                                           \
    if (!(p)) return moe_set_error(MOE_ERR_INVALID_ARG, "%s is NULL", name);     \
  } while (0)

#define MOE_TRY(expr)      \
  do {                     \
    int st_ = (expr);      \
    if (st_) return st_;   \
  } while (0)

GemmArgs gemm_base(const moe_shape& s, int mode, const int32_t* offsets) {
  GemmArgs g{};
  g.mode = mode;
  g.bf16 = s.dtype == MOE_BF16;
  g.offsets = offsets;
  g.ngroups = (int)s.E;
  g.dense_rows = 0;
  g.max_rows = s.T * s.k;
  g.d = (int)s.d;
  g.f = (int)s.f;
  g.act = s.act;
  g.act_alpha = s.act_alpha;
  g.act_limit = s.act_limit;
  return g;
}

// The shared expert (and the dense products of the auxiliary loss): SwiGLU.
// FP8 weight cache regions: codes of gate, up [E][f][d] and down [E][d][f],
// then the column maxima and scales of each (float32); with the data-gradient
// GEMMs (fp8 = 2) also the row codes of [W_gate | W_up] [E][d][2f] and of
// W_down [E][f][d] and their row scales.
struct CachePlan {
  size_t qg, qu, qd, ag, au, ad, sg, su, sd;
  size_t qgu_r, qd_r, sgu_r, sd_r;
  size_t total;
};
CachePlan cache_plan(const moe_shape& s) {
  CachePlan c{};
  size_t off = 0;
  const size_t efd = (size_t)s.E * s.f * s.d;
  c.qg = off; off += align_up(efd);
  c.qu = off; off += align_up(efd);
  c.qd = off; off += align_up(efd);
  c.ag = off; off += align_up((size_t)s.E * s.f * 4);
  c.au = off; off += align_up((size_t)s.E * s.f * 4);
  c.ad = off; off += align_up((size_t)s.E * s.d * 4);
  c.sg = off; off += align_up((size_t)s.E * s.f * 4);
  c.su = off; off += align_up((size_t)s.E * s.f * 4);
  c.sd = off; off += align_up((size_t)s.E * s.d * 4);
  const bool q2 = s.fp8 == 2;
  c.qgu_r = off; off += q2 ? align_up(2 * efd) : 0;
  c.qd_r = off; off += q2 ? align_up(efd) : 0;
  c.sgu_r = off; off += q2 ? align_up((size_t)s.E * s.d * 4) : 0;
  c.sd_r = off; off += q2 ? align_up((size_t)s.E * s.f * 4) : 0;
  c.total = off;
  return c;
}

GemmArgs gemm_dense(const moe_shape& s, int mode) {
  static const int kid[6] = {K_GEMM_SH_GATEUP_FWD, K_GEMM_SH_DOWN_FWD, K_GEMM_SH_DOWN_DGRAD,
                             K_GEMM_SH_GATEUP_DGRAD, K_GEMM_SH_DOWN_WGRAD, K_GEMM_SH_GATEUP_WGRAD};
  GemmArgs g = gemm_base(s, mode, nullptr);
  g.kid = kid[mode];
  g.ngroups = 1;
  g.dense_rows = s.T;
  g.max_rows = s.T;
  g.f = (int)s.f_shared;
  g.act = MOE_ACT_SWIGLU;
  g.fp8 = false;
  return g;
}

// maps (may be null): the forward layer's expert_offsets; the selection then
// also builds the permutation's block bases and offsets when it can, and
// *maps_built says whether it did
int do_route(const moe_shape& s, const void* x, const float* w_r, const float* bias, int32_t* topk_idx,
             float* topk_w, float* s_sel, int32_t* counts, void* ws, hipStream_t st, float* probs = nullptr,
             const float* threshold = nullptr, int32_t* maps_offsets = nullptr, int32_t* maps_row_of = nullptr,
             bool* maps_built = nullptr) {
  RouteArgs a{};
  if (maps_offsets) {
    a.hist = reinterpret_cast<int32_t*>(wsp(ws, plan(s).hist));
    a.sync = reinterpret_cast<int32_t*>(wsp(ws, plan(s).sync));
    a.cnt16 = reinterpret_cast<int32_t*>(wsp(ws, plan(s).cnt16));
    a.offsets = maps_offsets;
    a.row_of = maps_row_of;
  }
  a.probs = probs;
  a.threshold = threshold;
  a.wsplit = s.dtype == MOE_BF16 ? wsp(ws, plan(s).wsplit) : nullptr;
  a.lg = s.dtype == MOE_BF16 ? reinterpret_cast<double*>(wsp(ws, plan(s).lg)) : nullptr;
  a.x = x;
  a.w_r = w_r;
  a.bias = bias;
  a.T = s.T;
  a.d = (int)s.d;
  a.E = (int)epool(s);
  a.k = (int)s.k;
  a.router = s.router;
  a.bias_mode = s.bias_mode;
  a.n_groups = s.n_groups;
  a.topk_groups = s.topk_groups;
  a.route_scale = s.route_scale;
  a.bf16 = s.dtype == MOE_BF16;
  a.topk_idx = topk_idx;
  a.topk_w = topk_w;
  a.s_sel = s_sel;
  a.counts = counts;
  return launch_route(a, st, maps_built);
}

int do_permute(const moe_shape& s, const void* x, const int32_t* topk_idx, int32_t* offsets, int32_t* row_of,
               int32_t* token_of, void* x_perm, void* ws, hipStream_t st, bool fp8_rows = false,
               bool maps_ready = false) {
  PermArgs a{};
  a.maps_ready = maps_ready;
  a.cnt16 = reinterpret_cast<const int32_t*>(wsp(ws, plan(s).cnt16));
  a.x = x;
  a.topk_idx = topk_idx;
  a.T = s.T;
  a.d = (int)s.d;
  a.E = (int)epool(s);
  a.E_rows = (int)s.E;
  a.k = (int)s.k;
  a.bf16 = s.dtype == MOE_BF16;
  a.hist = reinterpret_cast<int32_t*>(wsp(ws, plan(s).hist));
  a.offsets = offsets;
  a.row_of = row_of;
  a.token_of = token_of;
  a.x_perm = x_perm;
  if (fp8_rows) {
    a.xq = reinterpret_cast<uint8_t*>(wsp(ws, plan(s).xq));
    a.sx = reinterpret_cast<float*>(wsp(ws, plan(s).sx));
  }
  return launch_permute(a, st);
}

// FP8 forward of the routed experts: E4M3 x rows (written by the permutation)
// and cached weights through the gate/up GEMM, E4M3 h rows through the down GEMM.
int do_gemm_fwd_fp8(const moe_shape& s, const int32_t* offsets, const void* cache, const void* b_gate,
                    const void* b_up, const void* b_down, void* gu, void* h, void* o, void* ws, hipStream_t st) {
  const Plan p = plan(s);
  const CachePlan c = cache_plan(s);
  const char* cb = static_cast<const char*>(cache);
  GemmArgs g = gemm_base(s, G_FWD_GATEUP, offsets);
  g.fp8 = true;
  g.a = wsp(ws, p.xq);
  g.a_scale = reinterpret_cast<const float*>(wsp(ws, p.sx));
  g.w0 = cb + c.qg;
  g.w1 = cb + c.qu;
  g.b_scale0 = reinterpret_cast<const float*>(cb + c.sg);
  g.b_scale1 = reinterpret_cast<const float*>(cb + c.su);
  g.bias0 = b_gate;
  g.bias1 = b_up;
  g.c0 = gu;
  g.c1 = h;
  MOE_TRY(launch_gemm(g, st));
  uint8_t* hq = reinterpret_cast<uint8_t*>(wsp(ws, p.hq));
  float* sh = reinterpret_cast<float*>(wsp(ws, p.sh));
  MOE_TRY(launch_quant_rows(h, nullptr, (int)s.f, 0, offsets, (int)s.E, s.T * s.k, hq, sh, st));
  g = gemm_base(s, G_FWD_DOWN, offsets);
  g.fp8 = true;
  g.a = hq;
  g.a_scale = sh;
  g.w0 = cb + c.qd;
  g.b_scale0 = reinterpret_cast<const float*>(cb + c.sd);
  g.bias0 = b_down;
  g.c0 = o;
  return launch_gemm(g, st);
}

// FP8 data-gradient GEMMs of the routed experts: E4M3 rows of d_o through the
// down dgrad (dSwiGLU in its epilogue, dgu stored bf16 for the weight
// gradients), E4M3 rows of dgu through the gate/up dgrad, both against the
// row-quantised weights of the cache.
int do_gemm_dgrad_fp8(const moe_shape& s, const int32_t* offsets, const void* cache, const void* gu, const void* d_o,
                      bool d_o_quantised, void* dgu, void* dx_perm, void* ws, hipStream_t st) {
  const Plan p = plan(s);
  const CachePlan c = cache_plan(s);
  const char* cb = static_cast<const char*>(cache);
  const int64_t R = s.T * s.k;
  uint8_t* doq = reinterpret_cast<uint8_t*>(wsp(ws, p.doq));
  float* sdo = reinterpret_cast<float*>(wsp(ws, p.sdo));
  if (!d_o_quantised)  // (the combine backward writes them where it can)
    MOE_TRY(launch_quant_rows(d_o, nullptr, (int)s.d, 0, offsets, (int)s.E, R, doq, sdo, st));
  GemmArgs g = gemm_base(s, G_DGRAD_DOWN, offsets);
  g.fp8 = true;
  g.a = doq;
  g.a_scale = sdo;
  g.w0 = cb + c.qd_r;
  g.b_scale0 = reinterpret_cast<const float*>(cb + c.sd_r);
  g.aux = gu;
  g.c0 = dgu;
  MOE_TRY(launch_gemm(g, st));
  uint8_t* dguq = reinterpret_cast<uint8_t*>(wsp(ws, p.dguq));
  float* sdgu = reinterpret_cast<float*>(wsp(ws, p.sdgu));
  MOE_TRY(launch_quant_rows(dgu, nullptr, 2 * (int)s.f, 0, offsets, (int)s.E, R, dguq, sdgu, st));
  g = gemm_base(s, G_DGRAD_GATEUP, offsets);
  g.fp8 = true;
  g.a = dguq;
  g.a_scale = sdgu;
  g.w0 = cb + c.qgu_r;
  g.b_scale0 = reinterpret_cast<const float*>(cb + c.sgu_r);
  g.c0 = dx_perm;
  return launch_gemm(g, st);
}

int do_gemm_fwd(const moe_shape& s, const void* x_perm, const int32_t* offsets, const void* w_gate, const void* w_up,
                const void* w_down, const void* b_gate, const void* b_up, const void* b_down, void* gu, void* h,
                void* o, hipStream_t st) {
  GemmArgs g = gemm_base(s, G_FWD_GATEUP, offsets);
  g.a = x_perm;
  g.w0 = w_gate;
  g.w1 = w_up;
  g.bias0 = b_gate;
  g.bias1 = b_up;
  g.c0 = gu;
  g.c1 = h;
  MOE_TRY(launch_gemm(g, st));
  g = gemm_base(s, G_FWD_DOWN, offsets);
  g.a = h;
  g.w0 = w_down;
  g.bias0 = b_down;
  g.c0 = o;
  return launch_gemm(g, st);
}

int do_gemm_bwd(const moe_shape& s, int passes, const void* x_perm, const int32_t* offsets, const void* gu,
                const void* h, const void* d_o, const void* w_gate, const void* w_up, const void* w_down, void* dgu,
                void* dx_perm, void* dw_gate, void* dw_up, void* dw_down, void* db_gate, void* db_up, void* db_down,
                hipStream_t st) {
  if (passes & MOE_DGRAD) {
    GemmArgs g = gemm_base(s, G_DGRAD_DOWN, offsets);
    g.a = d_o;
    g.w0 = w_down;
    g.aux = gu;
    g.c0 = dgu;
    MOE_TRY(launch_gemm(g, st));
    g = gemm_base(s, G_DGRAD_GATEUP, offsets);
    g.a = dgu;
    g.w0 = w_gate;
    g.w1 = w_up;
    g.c0 = dx_perm;
    MOE_TRY(launch_gemm(g, st));
  }
  if (passes & MOE_WGRAD) {
    GemmArgs g = gemm_base(s, G_WGRAD_DOWN, offsets);
    g.a = h;
    g.b = d_o;
    g.c0 = dw_down;
    g.db0 = db_down;
    g.accumulate = (passes & MOE_ACCUMULATE) != 0;
    MOE_TRY(launch_gemm(g, st));
    g = gemm_base(s, G_WGRAD_GATEUP, offsets);
    g.a = x_perm;
    g.b = dgu;
    g.c0 = dw_gate;
    g.c1 = dw_up;
    g.db0 = db_gate;
    g.db1 = db_up;
    g.accumulate = (passes & MOE_ACCUMULATE) != 0;
    MOE_TRY(launch_gemm(g, st));
  }
  return MOE_OK;
}

int do_shared_fwd(const moe_shape& s, const void* x, const void* wsg, const void* wsu, const void* wsd, void* gu_sh,
                  void* h_sh, void* o_sh, hipStream_t st) {
  GemmArgs g = gemm_dense(s, G_FWD_GATEUP);
  g.a = x;
  g.w0 = wsg;
  g.w1 = wsu;
  g.c0 = gu_sh;
  g.c1 = h_sh;
  MOE_TRY(launch_gemm(g, st));
  g = gemm_dense(s, G_FWD_DOWN);
  g.a = h_sh;
  g.w0 = wsd;
  g.c0 = o_sh;
  return launch_gemm(g, st);
}

// Shared expert backward: the input-gradient half (dgu_sh, dx_sh) ...
int do_shared_dgrad(const moe_shape& s, const void* dy, const void* gu_sh, const void* wsg, const void* wsu,
                    const void* wsd, void* dgu_sh, void* dx_sh, hipStream_t st) {
  GemmArgs g = gemm_dense(s, G_DGRAD_DOWN);
  g.a = dy;
  g.w0 = wsd;
  g.aux = gu_sh;
  g.c0 = dgu_sh;
  MOE_TRY(launch_gemm(g, st));
  g = gemm_dense(s, G_DGRAD_GATEUP);
  g.a = dgu_sh;
  g.w0 = wsg;
  g.w1 = wsu;
  g.c0 = dx_sh;
  return launch_gemm(g, st);
}

// ... and the weight-gradient half, from dgu_sh kept by the first.
int do_shared_wgrad(const moe_shape& s, const void* x, const void* dy, const void* h_sh, const void* dgu_sh,
                    void* dwsg, void* dwsu, void* dwsd, bool accumulate, hipStream_t st) {
  GemmArgs g = gemm_dense(s, G_WGRAD_DOWN);
  g.a = h_sh;
  g.b = dy;
  g.c0 = dwsd;
  g.accumulate = accumulate;
  MOE_TRY(launch_gemm(g, st));
  g = gemm_dense(s, G_WGRAD_GATEUP);
  g.a = x;
  g.b = dgu_sh;
  g.c0 = dwsg;
  g.c1 = dwsu;
  g.accumulate = accumulate;
  return launch_gemm(g, st);
}

int do_shared_bwd(const moe_shape& s, const void* x, const void* dy, const void* gu_sh, const void* h_sh,
                  const void* wsg, const void* wsu, const void* wsd, void* dgu_sh, void* dx_sh, void* dwsg, void* dwsu,
                  void* dwsd, hipStream_t st) {
  MOE_TRY(do_shared_dgrad(s, dy, gu_sh, wsg, wsu, wsd, dgu_sh, dx_sh, st));
  return do_shared_wgrad(s, x, dy, h_sh, dgu_sh, dwsg, dwsu, dwsd, false, st);
}

AuxArgs aux_args(const moe_shape& s, const moe_params* prm, const moe_saved* sv) {
  AuxArgs a{};
  a.probs = sv->router_probs;
  a.offsets = sv->expert_offsets;
  a.aux_f = prm->aux_f;
  a.T = s.T;
  a.E = (int)epool(s);
  a.k = (int)s.k;
  a.coef = s.aux_coef;
  a.E_ffn = has_zc(s) ? (int)s.E : (int)epool(s);
  a.zc_weight = s.zc_aux_weight;
  a.thr = is_thr(s);
  a.loss = sv->aux_loss;
  return a;
}

// Zero-computation experts' arguments of the gather-side kernels.
ZcArgs zc_args(const moe_shape& s, const moe_params* prm, const void* x, const void* dy, void* coef) {
  ZcArgs z{};
  z.on = has_zc(s);
  z.E_ffn = (int)s.E;
  z.n_zero = s.n_zero;
  z.n_copy = s.n_copy;
  z.n_const = s.n_const;
  z.x = x;
  z.v = prm->zc_v;
  z.wc = prm->zc_wc;
  z.coef = reinterpret_cast<float4*>(coef);
  z.dy = dy;
  return z;
}

RouteBwdArgs route_bwd_base(const moe_shape& s) {
  RouteBwdArgs a{};
  a.T = s.T;
  a.d = (int)s.d;
  a.E = (int)epool(s);
  a.k = (int)s.k;
  a.router = s.router;
  a.route_scale = s.route_scale;
  a.bf16 = s.dtype == MOE_BF16;
  return a;
}

}  // namespace
}  // namespace moe

using namespace moe;

// The Python binding mirrors these layouts field by field.
static_assert(sizeof(moe_shape) == 128 && offsetof(moe_shape, f_shared) == 56 &&
                  offsetof(moe_shape, aux_coef) == 88 && offsetof(moe_shape, zc_aux_weight) == 104 &&
                  offsetof(moe_shape, act_limit) == 116 && offsetof(moe_shape, fp8) == 120,
              "moe_shape layout");
static_assert(sizeof(moe_params) == 17 * sizeof(void*) && offsetof(moe_params, fp8_cache_bytes) == 128 &&
                  sizeof(moe_saved) == 15 * sizeof(void*) &&
                  sizeof(moe_grads) == 13 * sizeof(void*),
              "pointer struct layouts");

// ---------------------------------------------------------------------------
// exported entry points
// ---------------------------------------------------------------------------
namespace {
// The FP8 weight cache must hold the regions the shape's fp8 level reads.
int check_fp8_cache(const moe_shape& s, const moe_params* prm) {
  const size_t need = cache_plan(s).total;
  if (prm->fp8_cache_bytes < need)
    return moe_set_error(MOE_ERR_WORKSPACE, "params.fp8_cache_bytes %zu, the shape's cache needs %zu",
                         prm->fp8_cache_bytes, need);
  return MOE_OK;
}

// Argument checks of the layer backward; `phase` bit 1: input-gradient half,
// bit 2: weight-gradient half.
int check_layer_bwd(const moe_shape& s, const moe_params* prm, const void* x, const moe_saved* sv, const void* dy,
                    const void* dx, const moe_grads* gr, int phase) {
  MOE_NEED(prm, "params");
  MOE_NEED(sv, "saved");
  MOE_NEED(prm->w_r, "params.w_r");
  MOE_NEED(sv->expert_offsets, "saved.expert_offsets");
  if (s.fp8 == 2 && (phase & 1)) {
    MOE_NEED(prm->fp8_cache, "params.fp8_cache");
    MOE_TRY(check_fp8_cache(s, prm));
  }
  if (s.n_const > 0 && (phase & 1)) {
    MOE_NEED(prm->zc_v, "params.zc_v");
    MOE_NEED(prm->zc_wc, "params.zc_wc");
  }
  if (s.n_const > 0 && (phase & 2)) {
    MOE_NEED(gr, "grads");
    MOE_NEED(gr->dzc_v, "grads.dzc_v");
    MOE_NEED(gr->dzc_wc, "grads.dzc_wc");
  }
  if (is_thr(s) && (phase & 2)) {
    MOE_NEED(gr, "grads");
    MOE_NEED(gr->d_threshold, "grads.d_threshold");
  }
  if (phase & 1) {
    MOE_NEED(prm->w_gate, "params.w_gate");
    MOE_NEED(prm->w_up, "params.w_up");
    MOE_NEED(prm->w_down, "params.w_down");
    if (s.n_shared) {
      MOE_NEED(prm->ws_gate, "params.ws_gate");
      MOE_NEED(prm->ws_up, "params.ws_up");
      MOE_NEED(prm->ws_down, "params.ws_down");
    }
  }
  if (phase & 2) {
    MOE_NEED(gr, "grads");
    MOE_NEED(gr->dw_r, "grads.dw_r");
    MOE_NEED(gr->dw_gate, "grads.dw_gate");
    MOE_NEED(gr->dw_up, "grads.dw_up");
    MOE_NEED(gr->dw_down, "grads.dw_down");
    if (s.expert_bias) {
      MOE_NEED(gr->db_gate, "grads.db_gate");
      MOE_NEED(gr->db_up, "grads.db_up");
      MOE_NEED(gr->db_down, "grads.db_down");
    }
    if (s.n_shared) {
      MOE_NEED(gr->dws_gate, "grads.dws_gate");
      MOE_NEED(gr->dws_up, "grads.dws_up");
      MOE_NEED(gr->dws_down, "grads.dws_down");
    }
  }
  if (s.T > 0) {
    MOE_NEED(x, "x");
    MOE_NEED(dy, "dy");
    MOE_NEED(sv->topk_idx, "saved.topk_idx");
    if (phase & 1) {
      MOE_NEED(dx, "dx");
      MOE_NEED(sv->topk_w, "saved.topk_w");
      MOE_NEED(sv->row_of, "saved.row_of");
      MOE_NEED(sv->gu, "saved.gu");
      MOE_NEED(sv->o, "saved.o");
      if (is_sigm(s)) MOE_NEED(sv->s_sel, "saved.s_sel");
      if (s.n_shared) MOE_NEED(sv->gu_sh, "saved.gu_sh");
      if (has_aux(s)) MOE_NEED(sv->router_probs, "saved.router_probs");
    }
    if (phase & 2) {
      MOE_NEED(sv->token_of, "saved.token_of");
      MOE_NEED(sv->x_perm, "saved.x_perm");
      MOE_NEED(sv->h, "saved.h");
      if (s.n_shared) MOE_NEED(sv->h_sh, "saved.h_sh");
    }
  }
  return MOE_OK;
}

// Input-gradient half: combine backward with the router's dl, expert dgrads,
// shared-expert dgrad, and dx.  Leaves d_o, dgu, dl (and dgu_sh) in ws.
int layer_bwd_dgrad(const moe_shape& s, const moe_params* prm, const void* x, const moe_saved* sv, const void* dy,
                    void* dx, const Plan& p, void* ws, hipStream_t stream) {
  void* d_o = wsp(ws, p.d_o);
  void* dgu = wsp(ws, p.dgu);
  void* dx_perm = wsp(ws, p.dx_perm);
  float* dl = reinterpret_cast<float*>(wsp(ws, p.dl));
  float* w_rt = reinterpret_cast<float*>(wsp(ws, p.w_rt));
  // 1. combine backward with the router's dl fused in
  CombineBwdArgs cb{};
  cb.dy = dy;
  cb.o = sv->o;
  cb.topk_w = sv->topk_w;
  cb.row_of = sv->row_of;
  cb.d_o = d_o;
  cb.d_topk_w = nullptr;
  cb.T = s.T;
  cb.d = (int)s.d;
  cb.k = (int)s.k;
  cb.bf16 = s.dtype == MOE_BF16;
  cb.dl = dl;
  cb.s_sel = sv->s_sel;
  cb.router = s.router;
  cb.route_scale = s.route_scale;
  cb.topk_idx = sv->topk_idx;
  cb.zc = zc_args(s, prm, x, dy, wsp(ws, p.zc_coef));
  cb.dth = is_thr(s) ? reinterpret_cast<float*>(wsp(ws, p.dth)) : nullptr;
  // FP8 data gradients: the E4M3 rows of d_o come with it (except with
  // zero-computation experts, whose combine kernel does not write them)
  const bool doq_fused = s.fp8 == 2 && !has_zc(s);
  cb.doq = doq_fused ? reinterpret_cast<uint8_t*>(wsp(ws, p.doq)) : nullptr;
  cb.sdo = doq_fused ? reinterpret_cast<float*>(wsp(ws, p.sdo)) : nullptr;
  MOE_TRY(launch_combine_bwd(cb, stream));
  // 2. expert dgrads
  if (s.fp8 == 2)
    MOE_TRY(do_gemm_dgrad_fp8(s, sv->expert_offsets, prm->fp8_cache, sv->gu, d_o, doq_fused, dgu, dx_perm, ws,
                              stream));
  else
    MOE_TRY(do_gemm_bwd(s, MOE_DGRAD, nullptr, sv->expert_offsets, sv->gu, nullptr, d_o, prm->w_gate, prm->w_up,
                        prm->w_down, dgu, dx_perm, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, stream));
  // 3. W_r^T for the router dx fused into the unpermute (zero rows up to the
  //    auxiliary loss's padded expert count)
  const bool aux = has_aux(s) && s.T > 0;
  const int Ep = (int)epool(s);
  const int E_rt = aux ? aux_epad(s) : Ep;
  MOE_TRY(launch_wr_transpose_act(prm->w_r, w_rt, (int)s.d, Ep, E_rt, s.dtype == MOE_BF16, stream));
  // 3b. auxiliary loss: its dense logit gradient, kept for the weight half,
  //     and its router dx = dl_aux W_r^T (a dense down-projection product)
  void* aux_dx = nullptr;
  if (aux) {
    void* aux_dl = wsp(ws, p.aux_dl);
    aux_dx = wsp(ws, p.aux_dx);
    MOE_TRY(launch_aux_grad(aux_args(s, prm, sv), aux_dl, E_rt, reinterpret_cast<int32_t*>(wsp(ws, p.aux_off)),
                            aux_groups(s), aux_chunk(s), s.dtype == MOE_BF16, stream));
    GemmArgs g = gemm_base(s, G_FWD_DOWN, nullptr);
    g.ngroups = 1;
    g.dense_rows = s.T;
    g.max_rows = s.T;
    g.f = E_rt;
    g.a = aux_dl;
    g.w0 = w_rt;
    g.c0 = aux_dx;
    g.kid = K_GEMM_AUX_DX;
    MOE_TRY(launch_gemm(g, stream));
  }
  // 4. shared expert input gradient
  void* dx_sh = nullptr;
  if (s.n_shared) {
    dx_sh = wsp(ws, p.dx_sh);
    MOE_TRY(do_shared_dgrad(s, dy, sv->gu_sh, prm->ws_gate, prm->ws_up, prm->ws_down, wsp(ws, p.dgu_sh), dx_sh,
                            stream));
  }
  // 5. dx = unpermute(dx_perm) + router dx + shared dx
  UnpermuteArgs u{};
  u.dx_perm = dx_perm;
  u.row_of = sv->row_of;
  u.dx_router = nullptr;
  u.dx_shared = dx_sh;
  u.dx_aux = aux_dx;
  u.dl = dl;
  u.topk_idx = sv->topk_idx;
  u.w_rt = w_rt;
  u.dx = dx;
  u.T = s.T;
  u.d = (int)s.d;
  u.k = (int)s.k;
  u.bf16 = s.dtype == MOE_BF16;
  u.zc = zc_args(s, prm, x, dy, wsp(ws, p.zc_coef));
  return launch_unpermute(u, stream);
}

// Weight-gradient half, from d_o, dgu, dl (and dgu_sh) left in ws by the
// input-gradient half.
int layer_bwd_wgrad(const moe_shape& s, const moe_params* prm, const void* x, const moe_saved* sv, const void* dy,
                    const moe_grads* gr, bool accumulate, const Plan& p, void* ws, hipStream_t stream) {
  void* d_o = wsp(ws, p.d_o);
  void* dgu = wsp(ws, p.dgu);
  float* dl = reinterpret_cast<float*>(wsp(ws, p.dl));
  MOE_TRY(do_gemm_bwd(s, MOE_WGRAD | (accumulate ? MOE_ACCUMULATE : 0), sv->x_perm, sv->expert_offsets, nullptr,
                      sv->h, d_o, nullptr, nullptr, nullptr, dgu, nullptr, gr->dw_gate, gr->dw_up, gr->dw_down,
                      s.expert_bias ? gr->db_gate : nullptr, s.expert_bias ? gr->db_up : nullptr,
                      s.expert_bias ? gr->db_down : nullptr, stream));
  RouteBwdArgs rb = route_bwd_base(s);
  rb.x = x;
  rb.w_r = prm->w_r;
  rb.topk_idx = sv->topk_idx;
  rb.dl_in = dl;
  rb.offsets = sv->expert_offsets;
  rb.token_of = sv->token_of;
  rb.dw_r = gr->dw_r;
  rb.dx_router = nullptr;
  rb.partial = reinterpret_cast<float*>(wsp(ws, p.partial));
  rb.accumulate = accumulate;
  MOE_TRY(launch_route_bwd(rb, stream));
  if (has_aux(s) && s.T > 0) {
    // auxiliary loss: dW_r += x^T dl_aux, as per-chunk products of the grouped
    // weight-gradient GEMM (chunks of tokens as the groups), summed in order
    const int G = aux_groups(s), E_pad = aux_epad(s);
    const int32_t* off = reinterpret_cast<const int32_t*>(wsp(ws, p.aux_off));  // written with dl_aux
    void* part = wsp(ws, p.aux_wpart);
    GemmArgs g = gemm_base(s, G_WGRAD_DOWN, off);
    g.ngroups = G;
    g.max_rows = s.T;
    g.f = (int)s.d;
    g.d = E_pad;
    g.a = x;
    g.b = wsp(ws, p.aux_dl);
    g.c0 = part;
    g.kid = K_GEMM_AUX_DWR;
    MOE_TRY(launch_gemm(g, stream));
    MOE_TRY(launch_aux_dwr(part, G, (int)s.d, (int)epool(s), E_pad, s.dtype == MOE_BF16, gr->dw_r, stream));
  }
  if (is_thr(s))
    MOE_TRY(launch_threshold_grad(sv->expert_offsets, sv->token_of, reinterpret_cast<const float*>(wsp(ws, p.dth)),
                                  (int)s.E, gr->d_threshold, accumulate, stream));
  if (s.n_const > 0) {
    // constant experts' dv and dW_c over their rows
    ZcParamArgs z{};
    z.x = x;
    z.dy = dy;
    z.coef = reinterpret_cast<const float4*>(wsp(ws, p.zc_coef));
    z.offsets = sv->expert_offsets;
    z.token_of = sv->token_of;
    z.T = s.T;
    z.d = (int)s.d;
    z.k = (int)s.k;
    z.e0 = (int)(s.E + s.n_zero + s.n_copy);
    z.n_const = s.n_const;
    z.bf16 = s.dtype == MOE_BF16;
    z.partial = reinterpret_cast<float*>(wsp(ws, p.zc_part));
    z.dwc = gr->dzc_wc;
    z.dv = gr->dzc_v;
    z.accumulate = accumulate;
    MOE_TRY(launch_zc_param_grads(z, stream));
  }
  if (s.n_shared)
    MOE_TRY(do_shared_wgrad(s, x, dy, sv->h_sh, wsp(ws, p.dgu_sh), gr->dws_gate, gr->dws_up, gr->dws_down,
                            accumulate, stream));
  return MOE_OK;
}
}  // namespace

extern "C" {

const char* moe_status_string(int status) {
  switch (status) {
    case MOE_OK: return "ok";
    case MOE_ERR_INVALID_ARG: return "invalid argument";
    case MOE_ERR_UNSUPPORTED: return "unsupported shape or option";
    case MOE_ERR_HIP: return "HIP launch failure";
    case MOE_ERR_WORKSPACE: return "workspace missing or too small";
  }
  return "unknown status";
}

const char* moe_last_error(void) { return g_err; }

int moe_kernel_count(void) { return K_NUM_KERNELS; }
const char* moe_kernel_name(int id) { return kernel_name(id); }

int moe_timing_select(int id) {
  g_timing.sel = id;
  g_timing.used = 0;
  g_timing.open = false;
  return MOE_OK;
}

int moe_timing_read(double* total_ms, int* launches) {
  double tot = 0.0;
  for (int i = 0; i < g_timing.used; ++i) {
    if (hipEventSynchronize(g_timing.ev[2 * i + 1]) != hipSuccess)
      return moe_set_error(MOE_ERR_HIP, "event synchronize failed");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, g_timing.ev[2 * i], g_timing.ev[2 * i + 1]) != hipSuccess)
      return moe_set_error(MOE_ERR_HIP, "event elapsed time failed");
    tot += ms;
  }
  if (total_ms) *total_ms = tot;
  if (launches) *launches = g_timing.used;
  return MOE_OK;
}

int moe_fp8_cache_size(const moe_shape* shape, size_t* bytes) {
  MOE_TRY(check_shape(shape));
  if (!shape->fp8) return moe_set_error(MOE_ERR_UNSUPPORTED, "moe_fp8_cache_size: shape->fp8 is 0");
  MOE_NEED(bytes, "bytes");
  *bytes = cache_plan(*shape).total;
  return MOE_OK;
}

int moe_fp8_cache_build(const moe_shape* shape, const void* w_gate, const void* w_up, const void* w_down, void* cache,
                        size_t cache_bytes, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  if (!s.fp8) return moe_set_error(MOE_ERR_UNSUPPORTED, "moe_fp8_cache_build: shape->fp8 is 0");
  MOE_NEED(w_gate, "w_gate");
  MOE_NEED(w_up, "w_up");
  MOE_NEED(w_down, "w_down");
  const CachePlan c = cache_plan(s);
  MOE_TRY(check_ws(cache, cache_bytes, c.total));
  char* cb = static_cast<char*>(cache);
  auto F = [&](size_t off) { return reinterpret_cast<float*>(cb + off); };
  auto Q = [&](size_t off) { return reinterpret_cast<uint8_t*>(cb + off); };
  const int E = (int)s.E, d = (int)s.d, f = (int)s.f;
  MOE_TRY(launch_weight_quant(w_gate, E, d, f, F(c.ag), F(c.sg), Q(c.qg), stream));
  MOE_TRY(launch_weight_quant(w_up, E, d, f, F(c.au), F(c.su), Q(c.qu), stream));
  MOE_TRY(launch_weight_quant(w_down, E, f, d, F(c.ad), F(c.sd), Q(c.qd), stream));
  if (s.fp8 != 2) return MOE_OK;
  MOE_TRY(launch_quant_rows(w_gate, w_up, f, f, nullptr, E, (int64_t)E * d, Q(c.qgu_r), F(c.sgu_r), stream));
  return launch_quant_rows(w_down, nullptr, d, 0, nullptr, E, (int64_t)E * f, Q(c.qd_r), F(c.sd_r), stream);
}

int moe_workspace_size(const moe_shape* shape, size_t* fwd_ws, size_t* saved_bytes, size_t* bwd_ws) {
  MOE_TRY(check_shape(shape));
  const Plan p = plan(*shape);
  if (fwd_ws) *fwd_ws = p.fwd_total;
  if (saved_bytes) *saved_bytes = p.saved_total;
  if (bwd_ws) *bwd_ws = p.bwd_total;
  return MOE_OK;
}

int moe_route(const moe_shape* shape, const void* x, const float* w_r, const float* router_bias, int32_t* topk_idx,
              float* topk_w, float* s_sel, int32_t* expert_counts, void* ws, size_t ws_bytes, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  if (is_thr(s))
    return moe_set_error(MOE_ERR_UNSUPPORTED, "moe_route: the threshold router needs the layer entry points");
  if (s.T > 0) {
    MOE_NEED(x, "x");
    MOE_NEED(topk_idx, "topk_idx");
    MOE_NEED(topk_w, "topk_w");
  }
  MOE_NEED(w_r, "w_r");
  if (s.bias_mode != MOE_BIAS_NONE) MOE_NEED(router_bias, "router_bias");
  if (s.router == MOE_ROUTER_SIGMOID_GROUPED && s.T > 0) MOE_NEED(s_sel, "s_sel");
  MOE_TRY(check_ws(ws, ws_bytes, plan(s).fwd_total));
  return do_route(s, x, w_r, router_bias, topk_idx, topk_w, s_sel, expert_counts, ws, stream);
}

int moe_permute(const moe_shape* shape, const void* x, const int32_t* topk_idx, int32_t* expert_offsets,
                int32_t* row_of, int32_t* token_of, void* x_perm, void* ws, size_t ws_bytes, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  MOE_NEED(expert_offsets, "expert_offsets");
  if (s.T > 0) {
    MOE_NEED(x, "x");
    MOE_NEED(topk_idx, "topk_idx");
    MOE_NEED(row_of, "row_of");
    MOE_NEED(token_of, "token_of");
    MOE_NEED(x_perm, "x_perm");
  }
  MOE_TRY(check_ws(ws, ws_bytes, plan(s).fwd_total));
  return do_permute(s, x, topk_idx, expert_offsets, row_of, token_of, x_perm, ws, stream);
}

int moe_permute_noalloc(const moe_shape* shape, const void* x, const int32_t* topk_idx, int32_t* expert_offsets,
                        int32_t* row_of, int32_t* token_of, void* x_perm, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  MOE_NEED(expert_offsets, "expert_offsets");
  if (s.T > 0) {
    MOE_NEED(x, "x");
    MOE_NEED(topk_idx, "topk_idx");
    MOE_NEED(row_of, "row_of");
    MOE_NEED(token_of, "token_of");
    MOE_NEED(x_perm, "x_perm");
  }
  int32_t* hist = nullptr;
  MOE_TRY(permute_scratch((size_t)perm_blocks(s.T) * (size_t)epool(s) * sizeof(int32_t), &hist));
  PermArgs a{};
  a.x = x;
  a.topk_idx = topk_idx;
  a.T = s.T;
  a.d = (int)s.d;
  a.E = (int)epool(s);
  a.E_rows = (int)s.E;
  a.k = (int)s.k;
  a.bf16 = s.dtype == MOE_BF16;
  a.hist = hist;
  a.offsets = expert_offsets;
  a.row_of = row_of;
  a.token_of = token_of;
  a.x_perm = x_perm;
  return launch_permute(a, stream);
}

int moe_grouped_gemm_fwd(const moe_shape* shape, const void* x_perm, const int32_t* expert_offsets,
                         const void* w_gate, const void* w_up, const void* w_down, const void* b_gate,
                         const void* b_up, const void* b_down, void* gu, void* h, void* o, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  if (s.fp8)
    return moe_set_error(MOE_ERR_UNSUPPORTED, "moe_grouped_gemm_fwd: FP8 operands come from moe_layer_fwd");
  MOE_NEED(expert_offsets, "expert_offsets");
  MOE_NEED(w_gate, "w_gate");
  MOE_NEED(w_up, "w_up");
  MOE_NEED(w_down, "w_down");
  if (s.T > 0) {
    MOE_NEED(x_perm, "x_perm");
    MOE_NEED(gu, "gu");
    MOE_NEED(h, "h");
    MOE_NEED(o, "o");
  }
  if (s.expert_bias) {
    MOE_NEED(b_gate, "b_gate");
    MOE_NEED(b_up, "b_up");
    MOE_NEED(b_down, "b_down");
  } else {
    b_gate = b_up = b_down = nullptr;
  }
  return do_gemm_fwd(s, x_perm, expert_offsets, w_gate, w_up, w_down, b_gate, b_up, b_down, gu, h, o, stream);
}

int moe_grouped_gemm_bwd(const moe_shape* shape, int32_t passes, const void* x_perm, const int32_t* expert_offsets,
                         const void* gu, const void* h, const void* d_o, const void* w_gate, const void* w_up,
                         const void* w_down, void* dgu, void* dx_perm, void* dw_gate, void* dw_up, void* dw_down,
                         void* db_gate, void* db_up, void* db_down, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  if (passes <= 0 || passes > (MOE_DGRAD | MOE_WGRAD | MOE_ACCUMULATE) || !(passes & (MOE_DGRAD | MOE_WGRAD)))
    return moe_set_error(MOE_ERR_INVALID_ARG, "passes must be MOE_DGRAD, MOE_WGRAD or both (with MOE_ACCUMULATE)");
  if ((passes & MOE_ACCUMULATE) && !(passes & MOE_WGRAD))
    return moe_set_error(MOE_ERR_INVALID_ARG, "MOE_ACCUMULATE needs MOE_WGRAD");
  MOE_NEED(expert_offsets, "expert_offsets");
  if ((passes & MOE_DGRAD) && s.fp8 == 2)
    return moe_set_error(MOE_ERR_UNSUPPORTED, "moe_grouped_gemm_bwd: FP8 data-gradient operands come from moe_layer_bwd");
  if (passes & MOE_DGRAD) {
    MOE_NEED(w_gate, "w_gate");
    MOE_NEED(w_up, "w_up");
    MOE_NEED(w_down, "w_down");
    if (s.T > 0) {
      MOE_NEED(gu, "gu");
      MOE_NEED(d_o, "d_o");
      MOE_NEED(dgu, "dgu");
      MOE_NEED(dx_perm, "dx_perm");
    }
  }
  if (passes & MOE_WGRAD) {
    MOE_NEED(dw_gate, "dw_gate");
    MOE_NEED(dw_up, "dw_up");
    MOE_NEED(dw_down, "dw_down");
    if (s.T > 0) {
      MOE_NEED(x_perm, "x_perm");
      MOE_NEED(h, "h");
      MOE_NEED(d_o, "d_o");
      MOE_NEED(dgu, "dgu");
    }
    if (s.expert_bias) {
      MOE_NEED(db_gate, "db_gate");
      MOE_NEED(db_up, "db_up");
      MOE_NEED(db_down, "db_down");
    } else {
      db_gate = db_up = db_down = nullptr;
    }
  }
  return do_gemm_bwd(s, passes, x_perm, expert_offsets, gu, h, d_o, w_gate, w_up, w_down, dgu, dx_perm, dw_gate,
                     dw_up, dw_down, db_gate, db_up, db_down, stream);
}

int moe_combine_fwd(const moe_shape* shape, const void* o, const float* topk_w, const int32_t* row_of,
                    const void* shared_o, void* y, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  if (has_zc(s))
    return moe_set_error(MOE_ERR_UNSUPPORTED, "moe_combine_fwd: zero-computation experts need the layer entry points");
  if (s.T > 0) {
    MOE_NEED(o, "o");
    MOE_NEED(topk_w, "topk_w");
    MOE_NEED(row_of, "row_of");
    MOE_NEED(y, "y");
  }
  CombineFwdArgs a{o, topk_w, row_of, shared_o, y, s.T, (int)s.d, (int)s.k, s.dtype == MOE_BF16, nullptr, ZcArgs{}};
  return launch_combine_fwd(a, stream);
}

int moe_combine_bwd(const moe_shape* shape, const void* dy, const void* o, const float* topk_w,
                    const int32_t* row_of, void* d_o, float* d_topk_w, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  if (has_zc(s))
    return moe_set_error(MOE_ERR_UNSUPPORTED, "moe_combine_bwd: zero-computation experts need the layer entry points");
  if (s.T > 0) {
    MOE_NEED(dy, "dy");
    MOE_NEED(o, "o");
    MOE_NEED(topk_w, "topk_w");
    MOE_NEED(row_of, "row_of");
    MOE_NEED(d_o, "d_o");
    MOE_NEED(d_topk_w, "d_topk_w");
  }
  CombineBwdArgs a{};
  a.dy = dy;
  a.o = o;
  a.topk_w = topk_w;
  a.row_of = row_of;
  a.d_o = d_o;
  a.d_topk_w = d_topk_w;
  a.T = s.T;
  a.d = (int)s.d;
  a.k = (int)s.k;
  a.bf16 = s.dtype == MOE_BF16;
  a.router = s.router;
  a.route_scale = s.route_scale;
  return launch_combine_bwd(a, stream);
}

int moe_route_bwd(const moe_shape* shape, const void* x, const float* w_r, const int32_t* topk_idx,
                  const float* topk_w, const float* s_sel, const float* d_topk_w, const int32_t* expert_offsets,
                  const int32_t* token_of, float* dw_r, float* dx_router, void* ws, size_t ws_bytes,
                  hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  MOE_NEED(w_r, "w_r");
  MOE_NEED(dw_r, "dw_r");
  MOE_NEED(expert_offsets, "expert_offsets");
  if (s.T > 0) {
    MOE_NEED(x, "x");
    MOE_NEED(topk_idx, "topk_idx");
    MOE_NEED(topk_w, "topk_w");
    MOE_NEED(d_topk_w, "d_topk_w");
    MOE_NEED(token_of, "token_of");
    if (is_sigm(s)) MOE_NEED(s_sel, "s_sel");
  }
  const Plan p = plan(s);
  MOE_TRY(check_ws(ws, ws_bytes, p.bwd_total));
  RouteBwdArgs a = route_bwd_base(s);
  a.x = x;
  a.w_r = w_r;
  a.topk_idx = topk_idx;
  a.topk_w = topk_w;
  a.s_sel = s_sel;
  a.d_topk_w = d_topk_w;
  a.offsets = expert_offsets;
  a.token_of = token_of;
  a.dw_r = dw_r;
  a.dx_router = dx_router;
  a.dl = reinterpret_cast<float*>(wsp(ws, p.dl));
  a.partial = reinterpret_cast<float*>(wsp(ws, p.partial));
  a.w_rt = reinterpret_cast<float*>(wsp(ws, p.w_rt));
  return launch_route_bwd(a, stream);
}

int moe_unpermute_bwd(const moe_shape* shape, const void* dx_perm, const int32_t* row_of, const float* dx_router,
                      const void* dx_shared, void* dx, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  if (has_zc(s))
    return moe_set_error(MOE_ERR_UNSUPPORTED, "moe_unpermute_bwd: zero-computation experts need the layer entry points");
  if (s.T > 0) {
    MOE_NEED(dx_perm, "dx_perm");
    MOE_NEED(row_of, "row_of");
    MOE_NEED(dx, "dx");
  }
  UnpermuteArgs a{};
  a.dx_perm = dx_perm;
  a.row_of = row_of;
  a.dx_router = dx_router;
  a.dx_shared = dx_shared;
  a.dx = dx;
  a.T = s.T;
  a.d = (int)s.d;
  a.k = (int)s.k;
  a.bf16 = s.dtype == MOE_BF16;
  return launch_unpermute(a, stream);
}

int moe_shared_expert_fwd(const moe_shape* shape, const void* x, const void* ws_gate, const void* ws_up,
                          const void* ws_down, void* gu_sh, void* h_sh, void* o_sh, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  if (!s.n_shared) return moe_set_error(MOE_ERR_INVALID_ARG, "shape has no shared expert");
  MOE_NEED(ws_gate, "ws_gate");
  MOE_NEED(ws_up, "ws_up");
  MOE_NEED(ws_down, "ws_down");
  if (s.T > 0) {
    MOE_NEED(x, "x");
    MOE_NEED(gu_sh, "gu_sh");
    MOE_NEED(h_sh, "h_sh");
    MOE_NEED(o_sh, "o_sh");
  }
  return do_shared_fwd(s, x, ws_gate, ws_up, ws_down, gu_sh, h_sh, o_sh, stream);
}

int moe_shared_expert_bwd(const moe_shape* shape, const void* x, const void* dy, const void* gu_sh,
                          const void* h_sh, const void* ws_gate, const void* ws_up, const void* ws_down,
                          void* dx_shared, void* dws_gate, void* dws_up, void* dws_down, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  if (!s.n_shared) return moe_set_error(MOE_ERR_INVALID_ARG, "shape has no shared expert");
  MOE_NEED(ws_gate, "ws_gate");
  MOE_NEED(ws_up, "ws_up");
  MOE_NEED(ws_down, "ws_down");
  MOE_NEED(dws_gate, "dws_gate");
  MOE_NEED(dws_up, "dws_up");
  MOE_NEED(dws_down, "dws_down");
  if (s.T > 0) {
    MOE_NEED(x, "x");
    MOE_NEED(dy, "dy");
    MOE_NEED(gu_sh, "gu_sh");
    MOE_NEED(h_sh, "h_sh");
    MOE_NEED(dx_shared, "dx_shared");
  }
  const Plan p = plan(s);
  MOE_TRY(check_ws(ws, ws_bytes, p.bwd_total));
  return do_shared_bwd(s, x, dy, gu_sh, h_sh, ws_gate, ws_up, ws_down, wsp(ws, p.dgu_sh), dx_shared, dws_gate,
                       dws_up, dws_down, stream);
}

int moe_layer_fwd(const moe_shape* shape, const moe_params* prm, const void* x, const moe_saved* sv, void* y,
                  void* ws, size_t ws_bytes, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  MOE_NEED(prm, "params");
  MOE_NEED(sv, "saved");
  MOE_NEED(prm->w_r, "params.w_r");
  MOE_NEED(prm->w_gate, "params.w_gate");
  MOE_NEED(prm->w_up, "params.w_up");
  MOE_NEED(prm->w_down, "params.w_down");
  MOE_NEED(sv->expert_offsets, "saved.expert_offsets");
  if (s.bias_mode != MOE_BIAS_NONE) MOE_NEED(prm->router_bias, "params.router_bias");
  if (s.expert_bias) {
    MOE_NEED(prm->b_gate, "params.b_gate");
    MOE_NEED(prm->b_up, "params.b_up");
    MOE_NEED(prm->b_down, "params.b_down");
  }
  if (s.n_shared) {
    MOE_NEED(prm->ws_gate, "params.ws_gate");
    MOE_NEED(prm->ws_up, "params.ws_up");
    MOE_NEED(prm->ws_down, "params.ws_down");
  }
  if (s.T > 0) {
    MOE_NEED(x, "x");
    MOE_NEED(y, "y");
    MOE_NEED(sv->topk_idx, "saved.topk_idx");
    MOE_NEED(sv->topk_w, "saved.topk_w");
    MOE_NEED(sv->row_of, "saved.row_of");
    MOE_NEED(sv->token_of, "saved.token_of");
    MOE_NEED(sv->x_perm, "saved.x_perm");
    MOE_NEED(sv->gu, "saved.gu");
    MOE_NEED(sv->h, "saved.h");
    MOE_NEED(sv->o, "saved.o");
    if (is_sigm(s)) MOE_NEED(sv->s_sel, "saved.s_sel");
    if (s.n_shared) {
      MOE_NEED(sv->gu_sh, "saved.gu_sh");
      MOE_NEED(sv->h_sh, "saved.h_sh");
      MOE_NEED(sv->o_sh, "saved.o_sh");
    }
  }
  if (has_aux(s)) {
    MOE_NEED(sv->aux_loss, "saved.aux_loss");
    if (s.T > 0) MOE_NEED(sv->router_probs, "saved.router_probs");
  }
  if (s.n_const > 0) {
    MOE_NEED(prm->zc_v, "params.zc_v");
    MOE_NEED(prm->zc_wc, "params.zc_wc");
  }
  if (is_thr(s)) MOE_NEED(prm->gate_threshold, "params.gate_threshold");
  if (s.fp8) {
    MOE_NEED(prm->fp8_cache, "params.fp8_cache");
    MOE_TRY(check_fp8_cache(s, prm));
  }
  MOE_TRY(check_ws(ws, ws_bytes, plan(s).fwd_total));
  const void* bg = s.expert_bias ? prm->b_gate : nullptr;
  const void* bu = s.expert_bias ? prm->b_up : nullptr;
  const void* bd = s.expert_bias ? prm->b_down : nullptr;
  bool maps = false;
  MOE_TRY(do_route(s, x, prm->w_r, prm->router_bias, sv->topk_idx, sv->topk_w, sv->s_sel, nullptr, ws, stream,
                   has_aux(s) ? sv->router_probs : nullptr, prm->gate_threshold, sv->expert_offsets, sv->row_of,
                   &maps));
  MOE_TRY(do_permute(s, x, sv->topk_idx, sv->expert_offsets, sv->row_of, sv->token_of, sv->x_perm, ws, stream,
                     s.fp8 != 0, maps));
  if (has_aux(s)) {
    AuxArgs aa = aux_args(s, prm, sv);
    aa.part = reinterpret_cast<double*>(wsp(ws, plan(s).aux_part));
    MOE_TRY(launch_aux_stats(aa, stream));
  }
  if (s.fp8)
    MOE_TRY(do_gemm_fwd_fp8(s, sv->expert_offsets, prm->fp8_cache, bg, bu, bd, sv->gu, sv->h, sv->o, ws, stream));
  else
    MOE_TRY(do_gemm_fwd(s, sv->x_perm, sv->expert_offsets, prm->w_gate, prm->w_up, prm->w_down, bg, bu, bd, sv->gu,
                        sv->h, sv->o, stream));
  if (s.n_shared)
    MOE_TRY(do_shared_fwd(s, x, prm->ws_gate, prm->ws_up, prm->ws_down, sv->gu_sh, sv->h_sh, sv->o_sh, stream));
  CombineFwdArgs c{sv->o, sv->topk_w, sv->row_of, s.n_shared ? sv->o_sh : nullptr, y, s.T, (int)s.d, (int)s.k,
                   s.dtype == MOE_BF16, sv->topk_idx, zc_args(s, prm, x, nullptr, nullptr)};
  return launch_combine_fwd(c, stream);
}

int moe_layer_bwd(const moe_shape* shape, const moe_params* prm, const void* x, const moe_saved* sv, const void* dy,
                  void* dx, const moe_grads* gr, void* ws, size_t ws_bytes, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  MOE_TRY(check_layer_bwd(s, prm, x, sv, dy, dx, gr, 3));
  const Plan p = plan(s);
  MOE_TRY(check_ws(ws, ws_bytes, p.bwd_total));
  MOE_TRY(layer_bwd_dgrad(s, prm, x, sv, dy, dx, p, ws, stream));
  return layer_bwd_wgrad(s, prm, x, sv, dy, gr, false, p, ws, stream);
}

int moe_layer_bwd_dgrad(const moe_shape* shape, const moe_params* prm, const void* x, const moe_saved* sv,
                        const void* dy, void* dx, void* ws, size_t ws_bytes, hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  MOE_TRY(check_layer_bwd(s, prm, x, sv, dy, dx, nullptr, 1));
  const Plan p = plan(s);
  MOE_TRY(check_ws(ws, ws_bytes, p.bwd_total));
  return layer_bwd_dgrad(s, prm, x, sv, dy, dx, p, ws, stream);
}

int moe_layer_bwd_wgrad(const moe_shape* shape, const moe_params* prm, const void* x, const moe_saved* sv,
                        const void* dy, const moe_grads* gr, int32_t accumulate, void* ws, size_t ws_bytes,
                        hipStream_t stream) {
  MOE_TRY(check_shape(shape));
  const moe_shape& s = *shape;
  if (accumulate != 0 && accumulate != 1) return moe_set_error(MOE_ERR_INVALID_ARG, "accumulate must be 0 or 1");
  MOE_TRY(check_layer_bwd(s, prm, x, sv, dy, nullptr, gr, 2));
  const Plan p = plan(s);
  MOE_TRY(check_ws(ws, ws_bytes, p.bwd_total));
  return layer_bwd_wgrad(s, prm, x, sv, dy, gr, accumulate != 0, p, ws, stream);
}

}  // extern "C"
