/*
 * moe.h -- C ABI of libmoe: one Mixture-of-Experts layer, forward and
 * backward, on one AMD Instinct MI355X (gfx950).
 *
 * The layer is the one the PithTrain paper (arxiv 2605.31463) trains:
 * a router that picks the top-k experts of every token (section 3.2 and
 * appendix B.3 name the framework's top-k routing kernel), a scatter of the
 * tokens into expert-contiguous rows (section 3.2, its fused token scatter),
 * SwiGLU experts with fused forward and backward activation (section 3.2),
 * a gating-weighted combine, and the backward split into data-gradient and
 * weight-gradient passes so that the weight gradients can be delayed
 * (section 3.2, weight-gradient delay).  Routing outputs obey the paper's
 * routing-trace rules (appendix B.2.2): expert ids in [0, E), gating
 * weights non-negative and summing to one over the top-k (route_scale for
 * the DeepSeek-style router).
 *
 * Conventions shared by every entry point
 *   - Every tensor pointer is a DEVICE pointer owned by the caller; the
 *     compute entry points never allocate, free or synchronise.  Every call
 *     only enqueues work on `stream` and returns; results are ready when the
 *     stream reaches that point.  Pointers must be 16-byte aligned.  (The
 *     kernel-timing facility at the end, for benchmarks, is the exception:
 *     it creates HIP events on first use and moe_timing_read waits for them.)
 *   - Layouts are dense row-major.  T tokens, d hidden, E routed (FFN)
 *     experts, k experts per token, f expert width, R = T*k routed rows,
 *     E_pool = E + n_zero + n_copy + n_const experts the router chooses from
 *     (= E without zero-computation experts).
 *       x, y, dy, dx            [T][d]        activation dtype
 *       w_r, dw_r               [d][E_pool]   float32
 *       router_bias             [E_pool]      float32
 *       w_gate, w_up            [E][d][f]     activation dtype
 *       w_down                  [E][f][d]     activation dtype
 *       b_gate, b_up            [E][f];  b_down [E][d]
 *       topk_idx, row_of        [T][k]        int32
 *       topk_w, s_sel, d_topk_w [T][k]        float32
 *       expert_offsets          [E_pool+1]    int32 (exclusive scan of counts)
 *       token_of                [R]           int32 (= t*k + slot)
 *       x_perm, o, d_o, dx_perm [R][d]        activation dtype
 *       gu, dgu                 [R][2f]       columns [0,f) gate, [f,2f) up
 *       h                       [R][f]
 *     The activation dtype is moe_shape.dtype: MOE_F32 or MOE_BF16.  With
 *     MOE_BF16, products accumulate in float32 and every stored value is
 *     rounded to nearest-even.
 *   - Slot order: topk_idx[t][0..k-1] lists the chosen experts by
 *     descending selection key, equal keys to the lower expert index.
 *     Rows of expert e are expert_offsets[e] .. expert_offsets[e+1]-1, in
 *     ascending token order; row_of[t][s] is the row of (t, s).  Every slot
 *     has a row; the rows of zero-computation experts (ids >= E, after the
 *     FFN experts' rows) only list their tokens: x_perm, gu, h, o, d_o and
 *     dx_perm hold nothing there.
 *   - Results are bitwise reproducible run to run: no floating-point atomics.
 *   - Gradients overwrite their outputs, unless accumulation is asked for
 *     (MOE_ACCUMULATE in moe_grouped_gemm_bwd, accumulate = 1 in
 *     moe_layer_bwd_wgrad): then they are added to the buffers' contents.
 *   - Return value: MOE_OK or a negative MOE_ERR_* code.  Argument checks run
 *     on the host before anything is enqueued; on error nothing is enqueued
 *     and moe_last_error() gives a message (thread-local).
 *   - T = 0 is valid: token outputs are empty, counts/offsets and gradients
 *     are written as zeros.
 *
 * Limits (MOE_ERR_UNSUPPORTED beyond them): 1 <= E <= E_pool <= 256,
 * 1 <= k <= 16, d and f multiples of 64, d <= 16384, renorm = 1, and every
 * operand the GEMMs and the router stage through 32-bit buffer descriptors
 * below 4 GiB: R * max(d, 2f), T * max(d, 2 f_shared), d * 2f and, with the
 * auxiliary loss, T * E_pool elements of the activation dtype.
 *
 * Zero-computation experts (MoE++; appendix B.3 of the paper lists it among
 * the new-feature tasks: zero, copy and constant experts in the pool, the
 * router widened over them, the balance loss treating them explicitly).
 * Pool ids E .. E+n_zero-1 are zero experts (output 0), the next n_copy copy
 * experts (output x_t), the next n_const constant experts (output
 * a0 x_t + a1 v_c, (a0, a1) = softmax(W_c x_t), parameters zc_v [n_const][d]
 * and zc_wc [n_const][2][d], float32).  A slot that picks one adds
 * w * output to y_t and runs no GEMM.  Only the softmax routers support them,
 * and only through the layer entry points (moe_combine_fwd, moe_combine_bwd
 * and moe_unpermute_bwd refuse such shapes with MOE_ERR_UNSUPPORTED; route,
 * permute, grouped GEMMs and route backward work on the pool as documented).
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = -1, /* null pointer, non-positive size, k > E, bad groups */
  MOE_ERR_UNSUPPORTED = -2, /* valid but outside the limits above */
  MOE_ERR_HIP = -3,         /* a kernel launch failed (hipGetLastError) */
  MOE_ERR_WORKSPACE = -4    /* workspace pointer null or ws_bytes too small */
};

/* Router families.
 * SOFTMAX_TOPK: softmax over all E logits, keep the k largest, renormalise
 *   over the k (the Qwen3-30B-A3B router); equal to a softmax over the k
 *   selected logits.
 * TOPK_SOFTMAX: keep the k largest logits, softmax over those (GPT-OSS).
 * SIGMOID_GROUPED: s = sigmoid(logit); selection key s + router_bias; the E
 *   experts form n_groups contiguous groups, a group scores the sum of its two
 *   largest keys, the topk_groups best groups are kept and the top-k keys
 *   among their experts selected; weight = route_scale * s / sum of the
 *   selected s (DeepSeek-V3).
 * SIGMOID_THRESHOLD: the DynMoE task of the paper's appendix B.3 (per-expert
 *   sigmoid gates and a learned threshold, so the number of active experts
 *   varies per token).  Expert e is active for token t when
 *   logit - gate_threshold[e] > 0; the active experts fill the slots in
 *   descending order of that key, at most k of them (k is the slot capacity)
 *   and at least one (the best key, even when none passes); weights
 *   route_scale * s / sum of the active s, s = sigmoid(logit).  Empty slots
 *   hold topk_idx = -1, topk_w = s_sel = 0.  The thresholds get a gradient
 *   through a straight-through estimator of the activation indicator on the
 *   active experts: dL/dtheta_e = -sum over the slots holding e of
 *   s (route_scale omega - sum_j w_j omega_j) / sum of the active s.
 *   Needs n_groups = 1, bias_mode = NONE and no zero-computation experts;
 *   runs through the layer entry points (moe_route refuses it). */
enum {
  MOE_ROUTER_SOFTMAX_TOPK = 0,
  MOE_ROUTER_TOPK_SOFTMAX = 1,
  MOE_ROUTER_SIGMOID_GROUPED = 2,
  MOE_ROUTER_SIGMOID_THRESHOLD = 3
};

/* Router bias: none; added to the selection key only; added to the logits
 * (selection and weights).  The bias never receives a gradient. */
enum { MOE_BIAS_NONE = 0, MOE_BIAS_SELECT_ONLY = 1, MOE_BIAS_LOGIT = 2 };

enum { MOE_F32 = 0, MOE_BF16 = 1 };

/* Activation of the routed experts.  SWIGLU: h = silu(g) * u.  CLAMPED_GLU:
 * the GPT-OSS release's variant, gc = min(g, act_limit),
 * uc = clamp(u, -act_limit, act_limit), h = gc * sigmoid(act_alpha * gc) * (uc + 1)
 * (that release uses act_alpha = 1.702, act_limit = 7); in the backward a
 * clamp passes the gradient where the forward's value lies inside it, bounds
 * included.  The backward reads g and u from the saved gu, so with bf16
 * storage a value that rounding would carry across a clamp bound is stored
 * one bf16 step back on its own side: the clamp decisions taken on the
 * stored values are then the forward's.
 * The shared expert always uses SwiGLU. */
enum { MOE_ACT_SWIGLU = 0, MOE_ACT_CLAMPED_GLU = 1 };

/* passes of moe_grouped_gemm_bwd (bit mask).  MOE_ACCUMULATE (with
 * MOE_WGRAD): add the weight and bias gradients to what the output buffers
 * hold instead of overwriting them (bf16 gradients: the sum is taken in
 * float32 and rounded once more to bf16). */
enum { MOE_DGRAD = 1, MOE_WGRAD = 2, MOE_ACCUMULATE = 4 };

typedef struct moe_shape {
  int64_t T, d, E, k, f;       /* tokens, hidden, routed experts, top-k, expert width */
  int32_t n_groups;            /* expert groups for SIGMOID_GROUPED (1 = none) */
  int32_t topk_groups;         /* groups kept (= n_groups when not grouped) */
  int32_t n_shared;            /* 0 or 1 always-on shared expert of weight 1 */
  int64_t f_shared;            /* its width */
  int32_t router;              /* MOE_ROUTER_* */
  int32_t renorm;              /* must be 1: weights renormalised over the top-k */
  float route_scale;           /* factor on the renormalised weights (1, or 2.5) */
  int32_t bias_mode;           /* MOE_BIAS_* */
  int32_t expert_bias;         /* 1: experts carry b_gate, b_up, b_down */
  int32_t dtype;               /* MOE_F32 or MOE_BF16 activation / expert dtype */
  float aux_coef;              /* > 0: the layer entry points add the global-level
                                  load-balancing loss of this coefficient (softmax
                                  routers); 0: none */
  int32_t n_zero;              /* zero-computation experts in the pool: zero, */
  int32_t n_copy;              /*   copy */
  int32_t n_const;             /*   and constant experts (all 0: none) */
  float zc_aux_weight;         /* weight of a zero-computation expert's term in
                                  the load-balancing loss (FFN experts: 1; 0
                                  drops their terms); must be finite, >= 0 */
  int32_t act;                 /* MOE_ACT_* of the routed experts */
  float act_alpha;             /* CLAMPED_GLU: slope inside the sigmoid (> 0) */
  float act_limit;             /* CLAMPED_GLU: clamp bound (> 0) */
  int32_t fp8;                 /* routed experts' GEMMs on FP8 operands (see the
                                  FP8 section below): 0 none (bf16), 1 the
                                  forward ones, 2 the forward and the
                                  data-gradient ones */
} moe_shape;

/* Parameters of the layer (device pointers; unused ones may be NULL). */
typedef struct moe_params {
  const float* w_r;            /* [d][E_pool] */
  const float* router_bias;    /* [E_pool], bias_mode != NONE */
  const void* w_gate;          /* [E][d][f] */
  const void* w_up;            /* [E][d][f] */
  const void* w_down;          /* [E][f][d] */
  const void* b_gate;          /* [E][f], expert_bias */
  const void* b_up;            /* [E][f], expert_bias */
  const void* b_down;          /* [E][d], expert_bias */
  const void* ws_gate;         /* [d][f_shared], n_shared */
  const void* ws_up;           /* [d][f_shared], n_shared */
  const void* ws_down;         /* [f_shared][d], n_shared */
  const float* aux_f;          /* [E_pool] expert load fractions of the whole batch for
                                  the auxiliary loss (may be NULL: this call's
                                  routed-slot fractions counts / (T k)) */
  const float* zc_v;           /* [n_const][d] constant experts' vectors */
  const float* zc_wc;          /* [n_const][2][d] constant experts' mixing weights */
  const float* gate_threshold; /* [E] thresholds of MOE_ROUTER_SIGMOID_THRESHOLD */
  const void* fp8_cache;       /* shape->fp8 != 0: the weight cache moe_fp8_cache_build wrote */
  size_t fp8_cache_bytes;      /* its size; the layer entry points refuse a cache smaller
                                  than moe_fp8_cache_size gives for their shape
                                  (MOE_ERR_WORKSPACE) */
} moe_params;

/* Tensors the forward writes and the backward reads (caller-allocated). */
typedef struct moe_saved {
  int32_t* topk_idx;           /* [T][k] */
  float* topk_w;               /* [T][k] */
  float* s_sel;                /* [T][k], the sigmoid routers only (else may be NULL) */
  int32_t* expert_offsets;     /* [E_pool+1] */
  int32_t* row_of;             /* [T][k] */
  int32_t* token_of;           /* [R] */
  void* x_perm;                /* [R][d] */
  void* gu;                    /* [R][2f] */
  void* h;                     /* [R][f] */
  void* o;                     /* [R][d] */
  void* gu_sh;                 /* [T][2 f_shared], n_shared */
  void* h_sh;                  /* [T][f_shared], n_shared */
  void* o_sh;                  /* [T][d], n_shared */
  float* router_probs;         /* [T][E_pool] softmax over all experts, aux_coef > 0
                                  (threshold router: the sigmoid scores of all experts) */
  float* aux_loss;             /* [1] the auxiliary loss value, aux_coef > 0 */
} moe_saved;

/* Gradients of the parameters (overwritten). */
typedef struct moe_grads {
  float* dw_r;                 /* [d][E_pool] float32 */
  void* dw_gate;               /* [E][d][f] */
  void* dw_up;                 /* [E][d][f] */
  void* dw_down;               /* [E][f][d] */
  void* db_gate;               /* [E][f], expert_bias */
  void* db_up;                 /* [E][f], expert_bias */
  void* db_down;               /* [E][d], expert_bias */
  void* dws_gate;              /* [d][f_shared], n_shared */
  void* dws_up;                /* [d][f_shared], n_shared */
  void* dws_down;              /* [f_shared][d], n_shared */
  float* dzc_v;                /* [n_const][d], n_const > 0 */
  float* dzc_wc;               /* [n_const][2][d], n_const > 0 */
  float* d_threshold;          /* [E], MOE_ROUTER_SIGMOID_THRESHOLD */
} moe_grads;

/* Workspace bytes of the layer's scratch (section 3.2: the fused routing,
 * token-scatter and SwiGLU kernels and the wgrad-delay split between them).
 * fwd_ws: enough for moe_route, moe_permute and moe_layer_fwd (per-block
 * expert histograms, per-16-token expert counts, an arrival counter, the
 * router's split weights and float64 logits, FP8 rows);
 * bwd_ws: enough for moe_route_bwd, moe_grouped_gemm_bwd,
 * moe_shared_expert_bwd and moe_layer_bwd (which keeps d_o, dgu, dx_perm
 * and the router gradient scratch there, for the wgrad half); saved_bytes:
 * total size of the moe_saved tensors, for information.  Pure host
 * arithmetic; MOE_ERR_INVALID_ARG / MOE_ERR_UNSUPPORTED for a shape outside
 * the limits. */
int moe_workspace_size(const moe_shape* shape, size_t* fwd_ws, size_t* saved_bytes, size_t* bwd_ws);

/* Router forward: logits x W_r (+ bias), selection, weights, expert counts.
 * bf16 layers split W_r into three bf16 parts (a launch that also clears the
 * counts) and, with E_pool a multiple of 32, compute the logits as a tiled
 * MFMA product into the float64 logits of the workspace, then select in a
 * second kernel; other bf16 pools run one fused logits-and-selection kernel,
 * fp32 layers one kernel.
 * Logits are accumulated with float32 partial sums of 16 products folded
 * into a float64 total, and selection compares float64 keys.
 * out: topk_idx, topk_w [T][k]; s_sel [T][k] (SIGMOID_GROUPED, else may be
 * NULL); expert_counts [E_pool] int32 (may be NULL).  ws: fwd_ws bytes. */
int moe_route(const moe_shape* shape, const void* x, const float* w_r, const float* router_bias,
              int32_t* topk_idx, float* topk_w, float* s_sel, int32_t* expert_counts,
              void* ws, size_t ws_bytes, hipStream_t stream);

/* Token-to-expert permutation (section 3.2, EP token scatter, on one GPU):
 * per-block expert histogram, exclusive scan, then an atomic-free stable
 * scatter of x rows into expert-contiguous rows.
 * out: expert_offsets [E+1], row_of [T][k], token_of [R], x_perm [R][d].
 * Every topk_idx entry must lie in [0, E) and a token must not repeat an
 * expert (as moe_route produces); other values are undefined behaviour. */
int moe_permute(const moe_shape* shape, const void* x, const int32_t* topk_idx,
                int32_t* expert_offsets, int32_t* row_of, int32_t* token_of, void* x_perm,
                void* ws, size_t ws_bytes, hipStream_t stream);

/* moe_permute without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments and results as moe_permute (bitwise the
 * same outputs); its scratch, the per-block expert histograms of
 * ceil(T/256) * E_pool int32, lives in a fixed 4 MiB device array inside the
 * library (each GPU holds its own copy until the process ends), so it
 * allocates and frees nothing.  Shapes whose histograms exceed 4 MiB (for
 * instance T above 1M tokens with 256 experts) get MOE_ERR_UNSUPPORTED.
 * Every call on one GPU shares that array: calls that overlap on one GPU
 * (on different streams without ordering between them) race; calls ordered
 * on a stream are fine.  The first call on a device looks the array's
 * address up (MOE_ERR_HIP if that fails). */
int moe_permute_noalloc(const moe_shape* shape, const void* x, const int32_t* topk_idx,
                        int32_t* expert_offsets, int32_t* row_of, int32_t* token_of, void* x_perm,
                        hipStream_t stream);

/* Grouped SwiGLU expert forward (section 3.2, fused SwiGLU forward):
 *   [g|u] = x_perm_e [W_gate,e | W_up,e] (+ b_gate,e | b_up,e),
 *   h = silu(g) * u  (or the shape's MOE_ACT_*; from the float32 accumulators),
 *   o = h W_down,e (+ b_down,e),
 * for every expert e over its rows expert_offsets[e] .. expert_offsets[e+1]-1,
 * scheduled on the device from expert_offsets (no host synchronisation).
 * b_* may be NULL when shape->expert_bias is 0.  out: gu, h, o.
 * (bf16 operands: a shape with fp8 != 0 is refused; moe_layer_fwd runs it.) */
int moe_grouped_gemm_fwd(const moe_shape* shape, const void* x_perm, const int32_t* expert_offsets,
                         const void* w_gate, const void* w_up, const void* w_down,
                         const void* b_gate, const void* b_up, const void* b_down,
                         void* gu, void* h, void* o, hipStream_t stream);

/* Grouped expert backward, as one or both passes (section 3.2, wgrad delay):
 *  MOE_DGRAD: dh = d_o W_down^T with the fused SwiGLU backward
 *             dg = dh * u * sig(g) * (1 + g (1 - sig(g))), du = dh * silu(g)
 *             (or that of the shape's MOE_ACT_*; g, u read from gu) -> dgu;
 *             then dx_perm = [dg|du] [W_gate|W_up]^T.
 *  MOE_WGRAD: dW_down = h^T d_o, dW_gate = x_perm^T dg, dW_up = x_perm^T du
 *             per expert, and with expert_bias the column sums db_down, db_gate,
 *             db_up.  Reads dgu, so it runs after a DGRAD pass.  With
 *             MOE_ACCUMULATE the gradients are added to dw_* / db_*.
 * Pointers of a pass that is not requested may be NULL.  Errors:
 * MOE_ERR_INVALID_ARG for a passes value outside these bits or
 * MOE_ACCUMULATE without MOE_WGRAD; MOE_ERR_UNSUPPORTED for MOE_DGRAD with
 * shape->fp8 = 2 (moe_layer_bwd runs those passes).  With fp8 = 1 these are
 * the bf16 passes. */
int moe_grouped_gemm_bwd(const moe_shape* shape, int32_t passes,
                         const void* x_perm, const int32_t* expert_offsets,
                         const void* gu, const void* h, const void* d_o,
                         const void* w_gate, const void* w_up, const void* w_down,
                         void* dgu, void* dx_perm,
                         void* dw_gate, void* dw_up, void* dw_down,
                         void* db_gate, void* db_up, void* db_down, hipStream_t stream);

/* Weighted combine, the reverse of the token scatter (section 3.2; the
 * gating weights obey the routing-trace rules of appendix B.2.2): a gather
 * in fixed slot order with a float32 sum,
 *   y_t = sum_s topk_w[t][s] * o[row_of[t][s]]  (+ shared_o[t] if non-NULL).
 * One pass over the rows of o.  Out: y [T][d].  MOE_ERR_UNSUPPORTED with
 * zero-computation experts (the layer entry points run them). */
int moe_combine_fwd(const moe_shape* shape, const void* o, const float* topk_w,
                    const int32_t* row_of, const void* shared_o, void* y, hipStream_t stream);

/* Combine backward (the gradient of the weighted combine above; section
 * 3.2's fused backward kernels):
 *   d_o[row_of[t][s]] = topk_w[t][s] * dy_t,
 *   d_topk_w[t][s]    = <dy_t, o[row_of[t][s]]>  (float32),
 * one pass over dy and the rows of o.  Out: d_o [R][d], d_topk_w [T][k].
 * MOE_ERR_UNSUPPORTED with zero-computation experts. */
int moe_combine_bwd(const moe_shape* shape, const void* dy, const void* o, const float* topk_w,
                    const int32_t* row_of, void* d_o, float* d_topk_w, hipStream_t stream);

/* Router backward (the gradient of the top-k routing kernel of appendix
 * B.3 through the gating weights; weights as in the routing-trace rules of
 * appendix B.2.2).  dl on the selected experts only:
 *   softmax families: dl_j = w_j (omega_j - sum_i w_i omega_i / route_scale)
 *   SIGMOID_GROUPED, SIGMOID_THRESHOLD:
 *                     dl_j = (route_scale omega_j - sum_i w_i omega_i) / sum_i s_i
 *                            * s_j (1 - s_j)   (an empty slot has s = 0: dl = 0)
 * with omega = d_topk_w; then dw_r[:, e] = sum over the rows of expert e of
 * x[token] * dl (using expert_offsets and token_of from moe_permute, in row
 * order), and dx_router[t] = sum_s dl[t][s] * W_r[:, topk_idx[t][s]] over the
 * filled slots (float32, may be NULL to skip).  The thresholds' gradient
 * comes from the layer entry points only.  ws: bwd_ws bytes. */
int moe_route_bwd(const moe_shape* shape, const void* x, const float* w_r,
                  const int32_t* topk_idx, const float* topk_w, const float* s_sel,
                  const float* d_topk_w, const int32_t* expert_offsets, const int32_t* token_of,
                  float* dw_r, float* dx_router, void* ws, size_t ws_bytes, hipStream_t stream);

/* Unpermute-reduce, the backward of the token scatter (section 3.2): a
 * gather of each token's k rows in fixed slot order with a float32 sum,
 *   dx_t = sum_s dx_perm[row_of[t][s]]
 *          + dx_router[t] (float32, may be NULL) + dx_shared[t] (may be NULL).
 * Out: dx [T][d].  MOE_ERR_UNSUPPORTED with zero-computation experts. */
int moe_unpermute_bwd(const moe_shape* shape, const void* dx_perm, const int32_t* row_of,
                      const float* dx_router, const void* dx_shared, void* dx, hipStream_t stream);

/* Always-on shared expert (DeepSeek-V3 style, weight 1), forward:
 *   [g|u] = x [Ws_gate | Ws_up], h = silu(g) * u, o_sh = h Ws_down.
 * out: gu_sh [T][2 f_shared], h_sh [T][f_shared], o_sh [T][d]. */
int moe_shared_expert_fwd(const moe_shape* shape, const void* x,
                          const void* ws_gate, const void* ws_up, const void* ws_down,
                          void* gu_sh, void* h_sh, void* o_sh, hipStream_t stream);

/* Shared expert backward with upstream gradient dy (its weight is 1):
 * dWs_down = h_sh^T dy, SwiGLU backward into dgu_sh (kept in ws),
 * dWs_gate, dWs_up, and dx_shared = dgu_sh [Ws_gate|Ws_up]^T.
 * ws: bwd_ws bytes. */
int moe_shared_expert_bwd(const moe_shape* shape, const void* x, const void* dy,
                          const void* gu_sh, const void* h_sh,
                          const void* ws_gate, const void* ws_up, const void* ws_down,
                          void* dx_shared, void* dws_gate, void* dws_up, void* dws_down,
                          void* ws, size_t ws_bytes, hipStream_t stream);

/* Whole layer forward: route, permute, grouped SwiGLU experts, shared expert,
 * combine.  Fills every pointer of *saved (s_sel only for the sigmoid routers,
 * the *_sh tensors only with a shared expert) and y.  ws: fwd_ws bytes.
 * (On the two-kernel bf16 route path the selection also builds the
 * permutation's block counts, expert offsets and each slot's rank inside its
 * 16-token block, so the permutation runs only its copy, which finishes
 * row_of and token_of; the results are those of moe_route followed by
 * moe_permute, bitwise.) */
int moe_layer_fwd(const moe_shape* shape, const moe_params* params, const void* x,
                  const moe_saved* saved, void* y, void* ws, size_t ws_bytes, hipStream_t stream);

/* Whole layer backward of L = sum_t <dy_t, y_t>: combine backward, expert
 * dgrad and wgrad, router backward, shared expert backward, unpermute.
 * dx includes the expert, router and shared-expert paths (and the
 * zero-computation experts': copy slots w dy_t, constant slots
 * a0 w dy_t + W_c^T dz; their parameter gradients go to dzc_v, dzc_wc).
 * ws: bwd_ws bytes. */
int moe_layer_bwd(const moe_shape* shape, const moe_params* params, const void* x,
                  const moe_saved* saved, const void* dy, void* dx, const moe_grads* grads,
                  void* ws, size_t ws_bytes, hipStream_t stream);

/* The layer backward in two halves, for weight-gradient delay (section 3.2:
 * the input gradient is produced first, so that the previous layer's
 * backward can start; the weight gradients are computed later).
 * moe_layer_bwd equals moe_layer_bwd_dgrad followed by moe_layer_bwd_wgrad
 * with accumulate = 0, with bitwise equal results.
 *
 * moe_layer_bwd_dgrad: combine backward with the router's dl, expert dgrad
 *   (fused SwiGLU backward), shared-expert dgrad, unpermute -> dx (with the
 *   router and shared-expert paths).  Leaves d_o, dgu, dl (and the shared
 *   expert's dgu, the zero-computation slots' coefficients) in ws, which the
 *   caller must keep unchanged until the matching moe_layer_bwd_wgrad call.
 *   Pointers of *saved read: topk_idx, topk_w, s_sel (sigmoid routers),
 *   expert_offsets, row_of, gu, o, gu_sh.
 * moe_layer_bwd_wgrad: expert wgrads (+ biases), dW_r, shared-expert wgrads
 *   and the constant experts' dzc_v, dzc_wc into *grads, from what the dgrad
 *   half left in ws.  accumulate = 1 adds
 *   every gradient to the buffer's current value (gradient accumulation over
 *   micro-batches), 0 overwrites.  Pointers of *saved read: topk_idx,
 *   expert_offsets, token_of, x_perm, h, h_sh.
 * Both: ws of bwd_ws bytes (the same buffer for both halves); x and dy as for
 * moe_layer_bwd.  Errors as for moe_layer_bwd; accumulate outside {0, 1}
 * is MOE_ERR_INVALID_ARG. */
int moe_layer_bwd_dgrad(const moe_shape* shape, const moe_params* params, const void* x,
                        const moe_saved* saved, const void* dy, void* dx,
                        void* ws, size_t ws_bytes, hipStream_t stream);
int moe_layer_bwd_wgrad(const moe_shape* shape, const moe_params* params, const void* x,
                        const moe_saved* saved, const void* dy, const moe_grads* grads,
                        int32_t accumulate, void* ws, size_t ws_bytes, hipStream_t stream);

/* FP8 GEMMs of the routed experts (the paper's FP8 training: fused
 * quantisation, quantised weights cached across micro-batches; it states no
 * scaling recipe, so this one is the library's).  bf16 layers with d and f
 * multiples of 128.  A value v of a row (column) whose largest magnitude is
 * amax is stored as the OCP E4M3 value nearest to clamp(v * (448 / amax),
 * -448, 448) (float32 product, ties to even) with scale amax / 448 (1 for an
 * all-zero row); the GEMMs accumulate the code products in float32 and
 * multiply by the row and column scales.  gu, h, o, d_o and dgu stay bf16; the
 * shared expert and the weight-gradient GEMMs stay bf16.
 *
 * shape->fp8 = 1: moe_layer_fwd runs both forward expert GEMMs on E4M3
 * operands: the permutation also writes every routed row of x in E4M3 with
 * one scale per token, h is quantised per row after the gate/up GEMM, and the
 * weights (one scale per output column) come from the cache.  The backward is
 * the bf16 backward of those activations and of the bf16 weights
 * (quantisation taken as the identity).
 * shape->fp8 = 2: in addition, the backward's two data-gradient GEMMs
 * (dh = d_o W_down^T, dx_perm = [dg | du] [W_gate | W_up]^T) run on E4M3
 * operands: the stored d_o rows (quantised by the combine backward, or by a
 * pass of their own with zero-computation experts) and dgu rows (one scale
 * over a row's gate and up halves), and the weights quantised per row (an
 * output column of these products; one scale over a row of W_gate and W_up
 * together) from the cache.
 *
 * moe_fp8_cache_size: bytes of the cache for the shape (fp8 = 2 about twice
 * fp8 = 1).  moe_fp8_cache_build: quantises w_gate, w_up [E][d][f] and
 * w_down [E][f][d] (bf16) per output column into the caller's cache (codes
 * stored transposed, K-contiguous, with the scales) and, for fp8 = 2, per row
 * as well; call it again whenever the weights change, and reuse it for every
 * micro-batch in between.  The layer entry points read the cache as laid out
 * for their own shape: it must have been built for the same shape (E, d, f
 * and the fp8 level); a cache built for fp8 = 1 lacks the regions fp8 = 2
 * reads.  The standalone moe_grouped_gemm_fwd / _bwd refuse
 * FP8 passes (MOE_ERR_UNSUPPORTED): their operands are the layer's.  Errors:
 * MOE_ERR_UNSUPPORTED without shape->fp8, MOE_ERR_WORKSPACE for a cache below
 * the size. */
int moe_fp8_cache_size(const moe_shape* shape, size_t* bytes);
int moe_fp8_cache_build(const moe_shape* shape, const void* w_gate, const void* w_up, const void* w_down,
                        void* cache, size_t cache_bytes, hipStream_t stream);

/* Status code -> static string. */
const char* moe_status_string(int status);

/* Detail of the last failure on the calling thread ("" if none). */
const char* moe_last_error(void);

/* Kernel timing for benchmarks.  Kernels are numbered 0 .. moe_kernel_count()-1
 * and named by moe_kernel_name().  moe_timing_select(id) makes every later
 * launch of kernel id (in any entry point, on the calling thread) record a
 * pair of HIP events on its stream; id < 0 switches it off and drops the
 * records.  moe_timing_read() waits for the recorded events and returns the
 * summed milliseconds and the number of timed launches.  Up to 4096 launches
 * are kept.  Not for concurrent use from several threads. */
int moe_kernel_count(void);
const char* moe_kernel_name(int id);
int moe_timing_select(int id);
int moe_timing_read(double* total_ms, int* launches);

#ifdef __cplusplus
}
#endif

#endif /* MOE_H */
