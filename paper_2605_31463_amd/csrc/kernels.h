// Launchers of the libmoe kernels (host side).  Every launcher only enqueues
// on the given stream and returns a MOE_* status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

struct RouteArgs {
  const void* x;
  const float* w_r;
  const float* bias;
  int64_t T;
  int d, E, k;
  int router, bias_mode, n_groups, topk_groups;
  float route_scale;
  bool bf16;
  int32_t* topk_idx;
  float* topk_w;
  float* s_sel;
  int32_t* counts;  // may be null
  void* wsplit;      // bf16 [3][E][d] workspace for the MFMA path (bf16 x), or null
  double* lg;        // float64 [T][E] logits workspace for the MFMA path
  float* probs;      // [T][E] softmax over all experts (auxiliary loss), or null;
                     // the threshold router writes its sigmoid scores there
  const float* threshold;  // [E] thresholds of the threshold router
  // the permutation's maps inputs, built by the selection when these are set
  // and the path supports it (launch_route reports whether it did): per-block
  // expert counts turned into each block's base inside its expert
  // [perm_blocks(T)][E], expert_offsets [E+1], and one arrival counter
  int32_t* hist;
  int32_t* offsets;
  int32_t* sync;
  // and, for the permutation's copy to finish the maps: each 16-token
  // selection block's expert counts [ceil(T/16)][E] and, in row_of, each
  // slot's rank among the block's earlier tokens of its expert (-1: no expert)
  int32_t* cnt16;
  int32_t* row_of;
};
// maps_built (may be null): set to whether hist / offsets were produced
int launch_route(const RouteArgs& a, hipStream_t s, bool* maps_built = nullptr);
int zero_i32(int32_t* p, int64_t n, hipStream_t s);

// Permutation: histogram per block of PERM_TB tokens, scan, scatter.
constexpr int PERM_TB = 256;
__host__ __device__ inline int64_t perm_blocks(int64_t T) { return (T + PERM_TB - 1) / PERM_TB; }
struct PermArgs {
  const void* x;
  const int32_t* topk_idx;
  int64_t T;
  int d, E, k;       // E: experts ranked (the whole pool)
  int E_rows;        // the first E_rows experts' rows receive x (FFN experts)
  bool bf16;
  int32_t* hist;     // [nblk][E] workspace
  int32_t* offsets;  // [E+1]
  int32_t* row_of;   // [T][k]
  int32_t* token_of; // [R]
  void* x_perm;      // [R][d]
  uint8_t* xq;       // [R][d] E4M3 rows of the FFN experts (FP8 forward), or null
  float* sx;         // [R] their row scales
  bool maps_ready;   // the route built the maps' inputs: hist holds the block bases,
                     // offsets is written, row_of holds ranks inside 16-token blocks
                     // whose counts are in cnt16; the copy finishes row_of, token_of
  const int32_t* cnt16;
};
int launch_permute(const PermArgs& a, hipStream_t s);
// The allocation-free permutation's fixed scratch (per-block histograms):
// its size, and the current device's address of it (MOE_ERR_UNSUPPORTED when
// `need` bytes exceed it).
constexpr size_t kPermScratchBytes = (size_t)4 << 20;
constexpr int kMaxDevices = 64;
int permute_scratch(size_t need, int32_t** out);

// FP8: E4M3 rows of [s0 | s1] (bf16 [rows][w0] and [rows][w1], w1 may be 0;
// with offsets, only the rows below offsets[E]) and their scales.
int launch_quant_rows(const void* s0, const void* s1, int w0, int w1, const int32_t* offsets, int E, int64_t rows,
                      uint8_t* q, float* scale, hipStream_t s);
// FP8 weight cache of one expert weight W [E][K][N] (bf16): column maxima
// amax [E][N], scales [E][N] = amax / 448, codes Q [E][N][K] (transposed).
int launch_weight_quant(const void* w, int E, int K, int N, float* amax, float* scale, uint8_t* q, hipStream_t s);

// Zero-computation experts of the pool (MoE++): pool ids E_ffn .. are n_zero
// zero experts (out = 0), then n_copy copy experts (out = x), then n_const
// constant experts (out = a0 x + a1 v_c, (a0, a1) = softmax(W_c x)).
struct ZcArgs {
  bool on;                // false: no such experts (every slot is an FFN slot)
  int E_ffn, n_zero, n_copy, n_const;
  const void* x;          // [T][d] layer input, activation type
  const float* v;         // [n_const][d]
  const float* wc;        // [n_const][2][d]
  float4* coef;           // [T*k] per slot: (dz0, dz1, w a1, dy's factor in dx);
                          // written by the combine backward
  const void* dy;         // [T][d] (unpermute)
};

struct CombineFwdArgs {
  const void* o;
  const float* topk_w;
  const int32_t* row_of;
  const void* shared_o;
  void* y;
  int64_t T;
  int d, k;
  bool bf16;
  const int32_t* topk_idx;  // read with zero-computation experts
  ZcArgs zc;
};
int launch_combine_fwd(const CombineFwdArgs& a, hipStream_t s);

// Combine backward; with dl != null it also writes the router logit
// gradient of the selected experts (fused router backward, first step).
struct CombineBwdArgs {
  const void* dy;
  const void* o;
  const float* topk_w;
  const int32_t* row_of;
  void* d_o;
  float* d_topk_w;   // may be null
  int64_t T;
  int d, k;
  bool bf16;
  // fused dl
  float* dl;         // may be null
  const float* s_sel;
  int router;
  float route_scale;
  const int32_t* topk_idx;  // read with zero-computation experts
  ZcArgs zc;
  float* dth;        // threshold router: per slot -s (c omega - sum w omega) / sum s, or null
  // FP8 data gradients (bf16, without zero-computation experts): E4M3 rows of
  // d_o [R][d] and their scales [R], or null
  uint8_t* doq;
  float* sdo;
};
int launch_combine_bwd(const CombineBwdArgs& a, hipStream_t s);

struct RouteBwdArgs {
  const void* x;
  const float* w_r;
  const int32_t* topk_idx;
  const float* topk_w;
  const float* s_sel;
  const float* d_topk_w;   // omega; unused when dl_in is given
  const float* dl_in;      // precomputed dl [T][k] or null
  const int32_t* offsets;
  const int32_t* token_of;
  float* dw_r;
  float* dx_router;        // may be null
  int64_t T;
  int d, E, k;
  int router;
  float route_scale;
  bool bf16;
  // workspace
  float* dl;               // [T][k]
  float* partial;          // [route_dwr_tasks][d]
  float* w_rt;             // [E][d]
  bool accumulate;         // dw_r += the gradient (else dw_r = the gradient)
};
constexpr int DWR_ROWS = 256;  // rows per partial-sum task of dW_r
inline int64_t route_dwr_tasks(int64_t R, int64_t E) { return R / DWR_ROWS + E; }
int launch_route_bwd(const RouteBwdArgs& a, hipStream_t s);
int launch_wr_transpose(const float* w_r, float* w_rt, int d, int E, hipStream_t s);
// Threshold router: dtheta[e] (+)= sum over expert e's rows of g[token_of[row]]
// (g [T*k] per slot, from the combine backward).
int launch_threshold_grad(const int32_t* offsets, const int32_t* token_of, const float* g, int E, float* dtheta,
                          bool accumulate, hipStream_t s);
// W_r^T [Eo][d] in the activation type, rows E .. Eo-1 zero.
int launch_wr_transpose_act(const float* w_r, void* w_rt, int d, int E, int Eo, bool bf16, hipStream_t s);

// Global-level load-balancing loss: statistics and logit gradient.
struct AuxArgs {
  const float* probs;       // [T][E] softmax over all experts
  const int32_t* offsets;   // [E+1] expert_offsets (this call's loads)
  const float* aux_f;       // [E] given load fractions, or null
  int64_t T;
  int E, k;
  float coef;
  int E_ffn;                // experts E_ffn .. E-1 (zero-computation ones) weigh
  float zc_weight;          //   zc_weight in the loss, the others 1
  bool thr;                 // threshold router: probs hold sigmoid scores s, the loss
                            // uses p = s / sum s and fractions of the filled slots
  double* part;             // [aux_blocks(T)][E] workspace
  float* loss;              // [1]
};
inline int64_t aux_blocks(int64_t T) { return (T + 255) / 256; }
int launch_aux_stats(const AuxArgs& a, hipStream_t s);
// dl [T][E_pad] in the activation type (columns E .. E_pad-1 zero), and the
// row offsets [G+1] of the T tokens cut into chunks, for the grouped dW_r product
int launch_aux_grad(const AuxArgs& a, void* dl, int E_pad, int32_t* chunk_off, int G, int64_t chunk, bool bf16,
                    hipStream_t s);
// dw_r[i][e] += sum over the G chunks of part[g][i][e]
int launch_aux_dwr(const void* part, int G, int d, int E, int E_pad, bool bf16, float* dw_r, hipStream_t s);
// W_r^T in the activation type (bf16 rounding for bf16 layers)

struct UnpermuteArgs {
  const void* dx_perm;
  const int32_t* row_of;
  const float* dx_router;   // may be null
  const void* dx_shared;    // may be null
  const void* dx_aux;       // may be null: the auxiliary loss's router dx [T][d]
  // fused router dx: dx += sum_s dl[t][s] * w_rt[topk_idx[t][s]]
  const float* dl;          // may be null
  const int32_t* topk_idx;
  const void* w_rt;         // W_r^T [E][d] in the activation type
  void* dx;
  int64_t T;
  int d, k;
  bool bf16;
  ZcArgs zc;                // zero-computation slots: no dx_perm row, dx from coef
  int ns;                   // column slices (set by the launcher)
};
int launch_unpermute(const UnpermuteArgs& a, hipStream_t s);

// Gradients of the constant experts' parameters: over the rows of each
// constant expert (the permutation lists its tokens), in tasks of DWR_ROWS rows,
//   dW_c[c][j] = sum_rows dz_j x_token,  dv[c] = sum_rows (w a1) dy_token,
// per-task float32 partials summed in task order.
struct ZcParamArgs {
  const void* x;            // [T][d]
  const void* dy;           // [T][d]
  const float4* coef;       // [T*k] from the combine backward
  const int32_t* offsets;   // [E_pool+1]
  const int32_t* token_of;  // [T*k]
  int64_t T;
  int d, k;
  int e0, n_const;          // pool id of the first constant expert, their number
  bool bf16;
  float* partial;           // [route_dwr_tasks(T*k, n_const)][3][d] workspace
  float* dwc;               // [n_const][2][d]
  float* dv;                // [n_const][d]
  bool accumulate;
};
int launch_zc_param_grads(const ZcParamArgs& a, hipStream_t s);

// Grouped GEMMs.
enum GemmMode {
  G_FWD_GATEUP = 0,  // [g|u] = A W_gate|W_up (+b), h = silu(g) u      A=x_perm [rows][d]
  G_FWD_DOWN,        // o = h W_down (+b)                                A=h [rows][f]
  G_DGRAD_DOWN,      // dh = d_o W_down^T, dSwiGLU with gu -> dgu        A=d_o [rows][d]
  G_DGRAD_GATEUP,    // dx_perm = dgu [W_gate|W_up]^T                     A=dgu [rows][2f]
  G_WGRAD_DOWN,      // dW_down = h^T d_o, db_down                        K = rows
  G_WGRAD_GATEUP,    // dW_gate|dW_up = x_perm^T dgu, db_gate|db_up       K = rows
};
struct GemmArgs {
  int mode;
  bool bf16;
  const int32_t* offsets;  // [ngroups+1] device, or null for one group of dense_rows rows
  int ngroups;
  int64_t dense_rows;
  int64_t max_rows;        // upper bound of the total rows (for the grid)
  int d, f;
  // operands
  const void* a;           // row-major activations (x_perm, h, d_o, dgu)
  const void* b;           // second activation for wgrad (d_o, dgu)
  const void* w0;          // w_gate or w_down
  const void* w1;          // w_up
  const void* bias0;       // b_gate or b_down  (fwd)
  const void* bias1;       // b_up
  const void* aux;         // gu (dgrad down)
  // outputs
  void* c0;                // gu | o | dgu | dx_perm | dW_down | dW_gate
  void* c1;                // h  |   |     |         |         | dW_up
  void* db0;               // db_down | db_gate
  void* db1;               // db_up
  bool accumulate;         // wgrad passes: add into c0/c1/db0/db1 instead of overwriting
  int act;                 // MOE_ACT_*: activation of the gate/up forward and down dgrad epilogues
  float act_alpha, act_limit;
  // FP8 forward and data-gradient passes: a = E4M3 rows, w0 / w1 = the weight
  // cache's E4M3 codes (forward: [E][f][d] gate / up, [E][d][f] down; data
  // gradients: [E][f][d] down rows, [E][d][2f] [gate | up] rows), the float32
  // row and column scales
  bool fp8;
  const float* a_scale;    // [rows]
  const float* b_scale0;   // [E][N] column scales (gate, down, or [gate | up] rows)
  const float* b_scale1;   // [E][f] up column scales
  int kid;                 // timing id of the launch (0: the routed pass's own)
};
int launch_gemm(const GemmArgs& a, hipStream_t s);

}  // namespace moe
