// Grouped expert GEMMs: forward gate/up with the fused SwiGLU epilogue,
// forward down, the down data-gradient with the fused SwiGLU backward, the
// gate/up data-gradient, and both weight gradients (section 3.2: fused SwiGLU
// forward and backward kernels; wgrad kept as a separate pass so that it can
// be delayed).  The same kernels run the shared expert's dense passes.
//
// bf16 path (MFMA): one persistent kernel, gemm_bf16_persistent, with one
// workgroup per CU (two for the 128 x 128 tiles).  A workgroup of 8
// wavefronts computes 256 x 256 output tiles (2 x 4 or 4 x 2 wavefronts, each
// a 128 x 64 or 64 x 128 block of v_mfma_f32_32x32x16_bf16 32 x 32 products
// with float32 accumulators); experts with fewer than 192 rows on average use
// 128 x 128 tiles of 4 wavefronts.  K advances through 2 LDS stages of 64 k
// (4 of 32 k in the weight gradients) filled by buffer_load ... lds (global ->
// LDS without registers); the copies of the next stages are in flight while
// the current one is multiplied, also across tile boundaries.  Operands
// contiguous along K are read with ds_read_b128, operands contiguous along M
// or N (the weights in the forward, both operands of the weight gradients)
// with the transposing ds_read_b64_tr_b16, so no operand is ever transposed
// in registers or in HBM.
//
// Scheduling happens on the device from expert_offsets: every workgroup
// counts the row tiles of each expert (a block scan), the tiles are numbered
// expert by expert, each XCD owns a contiguous range of tile ids and its
// workgroups take them round-robin, so variable per-expert row counts need
// no host synchronisation.  Buffer descriptors bound each operand to its
// expert's rows, so rows past an expert's end (and, for the weight gradients,
// whose K is the expert's row count, k past the end) read as zero; outputs
// past M or N are not stored.  The epilogue is wavefront-local (each 32 x 32
// block staged through a private LDS slot, written as 64-byte row pieces).
//
// FP8: E4M3 instantiations of the forward and data-gradient passes
// (v_mfma_f32_32x32x64_f8f6f4, quantisation scales folded into the
// epilogues).  fp32 path: a plain kernel, one thread per output, for the
// fp32 workload; same modes, same epilogues.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace moe {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef int v4i32 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void* lds_void_t;
typedef __attribute__((address_space(3))) v4i16* lds_v4_t;


__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + __expf(-z)); }

// The experts' gated activation h = act(g, u) and its backward:
//   SwiGLU:      h = silu(g) u;
//   clamped GLU: gc = min(g, L), uc = clamp(u, -L, L), h = gc sig(alpha gc) (uc + 1)
//                (the GPT-OSS release's variant); the clamps pass the gradient
//                inside their bounds, bounds included.
// CL selects the clamped GLU at compile time (the bf16 epilogues are compiled
// for both and pick one per launch); the runtime forms below serve the others.
template <bool CL>
__device__ __forceinline__ float act_h_t(const GemmArgs& a, float g, float u) {
  if constexpr (CL) {
    const float L = a.act_limit;
    const float gc = fminf(g, L);
    const float uc = fminf(fmaxf(u, -L), L);
    return gc / (1.0f + __expf(-a.act_alpha * gc)) * (uc + 1.0f);
  } else {
    return silu_f(g) * u;
  }
}

// dg = dh * dact/dg, du = dh * dact/du at (g, u)
template <bool CL>
__device__ __forceinline__ void act_grad_t(const GemmArgs& a, float g, float u, float dh, float& dg, float& du) {
  if constexpr (CL) {
    const float L = a.act_limit, al = a.act_alpha;
    const float gc = fminf(g, L);
    const float uc = fminf(fmaxf(u, -L), L);
    const float s = 1.0f / (1.0f + __expf(-al * gc));
    dg = g <= L ? dh * (uc + 1.0f) * s * (1.0f + al * gc * (1.0f - s)) : 0.f;
    du = (u >= -L && u <= L) ? dh * gc * s : 0.f;
  } else {
    const float sgm = 1.0f / (1.0f + __expf(-g));
    dg = dh * u * sgm * (1.0f + g * (1.0f - sgm));
    du = dh * g * sgm;
  }
}

// bf16 storage of g and u for the clamped GLU: rounded to nearest even, but
// a value that rounding would carry across a clamp bound keeps the bound's side
// (one bf16 step back toward the value), so that the backward's clamp masks,
// taken on the stored values, decide as the forward did on the float32 ones.
__device__ __forceinline__ float bf16_keep_above(float v, float b) {  // side of v > b
  const float r = bf2f(f2bf(v));
  if ((v > b) == (r > b)) return r;
  const uint32_t bits = __float_as_uint(r);
  const bool up = v > r, pos = !(bits >> 31);
  return __uint_as_float(pos == up ? bits + 0x10000u : bits - 0x10000u);
}
template <bool CL>
__device__ __forceinline__ float act_store_g_t(const GemmArgs& a, float g) {
  if constexpr (CL) return bf16_keep_above(g, a.act_limit);
  else return g;
}
template <bool CL>
__device__ __forceinline__ float act_store_u_t(const GemmArgs& a, float u) {
  if constexpr (CL) return u >= 0.f ? bf16_keep_above(u, a.act_limit) : -bf16_keep_above(-u, a.act_limit);
  else return u;
}

__device__ __forceinline__ float act_h(const GemmArgs& a, float g, float u) {
  return a.act == MOE_ACT_CLAMPED_GLU ? act_h_t<true>(a, g, u) : act_h_t<false>(a, g, u);
}
__device__ __forceinline__ void act_grad(const GemmArgs& a, float g, float u, float dh, float& dg, float& du) {
  if (a.act == MOE_ACT_CLAMPED_GLU) act_grad_t<true>(a, g, u, dh, dg, du);
  else act_grad_t<false>(a, g, u, dh, dg, du);
}
__device__ __forceinline__ float act_store_g(const GemmArgs& a, float g) {
  return a.act == MOE_ACT_CLAMPED_GLU ? act_store_g_t<true>(a, g) : g;
}
__device__ __forceinline__ float act_store_u(const GemmArgs& a, float u) {
  return a.act == MOE_ACT_CLAMPED_GLU ? act_store_u_t<true>(a, u) : u;
}

template <int MODE>
__host__ __device__ constexpr bool is_wgrad() { return MODE == G_WGRAD_DOWN || MODE == G_WGRAD_GATEUP; }

// Tile shape: BM x BN outputs per workgroup, WM x WN wavefronts, S LDS
// stages of BK (32 or 64) k each.
template <int BM_, int BN_, int WM_, int WN_, int S_, int BK_ = 64>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, S = S_, BK = BK_;
  static constexpr int NW = WM * WN, NT = 64 * NW;
  static constexpr int TM = BM / WM, TN = BN / WN;  // wavefront tile
  static constexpr int MI = TM / 32, NI = TN / 32;  // 32x32 MFMA blocks per wavefront
  static constexpr int A_ELEMS = BM * BK, B_ELEMS = BN * BK;
  static constexpr int STAGE_ELEMS = A_ELEMS + B_ELEMS;
  static constexpr int LDS_BYTES = S * STAGE_ELEMS * 2;
  static_assert(BK == 32 || BK == 64, "k per stage");
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wavefront tile must be 32-aligned");
  static_assert(S >= 2 && S <= 5, "2..5 stages");
  static_assert(LDS_BYTES <= 150 * 1024, "LDS budget");
  static_assert((BM * BK * 2 / 1024) % NW == 0 && (BN * BK * 2 / 1024) % NW == 0,
                "every wavefront issues the same number of 1 KB copies");
};

// ---------------------------------------------------------------------------
// Tile decode
// ---------------------------------------------------------------------------
struct Tile {
  int g;          // expert
  int row_base;   // first row of the expert in the row-major activations
  int rows;       // rows of the expert (M for fwd/dgrad, K for wgrad)
  int m0, n0;     // tile origin in the output (n0 in j units for FWD_GATEUP)
  bool live;
};

// Output columns covered by one tile, and number of n-tiles.
template <int MODE, int BN>
__host__ __device__ inline int tile_cols() { return MODE == G_FWD_GATEUP ? BN / 2 : BN; }
template <int MODE, int BN>
__host__ __device__ inline int n_tiles(int d, int f) {
  const int N = (MODE == G_FWD_GATEUP || MODE == G_DGRAD_DOWN) ? f
              : (MODE == G_WGRAD_GATEUP ? 2 * f : d);
  return (N + tile_cols<MODE, BN>() - 1) / tile_cols<MODE, BN>();
}
template <int MODE>
__host__ __device__ inline int wgrad_m(int d, int f) { return MODE == G_WGRAD_DOWN ? f : d; }

// ---------------------------------------------------------------------------
// bf16 operand staging.
//
// Every operand tile is copied global -> LDS by buffer_load_dwordx4 ... lds
// (no registers): one instruction moves 64 lanes x 16 bytes into 1 KB of LDS
// at the wave-uniform address in M0, so each lane picks the global chunk that
// belongs at its LDS slot.  The copies are issued from inline assembly and
// counted by hand (s_waitcnt vmcnt), so that up to S-1 stages can be in
// flight while the compiler keeps scheduling the LDS fragment reads freely;
// the main loop issues no other vector-memory instruction.  A buffer
// descriptor spans exactly the valid rows of the operand (one expert's rows,
// or one expert's weight matrix), so reads past the last row return zeros:
// ragged expert tails and the weight gradients' K-tail need no masking.
//
// K-contiguous tiles (rows x BK k): a row is BK/8 chunks of 16 bytes whose
// index is XOR-swizzled by kswz<BK>(row); fragments are read with
// ds_read_b128 (32 consecutive rows of one chunk per half-wavefront).  The
// swizzles were chosen by measuring the fragment read pattern on gfx950:
// (row >> 1) & 7 for 128-byte rows and ((row >> 2) ^ (row >> 3)) & 3 for
// 64-byte rows read at ~190 B/clk per CU, unswizzled rows at 30-75.
// MN-contiguous tiles (BK k x columns): sub-tiles of 64 columns, one k-row =
// 8 chunks, chunk index XOR-swizzled by mswz(k); fragments read with
// ds_read_b64_tr_b16, whose lane i of each 16-lane group returns column i of
// a 4 (k) x 16 (columns) block addressed by its 16 lanes (~120 B/clk per CU
// whatever the swizzle).
// ---------------------------------------------------------------------------
template <int BK>
__device__ __forceinline__ int kswz(int r) { return BK == 64 ? (r >> 1) & 7 : ((r >> 2) ^ (r >> 3)) & 3; }
template <int BK>
__device__ __forceinline__ int k_off(int r, int c) { return r * BK + ((c ^ kswz<BK>(r)) << 3); }
__device__ __forceinline__ int mswz(int k) { return ((k >> 1) & 1) << 2; }
template <int BK>
__device__ __forceinline__ int mn_off(int k, int col) {
  return (col >> 6) * (64 * BK) + k * 64 + ((((col & 63) >> 3) ^ mswz(k)) << 3) + (col & 7);
}

// This wave's share of one K-contiguous ROWS x BK tile: 1 KB copies of
// 1024 / (2 BK) rows each.
template <int ROWS, int NW, int BK>
struct KOperand {
  static constexpr int CPR = BK / 8;                 // chunks per row
  static constexpr int NIW = ROWS * BK * 2 / 1024 / NW;  // copies per wave
  int32x4_t rsrc;
  uint32_t voff[NIW];
  __device__ __forceinline__ void init(int wave, int lane, int row0, int ld) {
#pragma unroll
    for (int j = 0; j < NIW; ++j) {
      const int q = (NIW * wave + j) * 64 + lane;
      const int row = q / CPR, phys = q % CPR;
      voff[j] = (uint32_t)(((int64_t)(row0 + row) * ld + 8 * (phys ^ kswz<BK>(row))) * 2);
    }
  }
  __device__ __forceinline__ void issue(uint32_t tile, int wave, uint32_t soff) const {
#pragma unroll
    for (int j = 0; j < NIW; ++j) dma16(rsrc, tile + (NIW * wave + j) * 1024, voff[j], soff);
  }
};

// FP8 gate/up weights: a K-contiguous ROWS x BK tile whose rows 0 .. ROWS/2-1
// are rows n0.. of the gate matrix and rows ROWS/2 .. of the same rows of the
// up matrix (each 1 KB copy lies in one half: the copy, wave-uniform, picks
// its descriptor).
template <int ROWS, int NW, int BK>
struct KOperandGU {
  static constexpr int CPR = BK / 8;
  static constexpr int NIW = ROWS * BK * 2 / 1024 / NW;
  static constexpr int RPC = 1024 / (2 * BK);              // rows per copy
  static_assert((ROWS / 2) % RPC == 0, "a copy never straddles the gate/up halves");
  int32x4_t rg, ru;
  uint32_t voff[NIW];
  __device__ __forceinline__ void init(int wave, int lane, int n0, int ld) {
#pragma unroll
    for (int j = 0; j < NIW; ++j) {
      const int q = (NIW * wave + j) * 64 + lane;
      const int row = q / CPR, phys = q % CPR;
      const int src_row = n0 + (row < ROWS / 2 ? row : row - ROWS / 2);
      voff[j] = (uint32_t)(((int64_t)src_row * ld + 8 * (phys ^ kswz<BK>(row))) * 2);
    }
  }
  __device__ __forceinline__ void issue(uint32_t tile, int wave, uint32_t soff) const {
#pragma unroll
    for (int j = 0; j < NIW; ++j) {
      const bool up = (NIW * wave + j) * RPC >= ROWS / 2;
      dma16(up ? ru : rg, tile + (NIW * wave + j) * 1024, voff[j], soff);
    }
  }
};

// This wave's share of one MN-contiguous BK x (64*NSUB) tile.  Copy t covers
// k-rows 8 (t % (BK/8)) .. +7 of sub-tile t / (BK/8); sub-tile s comes from
// descriptor src[s] starting at column col0[s].  The descriptors of this
// wave's copies are picked with constant indices (they stay in SGPRs).
template <int NSUB, int NW, int BK>
struct MNOperand {
  static constexpr int PER_SUB = BK / 8;               // copies per sub-tile
  static constexpr int NIW = NSUB * PER_SUB / NW;      // copies per wave
  int32x4_t rsrc[NIW];
  uint32_t voff[NIW];
  __device__ __forceinline__ void init(int wave, int lane, const int32x4_t* src, const int* col0, int ld) {
#pragma unroll
    for (int j = 0; j < NIW; ++j) {
      const int t = NIW * wave + j;
      const int sub = t / PER_SUB;
      const int krow = (t % PER_SUB) * 8 + (lane >> 3), phys = lane & 7;
      int c0 = 0;
#pragma unroll
      for (int q = 0; q < NSUB; ++q)
        if (q == sub) {
          rsrc[j] = src[q];
          c0 = col0[q];
        }
#pragma unroll
      for (int q = 0; q < 4; ++q) rsrc[j][q] = __builtin_amdgcn_readfirstlane(rsrc[j][q]);
      voff[j] = (uint32_t)(((int64_t)krow * ld + c0 + 8 * (phys ^ mswz(krow))) * 2);
    }
  }
  __device__ __forceinline__ void issue(uint32_t tile, int wave, uint32_t soff) const {
#pragma unroll
    for (int j = 0; j < NIW; ++j) dma16(rsrc[j], tile + (NIW * wave + j) * 1024, voff[j], soff);
  }
};

// Eight bf16 pairs (16 bytes each side) added in float32, rounded to nearest even.
__device__ __forceinline__ uint4 add_bf16x8(uint4 a, uint4 b) {
  const uint32_t x[4] = {a.x, a.y, a.z, a.w}, y[4] = {b.x, b.y, b.z, b.w};
  uint32_t r[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float lo = __uint_as_float(x[q] << 16) + __uint_as_float(y[q] << 16);
    const float hi = __uint_as_float(x[q] & 0xffff0000u) + __uint_as_float(y[q] & 0xffff0000u);
    r[q] = (uint32_t)f2bf(lo) | ((uint32_t)f2bf(hi) << 16);
  }
  return make_uint4(r[0], r[1], r[2], r[3]);
}

// 32x32x16 fragments.  K-contiguous: rows rb*32 + lane%32, k = ks*16 + 8*(lane/32) .. +7.
template <int BK>
__device__ __forceinline__ bf16x8 frag_k(const bf16_t* tile, int rb, int ks, int lane) {
  return *reinterpret_cast<const bf16x8*>(tile + k_off<BK>(rb * 32 + (lane & 31), 2 * ks + (lane >> 5)));
}
typedef int v8i __attribute__((ext_vector_type(8)));
// two 16-byte fragments as the 32-byte operand of the FP8 MFMA
__device__ __forceinline__ v8i pair8(bf16x8 lo, bf16x8 hi) {
  const v4i32 a = __builtin_bit_cast(v4i32, lo), b = __builtin_bit_cast(v4i32, hi);
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}
// MN-contiguous: columns cb*32 + lane%32, same k.
template <int BK>
__device__ __forceinline__ bf16x8 frag_mn(const bf16_t* tile, int cb, int ks, int lane) {
  const int G = lane >> 4, r = lane & 15;
  const int k = ks * 16 + 8 * (G >> 1) + (r >> 2);
  const int col = cb * 32 + 16 * (G & 1) + 4 * (r & 3);
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4_t)(tile + mn_off<BK>(k, col)));
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4_t)(tile + mn_off<BK>(k + 4, col)));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// ---------------------------------------------------------------------------
// Persistent variant.  One workgroup per CU walks its share of the tiles
// (each XCD owns a contiguous range of tile ids, its workgroups take them
// round-robin), and the LDS pipeline runs across tile boundaries: the copies
// of the next tile's first stages are in flight while the current tile's
// epilogue runs.  The epilogue is wavefront-local: each 32 x 32 block of
// results is staged through a private 2 KB LDS slot and written as 64-byte
// row pieces, with no workgroup barrier, so wavefronts that finish their
// multiplies early go on without waiting for the others.
// ---------------------------------------------------------------------------

// Logical tile count of a launch (block-wide; variable-row passes count the
// row tiles of every expert from expert_offsets into pre[]).
template <int MODE, int BM, int BN>
__device__ __forceinline__ int tile_count(const GemmArgs& a, int* pre, int* sbuf) {
  const int nt = n_tiles<MODE, BN>(a.d, a.f);
  if (is_wgrad<MODE>()) {
    const int G = a.offsets ? a.ngroups : 1;
    return G * ((wgrad_m<MODE>(a.d, a.f) + BM - 1) / BM) * nt;
  }
  if (!a.offsets) return (int)((a.dense_rows + BM - 1) / BM) * nt;
  const int G = a.ngroups;
  int c = 0;
  if ((int)threadIdx.x < G) c = (a.offsets[threadIdx.x + 1] - a.offsets[threadIdx.x] + BM - 1) / BM;
  __shared__ int total;
  const int ex = block_scan_256(c, sbuf, &total);
  if ((int)threadIdx.x < G) pre[threadIdx.x] = ex;
  __syncthreads();
  return total * nt;
}

// Tile with logical id `lin` (pre[] from tile_count for variable-row passes).
// Weight-gradient passes: ord (or null for the identity) maps the position of
// a group's tiles in the schedule to the group.
template <int MODE, int BM, int BN>
__device__ __forceinline__ Tile tile_at(const GemmArgs& a, int lin, const int* pre, const int* ord = nullptr) {
  Tile t;
  const int nt = n_tiles<MODE, BN>(a.d, a.f);
  t.live = true;
  if (is_wgrad<MODE>()) {
    const int mt = (wgrad_m<MODE>(a.d, a.f) + BM - 1) / BM;
    const int pos = lin / (mt * nt);
    t.g = ord ? ord[pos] : pos;
    const int rem = lin - pos * mt * nt;
    const int im = rem / nt;
    t.m0 = im * BM;
    t.n0 = (rem - im * nt) * BN;
    t.row_base = a.offsets ? a.offsets[t.g] : 0;
    t.rows = a.offsets ? a.offsets[t.g + 1] - t.row_base : (int)a.dense_rows;
    return t;
  }
  const int mt = lin / nt;
  constexpr int GM = 8;  // bands of row tiles (see below)
  if (!a.offsets) {
    t.g = 0;
    t.row_base = 0;
    t.rows = (int)a.dense_rows;
    const int mg = (t.rows + BM - 1) / BM;
    const int q = lin / (GM * nt), gm = min(GM, mg - q * GM);
    const int r = lin - q * GM * nt;
    t.m0 = (q * GM + r % gm) * BM;
    t.n0 = (r / gm) * tile_cols<MODE, BN>();
    return t;
  }
  int lo = 0, hi = a.ngroups - 1;  // last g with pre[g] <= mt
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pre[mid] <= mt) lo = mid; else hi = mid - 1;
  }
  t.g = lo;
  t.row_base = a.offsets[lo];
  t.rows = a.offsets[lo + 1] - t.row_base;
  // within the expert (or the one dense group), bands of up to GM row tiles
  // taken column by column (row tiles fastest): the neighbouring tiles that an
  // XCD runs together share their weight column tiles as well as their row
  // tiles
  const int local = lin - pre[lo] * nt, mg = (t.rows + BM - 1) / BM;  // (pre[] has no entry past the last group)
  const int q = local / (GM * nt), gm = min(GM, mg - q * GM);
  const int r = local - q * GM * nt;
  t.m0 = (q * GM + r % gm) * BM;
  t.n0 = (r / gm) * tile_cols<MODE, BN>();
  return t;
}

// Weight-gradient tiles cost in proportion to their expert's row count (the
// K of the product): a tile of group g costs ceil(rows_g / 32) + kWgradEpi
// units (the epilogue's share, so that empty experts, whose zero gradients
// are still written, count too).  The equal-count XCD ranges are kept when
// they leave no XCD more than 10% above the mean work (near-uniform experts,
// where re-dealing would only cost).  Otherwise the 8 XCD ranges split the
// total work evenly: each boundary is the first tile whose work midpoint lies
// at or past x/8 of the total, rounded to a multiple of the XCD's workgroup
// count.  When, besides, a single tile holds more than 1/8 of a workgroup's
// mean share (a few experts with most of the rows), round-robin dealing would
// still pile the big tiles onto some workgroups, so
//   * groups are taken in order of decreasing row count (ord[] maps a sorted
//     position to its group; ties keep the group order), so tiles of similar
//     cost sit next to each other, and
//   * inside an XCD the tiles are dealt in rounds of one tile per workgroup,
//     every other round in reverse workgroup order (snake).
// Sorting is not the default: it gathers many small experts on the same XCDs,
// where the fixed per-tile costs the work estimate leaves out add up.
// Returns whether the sorted order and snake deal are in use.
constexpr int kWgradEpi = 6;
template <int MODE, int BM, int BN>
__device__ __forceinline__ bool wgrad_schedule(const GemmArgs& a, int x, int per_x, int T, int* pre,
                                               int* ord, int* sbuf, int& lo, int& hi) {
  const int G = a.ngroups;
  const int tid = threadIdx.x;
  const int tpg = ((wgrad_m<MODE>(a.d, a.f) + BM - 1) / BM) * n_tiles<MODE, BN>(a.d, a.f);
  const int rows = tid < G ? a.offsets[tid + 1] - a.offsets[tid] : 0;
  __shared__ int wsum;
  auto scan_work = [&](int r) {
    const int w = tid < G ? (r + 31) / 32 + kWgradEpi : 0;
    const int ex = block_scan_256(w, sbuf, &wsum);
    if (tid < G) pre[tid] = ex;
    if (tid == 0) pre[G] = wsum;
    __syncthreads();
  };
  scan_work(rows);
  // per-tile work units: the tiles at position p start at tpg * pre[p]
  int64_t wall = (int64_t)tpg * wsum;
  auto work_before = [&](int t) -> int64_t {
    if (t >= T) return wall;
    const int p = t / tpg;
    return (int64_t)tpg * pre[p] + (int64_t)(t - p * tpg) * (pre[p + 1] - pre[p]);
  };
  int64_t wmax = 0;
  for (int xb = 0; xb < 8; ++xb) {
    const int l = xb * (T >> 3) + min(xb, T & 7);
    const int h = l + (T >> 3) + (xb < (T & 7) ? 1 : 0);
    wmax = max(wmax, work_before(h) - work_before(l));
  }
  if (wmax * 8 * 10 <= wall * 11) return false;  // lo, hi keep the equal-count ranges

  __shared__ int rmax;
  if (tid == 0) rmax = 0;
  __syncthreads();
  if (tid < G) atomicMax(&rmax, rows);
  __syncthreads();
  const bool sorted = ((int64_t)(rmax + 31) / 32 + kWgradEpi) * 64 * per_x > wall;
  if (sorted) {
    // rank of each group by decreasing rows, then the work prefix in that order
    if (tid < G) sbuf[tid] = rows;
    __syncthreads();
    int rank = 0;
    if (tid < G)
      for (int q = 0; q < G; ++q) {
        const int rq = sbuf[q];
        rank += (rq > rows) || (rq == rows && q < tid);
      }
    __syncthreads();
    if (tid < G) ord[rank] = tid;
    __syncthreads();
    scan_work(tid < G ? a.offsets[ord[tid] + 1] - a.offsets[ord[tid]] : 0);
    wall = (int64_t)tpg * wsum;
  }
  auto bound = [&](int xb) -> int {
    if (xb <= 0) return 0;
    if (xb >= 8) return T;
    const int64_t B = wall * xb / 8;
    int l = 0, h = G - 1;  // last position p with tpg * pre[p] <= B
    while (l < h) {
      const int mid = (l + h + 1) >> 1;
      if ((int64_t)tpg * pre[mid] <= B) l = mid; else h = mid - 1;
    }
    const int64_t w1 = pre[l + 1] - pre[l];
    const int64_t num = 2 * (B - (int64_t)tpg * pre[l]) - w1;  // tile j has midpoint >= B iff 2 w1 j >= num
    int64_t j = num <= 0 ? 0 : (num + 2 * w1 - 1) / (2 * w1);
    if (j > tpg) j = tpg;
    int64_t t = (int64_t)l * tpg + j;
    t = (t + per_x / 2) / per_x * per_x;
    return (int)(t < T ? t : T);
  };
  lo = bound(x);
  hi = bound(x + 1);
  return sorted;
}

template <int MODE>
__device__ __forceinline__ void tile_dims(const GemmArgs& a, const Tile& tl, int& K, int& M, int& N) {
  const int d = a.d, f = a.f;
  if (MODE == G_FWD_GATEUP) { K = d; M = tl.rows; N = f; }
  else if (MODE == G_FWD_DOWN) { K = f; M = tl.rows; N = d; }
  else if (MODE == G_DGRAD_DOWN) { K = d; M = tl.rows; N = f; }
  else if (MODE == G_DGRAD_GATEUP) { K = 2 * f; M = tl.rows; N = d; }
  else if (MODE == G_WGRAD_DOWN) { K = tl.rows; M = f; N = d; }
  else { K = tl.rows; M = d; N = 2 * f; }
}

// CL: the clamped GLU activation (gate/up forward and down dgrad epilogues);
// compiled as its own kernel so that the SwiGLU kernels carry none of its code.
// FP8 (forward and data-gradient passes): E4M3 operands, both K-contiguous
// (activation rows; the weight cache's transposed weights for the forward, its
// row-quantised natural layouts for the data gradients), staged exactly like
// bf16 data of half the K (a 16-byte chunk holds 16 codes);
// v_mfma_f32_32x32x64_f8f6f4 takes two bf16-sized fragments per operand (the
// same k subset on both sides); the epilogues multiply the float32
// accumulators by the row's and the column's quantisation scales.
template <int MODE, class C, bool CL = false, bool FP8 = false>
__global__ __launch_bounds__(C::NT, C::NW == 4 ? 2 : 1) void gemm_bf16_persistent(GemmArgs a) {
  static_assert(!FP8 || !is_wgrad<MODE>(), "FP8: the forward and data-gradient passes only");
  constexpr bool wgrad = is_wgrad<MODE>();
  constexpr bool a_mn = wgrad;
  constexpr bool b_mn = !FP8 && (MODE == G_FWD_GATEUP || MODE == G_FWD_DOWN || wgrad);
  constexpr int BM = C::BM, BN = C::BN, MI = C::MI, NI = C::NI, S = C::S, NW = C::NW, BK = C::BK;
  static_assert(MODE != G_FWD_GATEUP || NI % 2 == 0, "gate/up pairs need an even number of column blocks");
  __shared__ __align__(16) bf16_t lds[S][C::STAGE_ELEMS];
  __shared__ __align__(16) bf16_t epi[NW][wgrad ? 32 * 64 : 32 * 32];
  __shared__ int pre[257];
  __shared__ int sbuf[256];
  __shared__ int ord[wgrad ? 256 : 1];

  const int T = tile_count<MODE, BM, BN>(a, pre, sbuf);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / C::WN, wn = wave % C::WN;
  const int d = a.d, f = a.f;
  // this workgroup's tiles: in round r, lo + r * per_x + jx (or + per_x - 1 - jx
  // in the odd rounds of a snake deal), while < hi (grid is a multiple of 8)
  const int per_x = gridDim.x >> 3, x = blockIdx.x & 7, jx = blockIdx.x >> 3;
  int lo = x * (T >> 3) + min(x, T & 7);
  int hi = lo + (T >> 3) + (x < (T & 7) ? 1 : 0);
  bool snake = false;
  if (wgrad && a.offsets) {
    snake = wgrad_schedule<MODE, BM, BN>(a, x, per_x, T, pre, ord, sbuf, lo, hi);
    // the same in every lane (computed from LDS): keep the tile loops uniform
    lo = __builtin_amdgcn_readfirstlane(lo);
    hi = __builtin_amdgcn_readfirstlane(hi);
    snake = __builtin_amdgcn_readfirstlane((int)snake) != 0;
  }
  const int* tord = snake ? ord : nullptr;
  auto tile_of = [&](int r) { return lo + r * per_x + ((snake && (r & 1)) ? per_x - 1 - jx : jx); };

  const bf16_t* A = reinterpret_cast<const bf16_t*>(a.a);
  const bf16_t* Bact = reinterpret_cast<const bf16_t*>(a.b);
  const bf16_t* W0 = reinterpret_cast<const bf16_t*>(a.w0);
  const bf16_t* W1 = reinterpret_cast<const bf16_t*>(a.w1);

  // ---- producer: copies of (tile, k-step) stages in consumption order
  KOperand<BM, NW, BK> ka;
  MNOperand<BM / 64, NW, BK> ma;
  KOperand<BN, NW, BK> kb;
  KOperandGU<BN, NW, BK> kgu;
  MNOperand<BN / 64, NW, BK> mb;
  int32x4_t b_up = make_rsrc(W0, 0);
  int64_t a_kstride = 0, b_kstride = 0;
  int p_r = 0, p_t = tile_of(0), p_k = 0, p_nk = 0;
  auto setup = [&](const Tile& tl) {
    int K, M, N;
    tile_dims<MODE>(a, tl, K, M, N);
    const int g = tl.g;
    if (!a_mn) {
      // (FP8 rows: K codes = K/2 two-byte units)
      const int lda = (MODE == G_FWD_DOWN ? f : (MODE == G_DGRAD_GATEUP ? 2 * f : d)) / (FP8 ? 2 : 1);
      ka.rsrc = make_rsrc(A + (int64_t)tl.row_base * lda, (int64_t)M * lda * 2);
      ka.init(wave, lane, tl.m0, lda);
      a_kstride = 2;
    } else {
      const int lda = MODE == G_WGRAD_DOWN ? f : d;
      const int32x4_t r = make_rsrc(A + (int64_t)tl.row_base * lda, (int64_t)K * lda * 2);
      int32x4_t src[BM / 64];
      int col0[BM / 64];
#pragma unroll
      for (int s2 = 0; s2 < BM / 64; ++s2) {
        src[s2] = r;
        col0[s2] = tl.m0 + 64 * s2;
      }
      ma.init(wave, lane, src, col0, lda);
      a_kstride = (int64_t)lda * 2;
    }
    if (FP8 && MODE == G_FWD_GATEUP) {
      // cache rows: [E][f][d] codes of the gate and of the up weights
      const uint8_t* qg = reinterpret_cast<const uint8_t*>(a.w0) + (int64_t)g * f * d;
      const uint8_t* qu = reinterpret_cast<const uint8_t*>(a.w1) + (int64_t)g * f * d;
      kgu.rg = make_rsrc(qg, (int64_t)f * d);
      kgu.ru = make_rsrc(qu, (int64_t)f * d);
      kgu.init(wave, lane, tl.n0, d / 2);
      b_kstride = 2;
    } else if (FP8 && MODE == G_FWD_DOWN) {
      // cache rows: [E][d][f] codes of the down weights
      kb.rsrc = make_rsrc(reinterpret_cast<const uint8_t*>(a.w0) + (int64_t)g * d * f, (int64_t)d * f);
      kb.init(wave, lane, tl.n0, f / 2);
      b_kstride = 2;
    } else if (FP8 && MODE == G_DGRAD_DOWN) {
      // cache rows: [E][f][d] row codes of the down weights
      kb.rsrc = make_rsrc(reinterpret_cast<const uint8_t*>(a.w0) + (int64_t)g * f * d, (int64_t)f * d);
      kb.init(wave, lane, tl.n0, d / 2);
      b_kstride = 2;
    } else if (FP8 && MODE == G_DGRAD_GATEUP) {
      // cache rows: [E][d][2f] row codes of [W_gate | W_up]
      kb.rsrc = make_rsrc(reinterpret_cast<const uint8_t*>(a.w0) + (int64_t)g * d * 2 * f, (int64_t)d * 2 * f);
      kb.init(wave, lane, tl.n0, f);
      b_kstride = 2;
    } else if (MODE == G_FWD_GATEUP) {
      const int32x4_t rg = make_rsrc(W0 + (int64_t)g * d * f, (int64_t)d * f * 2);
      const int32x4_t ru = make_rsrc(W1 + (int64_t)g * d * f, (int64_t)d * f * 2);
      int32x4_t src[BN / 64];
      int col0[BN / 64];
#pragma unroll
      for (int s2 = 0; s2 < BN / 64; ++s2) {
        const bool up = s2 >= BN / 128;
        src[s2] = up ? ru : rg;
        col0[s2] = tl.n0 + 64 * (up ? s2 - BN / 128 : s2);
      }
      mb.init(wave, lane, src, col0, f);
      b_kstride = (int64_t)f * 2;
    } else if (MODE == G_FWD_DOWN) {
      const int32x4_t r = make_rsrc(W0 + (int64_t)g * f * d, (int64_t)f * d * 2);
      int32x4_t src[BN / 64];
      int col0[BN / 64];
#pragma unroll
      for (int s2 = 0; s2 < BN / 64; ++s2) {
        src[s2] = r;
        col0[s2] = tl.n0 + 64 * s2;
      }
      mb.init(wave, lane, src, col0, d);
      b_kstride = (int64_t)d * 2;
    } else if (MODE == G_DGRAD_DOWN) {
      kb.rsrc = make_rsrc(W0 + (int64_t)g * f * d, (int64_t)f * d * 2);
      kb.init(wave, lane, tl.n0, d);
      b_kstride = 2;
    } else if (MODE == G_DGRAD_GATEUP) {
      kb.rsrc = make_rsrc(W0 + (int64_t)g * d * f, (int64_t)d * f * 2);
      b_up = make_rsrc(W1 + (int64_t)g * d * f, (int64_t)d * f * 2);
      kb.init(wave, lane, tl.n0, f);
      b_kstride = 2;
    } else {
      const int ldb = MODE == G_WGRAD_DOWN ? d : 2 * f;
      const int32x4_t r = make_rsrc(Bact + (int64_t)tl.row_base * ldb, (int64_t)K * ldb * 2);
      int32x4_t src[BN / 64];
      int col0[BN / 64];
#pragma unroll
      for (int s2 = 0; s2 < BN / 64; ++s2) {
        src[s2] = r;
        col0[s2] = tl.n0 + 64 * s2;
      }
      mb.init(wave, lane, src, col0, ldb);
      b_kstride = (int64_t)ldb * 2;
    }
  };
  // advance the producer to the next tile with work (weight-gradient tiles
  // of experts without rows have none)
  auto p_seek = [&]() {
    while (p_t < hi) {
      const Tile tl = tile_at<MODE, BM, BN>(a, p_t, pre, tord);
      int K, M, N;
      tile_dims<MODE>(a, tl, K, M, N);
      if constexpr (FP8) K >>= 1;  // two-byte units of codes
      p_nk = (K + BK - 1) / BK;
      if (p_nk > 0) {
        setup(tl);
        return;
      }
      p_t = tile_of(++p_r);
    }
  };
  const uint32_t lds0 = lds_addr(&lds[0][0]);
  auto p_issue = [&](int buf) {
    const int k0 = p_k * BK;
    const uint32_t As = lds0 + buf * (C::STAGE_ELEMS * 2);
    const uint32_t Bs = As + C::A_ELEMS * 2;
    if (!a_mn) ka.issue(As, wave, (uint32_t)(k0 * a_kstride));
    else ma.issue(As, wave, (uint32_t)(k0 * a_kstride));
    if (FP8 && MODE == G_FWD_GATEUP) {
      kgu.issue(Bs, wave, (uint32_t)(k0 * b_kstride));
    } else if (MODE == G_DGRAD_GATEUP && !FP8) {
      KOperand<BN, NW, BK> kk = kb;
      if (k0 >= f) kk.rsrc = b_up;
      kk.issue(Bs, wave, (uint32_t)((k0 >= f ? k0 - f : k0) * b_kstride));
    } else if (MODE == G_DGRAD_DOWN || MODE == G_DGRAD_GATEUP || (FP8 && MODE == G_FWD_DOWN)) {
      kb.issue(Bs, wave, (uint32_t)(k0 * b_kstride));
    } else {
      mb.issue(Bs, wave, (uint32_t)(k0 * b_kstride));
    }
    if (++p_k == p_nk) {
      p_k = 0;
      p_t = tile_of(++p_r);
      p_seek();
    }
  };
  constexpr int NL = (BM + BN) * BK * 2 / 1024 / NW;  // copies per thread per stage
  int issued = 0, consumed = 0;
  int landed = 0;  // stages below this index are known to be in LDS
  p_seek();
#pragma unroll
  for (int i = 0; i < S - 1; ++i)
    if (p_t < hi) {
      p_issue(issued % S);
      ++issued;
    }

  auto bcol = [&](int j) {
    if (MODE == G_FWD_GATEUP)
      return (j < NI / 2) ? (wn * (NI / 2) + j) : (BN / 64 + wn * (NI / 2) + (j - NI / 2));
    return wn * NI + j;
  };
  bf16_t* ep = &epi[wave][0];
  const int hh = lane >> 5, r32 = lane & 31;
  // stage this lane's 4 x 4 values of a 32 x 32 block (row r32, columns
  // 8q + 4hh + t) and store the block's rows: dst(r) is row r's pointer at
  // the block's first column (null: row not stored), ncols valid columns
  auto put_block = [&](const float* v, auto&& dst, int ncols, bool accum = false) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo2 = (uint32_t)f2bf(v[4 * q]) | ((uint32_t)f2bf(v[4 * q + 1]) << 16);
      const uint32_t hi2 = (uint32_t)f2bf(v[4 * q + 2]) | ((uint32_t)f2bf(v[4 * q + 3]) << 16);
      *reinterpret_cast<uint2*>(ep + r32 * 32 + ((q ^ ((r32 >> 2) & 3)) << 3) + 4 * hh) = make_uint2(lo2, hi2);
    }
#pragma unroll
    for (int rep = 0; rep < 2; ++rep) {
      const int idx = lane + 64 * rep, r = idx >> 2, ch = idx & 3;
      const uint4 val = *reinterpret_cast<const uint4*>(ep + r * 32 + ((ch ^ ((r >> 2) & 3)) << 3));
      bf16_t* p = dst(r);
      if (p && 8 * ch < ncols) {
        uint4 w = val;
        if (accum) {  // (weight gradients) add to the stored values, in float32
          const uint4 old = *reinterpret_cast<const uint4*>(p + 8 * ch);
          w = add_bf16x8(old, val);
        }
        *reinterpret_cast<uint4*>(p + 8 * ch) = w;
      }
    }
  };

  for (int c_r = 0, c_t = tile_of(0); c_t < hi; c_t = tile_of(++c_r)) {
    const Tile tl = tile_at<MODE, BM, BN>(a, c_t, pre, tord);
    int K, M, N;
    tile_dims<MODE>(a, tl, K, M, N);
    if constexpr (FP8) K >>= 1;
    const int g = tl.g;
    const int nk = (K + BK - 1) / BK;
    // 32-row blocks of this wavefront that hold rows of the tile (a ragged
    // last tile of an expert has fewer): the others skip their fragment reads
    // and MFMAs (no rows at all: the SIMD partner has the matrix pipe alone)
    const int live = __builtin_amdgcn_readfirstlane(max(0, min(MI, (M - (tl.m0 + wm * C::TM) + 31) / 32)));
    const bool wave_rows = live > 0;
    const bool colsum = wgrad && a.db0 && tl.m0 == 0 && wm == 0;
    floatx16 acc[MI][NI];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
    float bsum[NI];
#pragma unroll
    for (int j = 0; j < NI; ++j) bsum[j] = 0.f;

    // the k loop, in two copies: tiles whose wavefront rows are all live run
    // the MFMA block without tests, ragged ones skip their dead row blocks
    auto k_loop = [&](auto all_live) {
    for (int kt = 0; kt < nk; ++kt) {
      const int ahead = issued - consumed - 1;  // stages issued after this one
      if (consumed < landed) {
        // landed before the previous tile's epilogue stores: no wait
      } else if (S >= 5 && ahead >= 3) wait_vmcnt<(S >= 5 ? 3 : 0) * NL>();
      else if (S >= 4 && ahead >= 2) wait_vmcnt<(S >= 4 ? 2 : 0) * NL>();
      else if (S >= 3 && ahead >= 1) wait_vmcnt<(S >= 3 ? 1 : 0) * NL>();
      else wait_vmcnt<0>();
      __syncthreads();
      if (p_t < hi) {
        p_issue(issued % S);
        ++issued;
      }
      const bf16_t* As = lds[consumed % S];
      const bf16_t* Bs = As + C::A_ELEMS;
      ++consumed;
      if (!wave_rows) continue;
      if constexpr (FP8) {
        // 64 codes of k per instruction: chunks 2ks, 2ks+1 of the bf16 layout
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
          v8i b8[NI];
#pragma unroll
          for (int j = 0; j < NI; ++j)
            b8[j] = pair8(frag_k<BK>(Bs, bcol(j), 2 * ks, lane), frag_k<BK>(Bs, bcol(j), 2 * ks + 1, lane));
#pragma unroll
          for (int i = 0; i < MI; ++i)
            if (decltype(all_live)::value || i < live) {
              const v8i a8 =
                  pair8(frag_k<BK>(As, wm * MI + i, 2 * ks, lane), frag_k<BK>(As, wm * MI + i, 2 * ks + 1, lane));
#pragma unroll
              for (int j = 0; j < NI; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(b8[j], a8, acc[i][j], 0, 0, 0, 127, 0,
                                                                            127);
            }
        }
      } else {
      bf16x8 af[2][MI], bfr[2][NI];
      auto load_frags = [&](int ks, int slot) {
#pragma unroll
        for (int i = 0; i < MI; ++i)
          af[slot][i] = a_mn ? frag_mn<BK>(As, wm * MI + i, ks, lane) : frag_k<BK>(As, wm * MI + i, ks, lane);
#pragma unroll
        for (int j = 0; j < NI; ++j)
          bfr[slot][j] = b_mn ? frag_mn<BK>(Bs, bcol(j), ks, lane) : frag_k<BK>(Bs, bcol(j), ks, lane);
      };
      constexpr int KS = BK / 16;
      load_frags(0, 0);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int cur = ks & 1;
        if (ks < KS - 1) load_frags(ks + 1, cur ^ 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < MI; ++i)
          if (decltype(all_live)::value || i < live)
#pragma unroll
            for (int j = 0; j < NI; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[cur][j], af[cur][i], acc[i][j], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
        if (colsum) {
#pragma unroll
          for (int j = 0; j < NI; ++j) {
            const uint4 u = __builtin_bit_cast(uint4, bfr[cur][j]);
            const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int q = 0; q < 4; ++q)
              bsum[j] += __uint_as_float(w4[q] << 16) + __uint_as_float(w4[q] & 0xffff0000u);
          }
        }
      }
      }  // bf16
    }
    };
    if (live == MI) k_loop(std::true_type{});
    else k_loop(std::false_type{});
    // weight gradients (few k-steps per tile, 128 KB of output per tile): every
    // copy in flight, the next tile's first stages, lands before this tile's
    // output stores are issued, so that those stages are multiplied without a
    // vmcnt wait (which would also wait for the stores) while the stores
    // drain (DeepSeek-V3 shape: gate/up wgrad 7.08 -> 6.67 ms; the forward and
    // data-gradient passes, with long k loops, were 1-4% slower with it)
    if constexpr (wgrad) {
      wait_vmcnt<0>();
      landed = issued;
    }

    // ---- epilogue (this wavefront's rows only).  Block (i, j) holds the
    // transposed product: lane l has row 32i + l%32, register v = 4q + t
    // column 32j + 8q + 4(l/32) + t.
    const int mrow0 = tl.m0 + wm * C::TM;
    if (MODE == G_FWD_GATEUP) {
      auto epi = [&](auto) {
        bf16_t* gu = reinterpret_cast<bf16_t*>(a.c0);
        bf16_t* h = reinterpret_cast<bf16_t*>(a.c1);
        const bf16_t* bgp = reinterpret_cast<const bf16_t*>(a.bias0);
        const bf16_t* bup = reinterpret_cast<const bf16_t*>(a.bias1);
        const int jbase = tl.n0 + wn * (C::TN / 2);
  #pragma unroll
        for (int j = 0; j < NI / 2; ++j) {
          const int jj0 = jbase + 32 * j;
          const int ncols = min(32, N - jj0);
          float bgv[16], buv[16], sgv[16], suv[16];
  #pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int c = jj0 + 8 * (v >> 2) + 4 * hh + (v & 3);
            bgv[v] = (bgp && c < N) ? bf2f(bgp[(int64_t)g * f + c]) : 0.f;
            buv[v] = (bup && c < N) ? bf2f(bup[(int64_t)g * f + c]) : 0.f;
            sgv[v] = 1.f;
            suv[v] = 1.f;
            if constexpr (FP8) {  // the weight columns' quantisation scales
              sgv[v] = c < N ? a.b_scale0[(int64_t)g * f + c] : 0.f;
              suv[v] = c < N ? a.b_scale1[(int64_t)g * f + c] : 0.f;
            }
          }
  #pragma unroll
          for (int i = 0; i < MI; ++i) {
            const int m0 = mrow0 + 32 * i;
            if (m0 >= M || ncols <= 0) continue;
            // FP8: the activation row's scale
            const float sr = FP8 ? (m0 + r32 < M ? a.a_scale[tl.row_base + m0 + r32] : 0.f) : 1.f;
            float gv[16], uv[16], hv[16];
  #pragma unroll
            for (int v = 0; v < 16; ++v) {
              gv[v] = FP8 ? __builtin_fmaf(acc[i][j][v], sr * sgv[v], bgv[v]) : acc[i][j][v] + bgv[v];
              uv[v] = FP8 ? __builtin_fmaf(acc[i][j + NI / 2][v], sr * suv[v], buv[v]) : acc[i][j + NI / 2][v] + buv[v];
              hv[v] = act_h_t<CL>(a, gv[v], uv[v]);
              gv[v] = act_store_g_t<CL>(a, gv[v]);
              uv[v] = act_store_u_t<CL>(a, uv[v]);
            }
            auto row_gu = [&](int half) {
              return [&, half](int r) -> bf16_t* {
                return m0 + r < M ? gu + (int64_t)(tl.row_base + m0 + r) * 2 * f + half * f + jj0 : nullptr;
              };
            };
            put_block(gv, row_gu(0), ncols);
            put_block(uv, row_gu(1), ncols);
            put_block(hv, [&](int r) -> bf16_t* {
              return m0 + r < M ? h + (int64_t)(tl.row_base + m0 + r) * f + jj0 : nullptr;
            }, ncols);
          }
        }
      };
      epi(0);
    } else if (MODE == G_DGRAD_DOWN) {
      auto epi = [&](auto) {
        // dSwiGLU with the saved gate/up values: for each 32-row block, every
        // gate/up load of the wavefront's columns is issued before any math
        const int nbase = tl.n0 + wn * C::TN;
        const bf16_t* gup = reinterpret_cast<const bf16_t*>(a.aux);
        bf16_t* out = reinterpret_cast<bf16_t*>(a.c0);
        constexpr int JB = NI > 2 ? 2 : NI;  // column blocks per batch of loads
  #pragma unroll
        for (int i = 0; i < MI; ++i) {
          const int m0 = mrow0 + 32 * i;
          if (m0 >= M) continue;
          const int m = m0 + r32;
          const int64_t row = tl.row_base + (m < M ? m : M - 1);
          // FP8: the d_o row's quantisation scale
          const float sr = FP8 ? (m < M ? a.a_scale[row] : 0.f) : 1.f;
  #pragma unroll
          for (int jb = 0; jb < NI; jb += JB) {
            uint2 gr[JB][4], ur[JB][4];
  #pragma unroll
            for (int jj = 0; jj < JB; ++jj)
  #pragma unroll
              for (int q = 0; q < 4; ++q) {
                const int c = nbase + 32 * (jb + jj) + 8 * q + 4 * hh;
                gr[jj][q] = make_uint2(0, 0);
                ur[jj][q] = make_uint2(0, 0);
                if (m < M && c < N) {
                  gr[jj][q] = *reinterpret_cast<const uint2*>(gup + row * 2 * f + c);
                  ur[jj][q] = *reinterpret_cast<const uint2*>(gup + row * 2 * f + f + c);
                }
              }
  #pragma unroll
            for (int jj = 0; jj < JB; ++jj) {
              const int j = jb + jj;
              const int n0 = nbase + 32 * j;
              const int ncols = min(32, N - n0);
              if (ncols <= 0) continue;
              float dg[16], du[16];
  #pragma unroll
              for (int q = 0; q < 4; ++q) {
                const float gv[4] = {__uint_as_float(gr[jj][q].x << 16), __uint_as_float(gr[jj][q].x & 0xffff0000u),
                                     __uint_as_float(gr[jj][q].y << 16), __uint_as_float(gr[jj][q].y & 0xffff0000u)};
                const float uv[4] = {__uint_as_float(ur[jj][q].x << 16), __uint_as_float(ur[jj][q].x & 0xffff0000u),
                                     __uint_as_float(ur[jj][q].y << 16), __uint_as_float(ur[jj][q].y & 0xffff0000u)};
                float sc[4] = {1.f, 1.f, 1.f, 1.f};
                if constexpr (FP8) {  // the W_down rows' scales (dh columns c .. c + 3)
                  const int c = n0 + 8 * q + 4 * hh;
                  const float4 s4 = c < N ? *reinterpret_cast<const float4*>(a.b_scale0 + (int64_t)g * f + c)
                                          : make_float4(0.f, 0.f, 0.f, 0.f);
                  sc[0] = sr * s4.x;
                  sc[1] = sr * s4.y;
                  sc[2] = sr * s4.z;
                  sc[3] = sr * s4.w;
                }
  #pragma unroll
                for (int t = 0; t < 4; ++t)
                  act_grad_t<CL>(a, gv[t], uv[t], FP8 ? acc[i][j][4 * q + t] * sc[t] : acc[i][j][4 * q + t],
                                 dg[4 * q + t], du[4 * q + t]);
              }
              put_block(dg, [&](int r) -> bf16_t* {
                return m0 + r < M ? out + (int64_t)(tl.row_base + m0 + r) * 2 * f + n0 : nullptr;
              }, ncols);
              put_block(du, [&](int r) -> bf16_t* {
                return m0 + r < M ? out + (int64_t)(tl.row_base + m0 + r) * 2 * f + f + n0 : nullptr;
              }, ncols);
            }
          }
        }
      };
      epi(0);
    } else if (MODE == G_FWD_DOWN || MODE == G_DGRAD_GATEUP) {
      const int nbase = tl.n0 + wn * C::TN;
      const bf16_t* bdp = MODE == G_FWD_DOWN ? reinterpret_cast<const bf16_t*>(a.bias0) : nullptr;
      bf16_t* out = reinterpret_cast<bf16_t*>(a.c0);
      if (MODE == G_FWD_DOWN && !FP8 && !bdp) {
        // nothing to load per column block: row blocks outer, so that the two
        // 64-byte pieces of a row's 128-byte line leave one after the other
        // (down forward, Qwen3 shape 286 -> 267 us, DeepSeek-V3 2365 -> 2352;
        // the gate/up dgrad's 4 x 2 wavefront tiles were 1-3% slower with it)
#pragma unroll
        for (int i = 0; i < MI; ++i) {
          const int m0 = mrow0 + 32 * i;
          if (m0 >= M) continue;
#pragma unroll
          for (int j = 0; j < NI; ++j) {
            const int n0 = nbase + 32 * j;
            const int ncols = min(32, N - n0);
            if (ncols <= 0) continue;
            float o[16];
#pragma unroll
            for (int v = 0; v < 16; ++v) o[v] = acc[i][j][v];
            put_block(o, [&](int r) -> bf16_t* {
              return m0 + r < M ? out + (int64_t)(tl.row_base + m0 + r) * N + n0 : nullptr;
            }, ncols);
          }
        }
      } else
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int n0 = nbase + 32 * j;
        const int ncols = min(32, N - n0);
        float bd[16], sc[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int c = n0 + 8 * (v >> 2) + 4 * hh + (v & 3);
          bd[v] = (bdp && c < N) ? bf2f(bdp[(int64_t)g * d + c]) : 0.f;
          sc[v] = 1.f;
          if constexpr (FP8) sc[v] = c < N ? a.b_scale0[(int64_t)g * N + c] : 0.f;  // weight column scales
        }
#pragma unroll
        for (int i = 0; i < MI; ++i) {
          const int m0 = mrow0 + 32 * i;
          if (m0 >= M || ncols <= 0) continue;
          const float sr = FP8 ? (m0 + r32 < M ? a.a_scale[tl.row_base + m0 + r32] : 0.f) : 1.f;
          float o[16];
#pragma unroll
          for (int v = 0; v < 16; ++v) o[v] = FP8 ? __builtin_fmaf(acc[i][j][v], sr * sc[v], bd[v]) : acc[i][j][v] + bd[v];
          put_block(o, [&](int r) -> bf16_t* {
            return m0 + r < M ? out + (int64_t)(tl.row_base + m0 + r) * N + n0 : nullptr;
          }, ncols);
        }
      }
    } else {
      const int nbase = tl.n0 + wn * C::TN;
      bf16_t* c0 = reinterpret_cast<bf16_t*>(a.c0);
      bf16_t* c1 = reinterpret_cast<bf16_t*>(a.c1);
      if (!a.accumulate) {
        // two adjacent 32 x 32 blocks staged together, so that each row leaves
        // as one whole 128-byte line, with nontemporal stores: the gradients
        // are not read again by the layer (DeepSeek-V3 shape: down wgrad
        // 3.56 -> 3.06 ms, gate/up 7.20 -> 7.09; with 64-byte half lines
        // nontemporal stores were slower than plain ones)
#pragma unroll
        for (int i = 0; i < MI; ++i) {
          const int m0 = mrow0 + 32 * i;
#pragma unroll
          for (int jp = 0; jp < NI / 2; ++jp) {
            const int n0 = nbase + 64 * jp;
            const int ncols = min(64, N - n0);
            if (m0 >= M || ncols <= 0) continue;
#pragma unroll
            for (int half = 0; half < 2; ++half)
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const floatx16& v = acc[i][2 * jp + half];
                const uint32_t lo2 = (uint32_t)f2bf(v[4 * q]) | ((uint32_t)f2bf(v[4 * q + 1]) << 16);
                const uint32_t hi2 = (uint32_t)f2bf(v[4 * q + 2]) | ((uint32_t)f2bf(v[4 * q + 3]) << 16);
                *reinterpret_cast<uint2*>(ep + r32 * 64 + (((4 * half + q) ^ (r32 & 7)) << 3) + 4 * hh) =
                    make_uint2(lo2, hi2);
              }
#pragma unroll
            for (int rep = 0; rep < 4; ++rep) {
              const int idx = lane + 64 * rep, r = idx >> 3, ch = idx & 7;
              const uint4 val = *reinterpret_cast<const uint4*>(ep + r * 64 + ((ch ^ (r & 7)) << 3));
              const int m = m0 + r;
              bf16_t* pp = m >= M ? nullptr
                         : MODE == G_WGRAD_DOWN ? c0 + ((int64_t)g * f + m) * d + n0
                         : n0 < f ? c0 + ((int64_t)g * d + m) * f + n0
                                  : c1 + ((int64_t)g * d + m) * f + (n0 - f);
              if (pp && 8 * ch < ncols)
                __builtin_nontemporal_store(__builtin_bit_cast(v4i32, val), reinterpret_cast<v4i32*>(pp + 8 * ch));
            }
          }
        }
      } else
      // row blocks outer: the adjacent 64-byte pieces of a row go out together
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const int m0 = mrow0 + 32 * i;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
          const int n0 = nbase + 32 * j;
          const int ncols = min(32, N - n0);
          if (m0 >= M || ncols <= 0) continue;
          float o[16];
#pragma unroll
          for (int v = 0; v < 16; ++v) o[v] = acc[i][j][v];
          put_block(o, [&](int r) -> bf16_t* {
            const int m = m0 + r;
            if (m >= M) return nullptr;
            if (MODE == G_WGRAD_DOWN) return c0 + ((int64_t)g * f + m) * d + n0;
            if (n0 < f) return c0 + ((int64_t)g * d + m) * f + n0;
            return c1 + ((int64_t)g * d + m) * f + (n0 - f);
          }, ncols, a.accumulate);
        }
      }
      if (colsum) {
#pragma unroll
        for (int j = 0; j < NI; ++j) {
          float v = bsum[j];
          v += __shfl_xor(v, 32, 64);
          const int col = tl.n0 + wn * C::TN + j * 32 + r32;
          if (lane < 32 && col < N) {
            bf16_t* p = MODE == G_WGRAD_DOWN ? reinterpret_cast<bf16_t*>(a.db0) + (int64_t)g * d + col
                      : col < f ? reinterpret_cast<bf16_t*>(a.db0) + (int64_t)g * f + col
                                : reinterpret_cast<bf16_t*>(a.db1) + (int64_t)g * f + col - f;
            *p = f2bf(a.accumulate ? bf2f(*p) + v : v);
          }
        }
      }
    }
  }
  wait_vmcnt<0>();  // no copy may still target this workgroup's LDS at exit
}

// ---------------------------------------------------------------------------
// fp32 path: plain kernel, 16x16 outputs per 256-thread block
// ---------------------------------------------------------------------------
template <int MODE>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  __shared__ int pre[257];
  __shared__ int sbuf[256];
  constexpr int TS = 16;
  constexpr bool wgrad = MODE == G_WGRAD_DOWN || MODE == G_WGRAD_GATEUP;
  const int d = a.d, f = a.f;
  const float* A = reinterpret_cast<const float*>(a.a);
  const float* Bact = reinterpret_cast<const float*>(a.b);
  const float* W0 = reinterpret_cast<const float*>(a.w0);
  const float* W1 = reinterpret_cast<const float*>(a.w1);
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  int g, row_base, rows, m, n;
  if (wgrad) {
    const int Mfix = MODE == G_WGRAD_DOWN ? f : d;
    const int Nfix = MODE == G_WGRAD_DOWN ? d : 2 * f;
    const int mt = (Mfix + TS - 1) / TS, nt = (Nfix + TS - 1) / TS;
    const int lin = blockIdx.x;
    g = lin / (mt * nt);
    const int rem = lin - g * mt * nt;
    m = (rem / nt) * TS + ty;
    n = (rem % nt) * TS + tx;
    row_base = a.offsets ? a.offsets[g] : 0;
    rows = a.offsets ? a.offsets[g + 1] - row_base : (int)a.dense_rows;
    if (m >= Mfix || n >= Nfix) return;
    float acc = 0.f, bs = 0.f;
    const bool colsum = a.db0 && m == 0;
    for (int r = 0; r < rows; ++r) {
      const int64_t rr = row_base + r;
      const float bv = MODE == G_WGRAD_DOWN ? Bact[rr * d + n] : Bact[rr * 2 * f + n];
      const float av = MODE == G_WGRAD_DOWN ? A[rr * f + m] : A[rr * d + m];
      acc = __builtin_fmaf(av, bv, acc);
      bs += bv;
    }
    float* c0 = reinterpret_cast<float*>(a.c0);
    float* c1 = reinterpret_cast<float*>(a.c1);
    auto put = [&](float* p, float v) { *p = a.accumulate ? *p + v : v; };
    if (MODE == G_WGRAD_DOWN) {
      put(c0 + ((int64_t)g * f + m) * d + n, acc);
      if (colsum) put(reinterpret_cast<float*>(a.db0) + (int64_t)g * d + n, bs);
    } else if (n < f) {
      put(c0 + ((int64_t)g * d + m) * f + n, acc);
      if (colsum) put(reinterpret_cast<float*>(a.db0) + (int64_t)g * f + n, bs);
    } else {
      put(c1 + ((int64_t)g * d + m) * f + n - f, acc);
      if (colsum) put(reinterpret_cast<float*>(a.db1) + (int64_t)g * f + n - f, bs);
    }
    return;
  }
  const int N = (MODE == G_FWD_GATEUP || MODE == G_DGRAD_DOWN) ? f : d;
  const int nt = (N + TS - 1) / TS;
  const int mtile = blockIdx.x / nt;
  n = (blockIdx.x % nt) * TS + tx;
  if (a.offsets) {
    const int G = a.ngroups;
    int c = 0;
    if ((int)threadIdx.x < G) c = (a.offsets[threadIdx.x + 1] - a.offsets[threadIdx.x] + TS - 1) / TS;
    __shared__ int total;
    const int ex = block_scan_256(c, sbuf, &total);
    if ((int)threadIdx.x < G) pre[threadIdx.x] = ex;
    __syncthreads();
    if (mtile >= total) return;
    int lo = 0, hi = G - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (pre[mid] <= mtile) lo = mid; else hi = mid - 1;
    }
    g = lo;
    row_base = a.offsets[g];
    rows = a.offsets[g + 1] - row_base;
    m = (mtile - pre[g]) * TS + ty;
  } else {
    g = 0;
    row_base = 0;
    rows = (int)a.dense_rows;
    m = mtile * TS + ty;
  }
  if (m >= rows || n >= N) return;
  const int64_t row = row_base + m;
  if (MODE == G_FWD_GATEUP) {
    float ag = 0.f, au = 0.f;
    const float* wg = W0 + (int64_t)g * d * f + n;
    const float* wu = W1 + (int64_t)g * d * f + n;
    for (int k = 0; k < d; ++k) {
      const float xv = A[row * d + k];
      ag = __builtin_fmaf(xv, wg[(int64_t)k * f], ag);
      au = __builtin_fmaf(xv, wu[(int64_t)k * f], au);
    }
    if (a.bias0) ag += reinterpret_cast<const float*>(a.bias0)[(int64_t)g * f + n];
    if (a.bias1) au += reinterpret_cast<const float*>(a.bias1)[(int64_t)g * f + n];
    float* gu = reinterpret_cast<float*>(a.c0);
    gu[row * 2 * f + n] = ag;
    gu[row * 2 * f + f + n] = au;
    reinterpret_cast<float*>(a.c1)[row * f + n] = act_h(a, ag, au);
  } else if (MODE == G_FWD_DOWN) {
    float acc = 0.f;
    const float* w = W0 + (int64_t)g * f * d + n;
    for (int k = 0; k < f; ++k) acc = __builtin_fmaf(A[row * f + k], w[(int64_t)k * d], acc);
    if (a.bias0) acc += reinterpret_cast<const float*>(a.bias0)[(int64_t)g * d + n];
    reinterpret_cast<float*>(a.c0)[row * d + n] = acc;
  } else if (MODE == G_DGRAD_DOWN) {
    float dh = 0.f;
    const float* w = W0 + (int64_t)g * f * d + (int64_t)n * d;
    for (int k = 0; k < d; ++k) dh = __builtin_fmaf(A[row * d + k], w[k], dh);
    const float* gu = reinterpret_cast<const float*>(a.aux);
    const float gv = gu[row * 2 * f + n], uv = gu[row * 2 * f + f + n];
    float* dgu = reinterpret_cast<float*>(a.c0);
    act_grad(a, gv, uv, dh, dgu[row * 2 * f + n], dgu[row * 2 * f + f + n]);
  } else {  // G_DGRAD_GATEUP
    float acc = 0.f;
    const float* wg = W0 + (int64_t)g * d * f + (int64_t)n * f;
    const float* wu = W1 + (int64_t)g * d * f + (int64_t)n * f;
    for (int k = 0; k < f; ++k) acc = __builtin_fmaf(A[row * 2 * f + k], wg[k], acc);
    for (int k = 0; k < f; ++k) acc = __builtin_fmaf(A[row * 2 * f + f + k], wu[k], acc);
    reinterpret_cast<float*>(a.c0)[row * d + n] = acc;
  }
}

const int kGemmKernelId[6] = {K_GEMM_GATEUP_FWD, K_GEMM_DOWN_FWD, K_GEMM_DOWN_DGRAD,
                              K_GEMM_GATEUP_DGRAD, K_GEMM_DOWN_WGRAD, K_GEMM_GATEUP_WGRAD};
const char* kGemmName[6] = {"gemm_gateup_fwd", "gemm_down_fwd", "gemm_down_dgrad",
                            "gemm_gateup_dgrad", "gemm_down_wgrad", "gemm_gateup_wgrad"};
// Timing id of a launch: the caller's (the shared expert's and the auxiliary
// loss's dense passes have ids of their own), else the routed pass's.
template <int MODE>
int gemm_kernel_id(const GemmArgs& a) { return a.kid > 0 ? a.kid : kGemmKernelId[MODE]; }

// Tile shapes per pass, chosen by timing the whole layer at the Qwen3 shape
// (512 +- 33 rows per expert): 256 x 256 tiles, 8 wavefronts, 2 x 64-k or
// 4 x 32-k LDS stages.  Experts with fewer than 192 rows on average use
// 128 x 128 (with the ragged row blocks skipped, 256-row tiles win already at
// the DeepSeek-V3 shape's 256 rows per expert: 34.1 -> 30.1 ms per step).
using CfgWide = Cfg<256, 256, 2, 4, 2, 64>;    // wavefront tile 128 x 64
using CfgTall = Cfg<256, 256, 4, 2, 2, 64>;    // wavefront tile 64 x 128
using CfgTall32 = Cfg<256, 256, 4, 2, 3, 32>;  // 3 stages of 32 k (room for the 4 KB epilogue slots)
using CfgSmall = Cfg<128, 128, 2, 2, 2, 64>;
template <int MODE> struct GemmShape { using big = CfgTall32; };
template <> struct GemmShape<G_FWD_GATEUP> { using big = CfgWide; };
template <> struct GemmShape<G_FWD_DOWN> { using big = CfgWide; };
template <> struct GemmShape<G_DGRAD_DOWN> { using big = CfgTall; };
template <> struct GemmShape<G_DGRAD_GATEUP> { using big = CfgTall; };

// Persistent launch: one workgroup per CU (a multiple of 8, so that every
// XCD gets the same number), never more than the tiles' upper bound.
inline int cu_count() {
  static int n = 0;
  if (n == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess && hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
      n = v;
    else
      n = 256;
  }
  return n;
}

template <int MODE, class C, bool CL = false, bool FP8 = false>
int launch_bf16_persistent(const GemmArgs& a, hipStream_t s) {
  const int G = a.offsets ? a.ngroups : 1;
  const int nt = n_tiles<MODE, C::BN>(a.d, a.f);
  int64_t nb;
  if (is_wgrad<MODE>()) {
    nb = (int64_t)G * ((wgrad_m<MODE>(a.d, a.f) + C::BM - 1) / C::BM) * nt;
  } else {
    const int64_t mt = a.offsets ? (a.max_rows + (int64_t)G * (C::BM - 1)) / C::BM
                                 : (a.dense_rows + C::BM - 1) / C::BM;
    nb = mt * nt;
  }
  if (nb <= 0) return MOE_OK;
  // workgroups per CU that fit in LDS (stages, epilogue slots, tables)
  constexpr int kLdsPerBlock = C::LDS_BYTES + C::NW * (is_wgrad<MODE>() ? 4096 : 2048) + (is_wgrad<MODE>() ? 3 : 2) * 1024 + 64;
  constexpr int kOcc = (160 * 1024) / kLdsPerBlock > 0 ? (160 * 1024) / kLdsPerBlock : 1;
  const int64_t grid = std::min<int64_t>((cu_count() * kOcc / 8) * 8, (nb + 7) / 8 * 8);
  return launch(gemm_kernel_id<MODE>(a), s, kGemmName[MODE],
                [&] { gemm_bf16_persistent<MODE, C, CL, FP8><<<(int)grid, C::NT, 0, s>>>(a); });
}

template <int MODE>
int launch_mode(const GemmArgs& a, hipStream_t s) {
  if (a.fp8 && !(a.bf16 && !is_wgrad<MODE>()))
    return moe_set_error(MOE_ERR_UNSUPPORTED, "gemm: FP8 runs the bf16 forward and data-gradient passes only");
  if (a.accumulate && !is_wgrad<MODE>())
    return moe_set_error(MOE_ERR_INVALID_ARG, "gemm: accumulate applies to the weight-gradient passes only");
  if (a.bf16) {
    const int G = a.offsets ? a.ngroups : 1;
    const int64_t rows_per_group = a.offsets ? a.max_rows / G : a.dense_rows;
    if constexpr (!is_wgrad<MODE>()) {
      if (a.fp8) {
        // FP8: 2 x 4 wavefronts in every pass (the data-gradient passes ran
        // 9% faster than with the bf16 kernels' 4 x 2, Qwen3 shape)
        if constexpr (MODE == G_FWD_GATEUP || MODE == G_DGRAD_DOWN) {
          if (a.act == MOE_ACT_CLAMPED_GLU) {
            if (rows_per_group < 192) return launch_bf16_persistent<MODE, CfgSmall, true, true>(a, s);
            return launch_bf16_persistent<MODE, CfgWide, true, true>(a, s);
          }
        }
        if (rows_per_group < 192) return launch_bf16_persistent<MODE, CfgSmall, false, true>(a, s);
        return launch_bf16_persistent<MODE, CfgWide, false, true>(a, s);
      }
    }
    if constexpr (MODE == G_FWD_GATEUP || MODE == G_DGRAD_DOWN) {
      if (a.act == MOE_ACT_CLAMPED_GLU) {
        if (rows_per_group < 192) return launch_bf16_persistent<MODE, CfgSmall, true>(a, s);
        return launch_bf16_persistent<MODE, typename GemmShape<MODE>::big, true>(a, s);
      }
    }
    if (!is_wgrad<MODE>() && rows_per_group < 192) return launch_bf16_persistent<MODE, CfgSmall>(a, s);
    return launch_bf16_persistent<MODE, typename GemmShape<MODE>::big>(a, s);
  }
  constexpr bool wgrad = is_wgrad<MODE>();
  const int G = a.offsets ? a.ngroups : 1;
  int64_t nb;
  constexpr int TS = 16;
  if (wgrad) {
    const int Mfix = MODE == G_WGRAD_DOWN ? a.f : a.d;
    const int Nfix = MODE == G_WGRAD_DOWN ? a.d : 2 * a.f;
    nb = (int64_t)G * ((Mfix + TS - 1) / TS) * ((Nfix + TS - 1) / TS);
  } else {
    const int N = (MODE == G_FWD_GATEUP || MODE == G_DGRAD_DOWN) ? a.f : a.d;
    const int64_t mt = a.offsets ? (a.max_rows + (int64_t)G * (TS - 1)) / TS : (a.dense_rows + TS - 1) / TS;
    nb = mt * ((N + TS - 1) / TS);
  }
  if (nb <= 0) return MOE_OK;
  return launch(gemm_kernel_id<MODE>(a), s, kGemmName[MODE],
                [&] { gemm_f32_kernel<MODE><<<(int)nb, 256, 0, s>>>(a); });
}

}  // namespace

int launch_gemm(const GemmArgs& a, hipStream_t s) {
  switch (a.mode) {
    case G_FWD_GATEUP: return launch_mode<G_FWD_GATEUP>(a, s);
    case G_FWD_DOWN: return launch_mode<G_FWD_DOWN>(a, s);
    case G_DGRAD_DOWN: return launch_mode<G_DGRAD_DOWN>(a, s);
    case G_DGRAD_GATEUP: return launch_mode<G_DGRAD_GATEUP>(a, s);
    case G_WGRAD_DOWN: return launch_mode<G_WGRAD_DOWN>(a, s);
    case G_WGRAD_GATEUP: return launch_mode<G_WGRAD_GATEUP>(a, s);
  }
  return moe_set_error(MOE_ERR_INVALID_ARG, "gemm: unknown mode %d", a.mode);
}

}  // namespace moe
