// Grouped expert GEMMs: forward gate/up with the fused SwiGLU epilogue,
// forward down, the down data-gradient with the fused SwiGLU backward, the
// gate/up data-gradient, and both weight gradients (section 3.2: fused SwiGLU
// forward and backward kernels; wgrad kept as a separate pass so that it can
// be delayed).
//
// bf16 path (MFMA): one 256-thread workgroup computes a 128x128 output tile
// with 4 wavefronts in a 2x2 arrangement (64x64 each, 4x4 blocks of
// v_mfma_f32_16x16x32_bf16, float32 accumulators).  K advances 64 at a time
// through two LDS buffers; the next tile's global loads are in flight while
// the current one is multiplied.  Both operands sit in LDS as [row][64 k]
// with the 16-byte chunk index XOR-swizzled by ((row>>1) ^ (row>>3)) & 7, so
// that the MFMA fragment reads (16 rows, same chunk) and the transposing
// stores of MN-contiguous operands both spread over the 64 LDS banks.
// Operands that are contiguous along K are copied with 16-byte loads and
// stores; operands contiguous along M or N (the weights in the forward, both
// operands of the weight gradients) are loaded as 4 k-rows x 8 columns per
// thread and transposed in registers before the LDS store.
//
// Scheduling happens on the device from expert_offsets: a block derives the
// per-expert m-tile prefix in LDS and finds its (expert, m-tile, n-tile), so
// variable per-expert row counts need no host synchronisation; blocks beyond
// the real tile count exit.  Rows past an expert's end, columns past N and
// (for the weight gradients, whose K is the expert's row count) k past the
// end are zero-filled on load and not stored.  Block ids are remapped so that
// each XCD works on a contiguous range of tiles.
//
// fp32 path: a plain kernel, one thread per output (or output pair), for the
// fp32 workload; same modes, same epilogues.
#include "common.h"
#include "kernels.h"

namespace moe {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int TILE_ELEMS = 128 * BK;

__device__ __forceinline__ int swz(int r) { return ((r >> 1) ^ (r >> 3)) & 7; }
// element offset of 16-byte chunk c (0..7) of row r
__device__ __forceinline__ int lds_off(int r, int c) { return r * BK + ((c ^ swz(r)) << 3); }

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + __expf(-z)); }

// ---------------------------------------------------------------------------
// Tile decode
// ---------------------------------------------------------------------------
struct Tile {
  int g;          // expert
  int row_base;   // first row of the expert in the row-major activations
  int rows;       // rows of the expert (M for fwd/dgrad, K for wgrad)
  int m0, n0;     // tile origin in the output
  int ntile;      // n-tile index
  bool live;
};

template <int MODE>
__device__ __forceinline__ Tile decode_tile(const GemmArgs& a, int* pre, int* sbuf) {
  Tile t;
  constexpr bool wgrad = MODE == G_WGRAD_DOWN || MODE == G_WGRAD_GATEUP;
  const int nb = gridDim.x;
  const int lin = xcd_remap(blockIdx.x, nb);
  if (wgrad) {
    const int Mfix = MODE == G_WGRAD_DOWN ? a.f : a.d;
    const int Nfix = MODE == G_WGRAD_DOWN ? a.d : 2 * a.f;
    const int mt = (Mfix + BM - 1) / BM, nt = (Nfix + BN - 1) / BN;
    t.g = lin / (mt * nt);
    const int rem = lin - t.g * mt * nt;
    const int im = rem / nt;
    t.ntile = rem - im * nt;
    t.m0 = im * BM;
    t.n0 = t.ntile * BN;
    if (a.offsets) {
      t.row_base = a.offsets[t.g];
      t.rows = a.offsets[t.g + 1] - t.row_base;
    } else {
      t.row_base = 0;
      t.rows = (int)a.dense_rows;
    }
    t.live = t.g < (a.offsets ? a.ngroups : 1);
    return t;
  }
  int ntiles;
  if (MODE == G_FWD_GATEUP) ntiles = a.f / 64;
  else if (MODE == G_FWD_DOWN || MODE == G_DGRAD_GATEUP) ntiles = (a.d + BN - 1) / BN;
  else ntiles = (a.f + BN - 1) / BN;
  const int mt = lin / ntiles;
  t.ntile = lin - mt * ntiles;
  t.n0 = t.ntile * (MODE == G_FWD_GATEUP ? 64 : BN);
  if (!a.offsets) {
    t.g = 0;
    t.row_base = 0;
    t.rows = (int)a.dense_rows;
    t.m0 = mt * BM;
    t.live = t.m0 < t.rows;
    return t;
  }
  const int G = a.ngroups;
  int c = 0;
  if ((int)threadIdx.x < G) c = (a.offsets[threadIdx.x + 1] - a.offsets[threadIdx.x] + BM - 1) / BM;
  __shared__ int total;
  const int ex = block_scan_256(c, sbuf, &total);
  if ((int)threadIdx.x < G) pre[threadIdx.x] = ex;
  __syncthreads();
  t.live = mt < total;
  if (!t.live) return t;
  int lo = 0, hi = G - 1;  // last g with pre[g] <= mt (empty experts share a prefix: take the last)
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pre[mid] <= mt) lo = mid; else hi = mid - 1;
  }
  t.g = lo;
  t.row_base = a.offsets[lo];
  t.rows = a.offsets[lo + 1] - t.row_base;
  t.m0 = (mt - pre[lo]) * BM;
  return t;
}

// ---------------------------------------------------------------------------
// Operand loaders (bf16).  Each thread moves 4 x 16 bytes per 128x64 tile.
// ---------------------------------------------------------------------------

// K-contiguous source: row r of the tile starts at rowptr[i] (+ k0).
struct KLoader {
  const bf16_t* ptr[4];
  bool ok[4];
  int lds[4];
  uint4 reg[4];
  __device__ __forceinline__ void load(int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      reg[i] = ok[i] ? *reinterpret_cast<const uint4*>(ptr[i] + k0) : make_uint4(0, 0, 0, 0);
  }
  __device__ __forceinline__ void store(bf16_t* tile) {
#pragma unroll
    for (int i = 0; i < 4; ++i) *reinterpret_cast<uint4*>(tile + lds[i]) = reg[i];
  }
};

// MN-contiguous source [K][ld]: thread owns 8 columns (one 16-byte chunk)
// and 4 consecutive k rows of the tile; stores them transposed.
struct MNLoader {
  const bf16_t* col;   // element (k=0, this thread's first column), k rows ld apart
  int64_t ld;
  bool colok;
  int kbase;           // 4*kg: first k row of this thread inside the tile
  int klimit;          // rows valid (k < klimit), relative to the tile start
  int lds[8];          // LDS element offsets of columns c = 0..7 (+ k position)
  uint4 reg[4];
  __device__ __forceinline__ void load(int k0) {  // k0: tile start (relative)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int k = k0 + kbase + q;
      reg[q] = (colok && k < klimit) ? *reinterpret_cast<const uint4*>(col + (int64_t)k * ld)
                                     : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(bf16_t* tile) {
    const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&reg[0]);
    const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&reg[1]);
    const uint32_t* r2 = reinterpret_cast<const uint32_t*>(&reg[2]);
    const uint32_t* r3 = reinterpret_cast<const uint32_t*>(&reg[3]);
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int w = c >> 1;
      uint32_t lo, hi;
      if (c & 1) {
        lo = (r0[w] >> 16) | (r1[w] & 0xffff0000u);
        hi = (r2[w] >> 16) | (r3[w] & 0xffff0000u);
      } else {
        lo = (r0[w] & 0xffffu) | (r1[w] << 16);
        hi = (r2[w] & 0xffffu) | (r3[w] << 16);
      }
      *reinterpret_cast<uint2*>(tile + lds[c]) = make_uint2(lo, hi);
    }
  }
};

__device__ __forceinline__ void kloader_init(KLoader& L, int tid) {
  const int c = tid & 7;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = (tid >> 3) + 32 * i;
    L.lds[i] = lds_off(r, c);
  }
}

__device__ __forceinline__ void mnloader_init(MNLoader& L, int tid) {
  const int nc = tid & 15, kg = tid >> 4;
  L.kbase = 4 * kg;
#pragma unroll
  for (int c = 0; c < 8; ++c) L.lds[c] = lds_off(8 * nc + c, kg >> 1) + 4 * (kg & 1);
}

// ---------------------------------------------------------------------------
// The bf16 MFMA kernel
// ---------------------------------------------------------------------------
template <int MODE>
__global__ __launch_bounds__(256, 2) void gemm_bf16_kernel(GemmArgs a) {
  __shared__ __align__(16) bf16_t lds[2][2][TILE_ELEMS];
  __shared__ int pre[257];
  __shared__ int sbuf[256];
  constexpr bool wgrad = MODE == G_WGRAD_DOWN || MODE == G_WGRAD_GATEUP;

  const Tile tl = decode_tile<MODE>(a, pre, sbuf);
  if (!tl.live) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int d = a.d, f = a.f;
  const int g = tl.g;

  // problem extents
  int K, M, N;
  if (MODE == G_FWD_GATEUP) { K = d; M = tl.rows; N = f; }
  else if (MODE == G_FWD_DOWN) { K = f; M = tl.rows; N = d; }
  else if (MODE == G_DGRAD_DOWN) { K = d; M = tl.rows; N = f; }
  else if (MODE == G_DGRAD_GATEUP) { K = 2 * f; M = tl.rows; N = d; }
  else if (MODE == G_WGRAD_DOWN) { K = tl.rows; M = f; N = d; }
  else { K = tl.rows; M = d; N = 2 * f; }

  const bf16_t* A = reinterpret_cast<const bf16_t*>(a.a);
  const bf16_t* Bact = reinterpret_cast<const bf16_t*>(a.b);
  const bf16_t* W0 = reinterpret_cast<const bf16_t*>(a.w0);
  const bf16_t* W1 = reinterpret_cast<const bf16_t*>(a.w1);

  // ---- operand A
  KLoader la;
  MNLoader ma;
  if (!wgrad) {
    kloader_init(la, tid);
    const int lda = MODE == G_FWD_DOWN ? f : (MODE == G_DGRAD_GATEUP ? 2 * f : d);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = tl.m0 + (tid >> 3) + 32 * i;
      la.ok[i] = r < M;
      la.ptr[i] = A + (int64_t)(tl.row_base + (r < M ? r : 0)) * lda + 8 * (tid & 7);
    }
  } else {
    mnloader_init(ma, tid);
    const int lda = MODE == G_WGRAD_DOWN ? f : d;  // h rows [f] or x_perm rows [d]
    const int col = tl.m0 + 8 * (tid & 15);
    ma.colok = col < M;
    ma.col = A + (int64_t)tl.row_base * lda + (ma.colok ? col : 0);
    ma.ld = lda;
    ma.klimit = K;
  }
  // ---- operand B
  KLoader lb;
  MNLoader mb;
  const bf16_t* bk_gate = nullptr;  // DGRAD_GATEUP: per-row pointers into W_gate / W_up
  const bf16_t* bk_up = nullptr;
  if (MODE == G_FWD_GATEUP || MODE == G_FWD_DOWN) {
    mnloader_init(mb, tid);
    const int nc = tid & 15;
    if (MODE == G_FWD_GATEUP) {
      // tile columns: wave-column wn holds 32 gate then 32 up columns of the
      // same 32 j's; chunk nc -> j = n0 + 32*(nc/8) + 16*((nc%8)/2 % 2) + 8*(nc%2)
      const int q = nc & 7;
      const int j = tl.n0 + 32 * (nc >> 3) + 16 * ((q >> 1) & 1) + 8 * (q & 1);
      const bf16_t* W = (q >> 2) ? W1 : W0;
      mb.col = W + (int64_t)g * d * f + j;
      mb.ld = f;
      mb.colok = true;
    } else {
      const int n = tl.n0 + 8 * nc;
      mb.colok = n < N;
      mb.col = W0 + (int64_t)g * f * d + (mb.colok ? n : 0);
      mb.ld = d;
    }
    mb.klimit = K;
  } else if (MODE == G_DGRAD_DOWN || MODE == G_DGRAD_GATEUP) {
    kloader_init(lb, tid);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int n = tl.n0 + (tid >> 3) + 32 * i;
      lb.ok[i] = n < N;
      const int nn = n < N ? n : 0;
      if (MODE == G_DGRAD_DOWN)  // B[k=i][n=j] = W_down[g][j][i]
        lb.ptr[i] = W0 + (int64_t)g * f * d + (int64_t)nn * d + 8 * (tid & 7);
      else  // B[k=j][n=i] = W_gate[g][i][j] (k < f) or W_up[g][i][j-f]
        lb.ptr[i] = W0 + (int64_t)g * d * f + (int64_t)nn * f + 8 * (tid & 7);
    }
    if (MODE == G_DGRAD_GATEUP) {
      bk_gate = W0;
      bk_up = W1;
    }
  } else {
    mnloader_init(mb, tid);
    const int ldb = MODE == G_WGRAD_DOWN ? d : 2 * f;  // d_o rows or dgu rows
    const int n = tl.n0 + 8 * (tid & 15);
    mb.colok = n < N;
    mb.col = Bact + (int64_t)tl.row_base * ldb + (mb.colok ? n : 0);
    mb.ld = ldb;
    mb.klimit = K;
  }

  floatx4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // bias-gradient column sums (weight-gradient passes, first m-tile, wm == 0)
  const bool colsum = wgrad && a.db0 && tl.m0 == 0 && wm == 0;
  float bsum[4] = {0.f, 0.f, 0.f, 0.f};

  auto load_tile = [&](int k0) {
    if (!wgrad) la.load(k0); else ma.load(k0);
    if (MODE == G_DGRAD_GATEUP) {
      // whole k-tile lies in W_gate (k0 < f) or in W_up; f % 64 == 0
      const int64_t shift = (k0 < f) ? (int64_t)k0 : (int64_t)(k0 - f) + (bk_up - bk_gate);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        lb.reg[i] = lb.ok[i] ? *reinterpret_cast<const uint4*>(lb.ptr[i] + shift) : make_uint4(0, 0, 0, 0);
    } else if (MODE == G_DGRAD_DOWN) {
      lb.load(k0);
    } else {
      mb.load(k0);
    }
  };
  auto store_tile = [&](int buf) {
    if (!wgrad) la.store(lds[buf][0]); else ma.store(lds[buf][0]);
    if (MODE == G_DGRAD_DOWN || MODE == G_DGRAD_GATEUP) lb.store(lds[buf][1]); else mb.store(lds[buf][1]);
  };

  const int nk = (K + BK - 1) / BK;
  if (nk > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();
  const int r16 = lane & 15, kq = lane >> 4;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_tile((kt + 1) * BK);
    const bf16_t* As = lds[cur][0];
    const bf16_t* Bs = lds[cur][1];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        af[i] = *reinterpret_cast<const bf16x8*>(As + lds_off(wm * 64 + i * 16 + r16, ks * 4 + kq));
        bfr[i] = *reinterpret_cast<const bf16x8*>(Bs + lds_off(wn * 64 + i * 16 + r16, ks * 4 + kq));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
      if (colsum) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint4 u = __builtin_bit_cast(uint4, bfr[j]);
          const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int q = 0; q < 4; ++q)
            bsum[j] += __uint_as_float(w4[q] << 16) + __uint_as_float(w4[q] & 0xffff0000u);
        }
      }
    }
    if (kt + 1 < nk) store_tile(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue
  const int rq = 4 * (lane >> 4);  // row offset of this lane's 4 values in a 16x16 block
  if (MODE == G_FWD_GATEUP) {
    bf16_t* gu = reinterpret_cast<bf16_t*>(a.c0);
    bf16_t* h = reinterpret_cast<bf16_t*>(a.c1);
    const bf16_t* bgp = reinterpret_cast<const bf16_t*>(a.bias0);
    const bf16_t* bup = reinterpret_cast<const bf16_t*>(a.bias1);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = tl.n0 + wn * 32 + j * 16 + r16;
      const float bg = bgp ? bf2f(bgp[(int64_t)g * f + col]) : 0.f;
      const float bu = bup ? bf2f(bup[(int64_t)g * f + col]) : 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int m = tl.m0 + wm * 64 + i * 16 + rq + v;
          if (m < M) {
            const int64_t row = tl.row_base + m;
            const float gv = acc[i][j][v] + bg;
            const float uv = acc[i][j + 2][v] + bu;
            gu[row * 2 * f + col] = f2bf(gv);
            gu[row * 2 * f + f + col] = f2bf(uv);
            h[row * f + col] = f2bf(silu_f(gv) * uv);
          }
        }
    }
  } else if (MODE == G_FWD_DOWN || MODE == G_DGRAD_GATEUP) {
    bf16_t* out = reinterpret_cast<bf16_t*>(a.c0);
    const bf16_t* bdp = MODE == G_FWD_DOWN ? reinterpret_cast<const bf16_t*>(a.bias0) : nullptr;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = tl.n0 + wn * 64 + j * 16 + r16;
      if (col >= N) continue;
      const float bd = bdp ? bf2f(bdp[(int64_t)g * d + col]) : 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int m = tl.m0 + wm * 64 + i * 16 + rq + v;
          if (m < M) out[(int64_t)(tl.row_base + m) * N + col] = f2bf(acc[i][j][v] + bd);
        }
    }
  } else if (MODE == G_DGRAD_DOWN) {
    const bf16_t* gu = reinterpret_cast<const bf16_t*>(a.aux);
    bf16_t* dgu = reinterpret_cast<bf16_t*>(a.c0);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = tl.n0 + wn * 64 + j * 16 + r16;
      if (col >= N) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int m = tl.m0 + wm * 64 + i * 16 + rq + v;
          if (m < M) {
            const int64_t row = tl.row_base + m;
            const float gv = bf2f(gu[row * 2 * f + col]);
            const float uv = bf2f(gu[row * 2 * f + f + col]);
            const float sg = 1.0f / (1.0f + __expf(-gv));
            const float dh = acc[i][j][v];
            dgu[row * 2 * f + col] = f2bf(dh * uv * sg * (1.0f + gv * (1.0f - sg)));
            dgu[row * 2 * f + f + col] = f2bf(dh * gv * sg);
          }
        }
    }
  } else {
    // weight gradients of expert g: [M][N] at c0 (+ c1 for the up half)
    bf16_t* c0 = reinterpret_cast<bf16_t*>(a.c0);
    bf16_t* c1 = reinterpret_cast<bf16_t*>(a.c1);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = tl.n0 + wn * 64 + j * 16 + r16;
      if (col >= N) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int m = tl.m0 + wm * 64 + i * 16 + rq + v;
          if (m >= M) continue;
          if (MODE == G_WGRAD_DOWN) {
            c0[((int64_t)g * f + m) * d + col] = f2bf(acc[i][j][v]);
          } else if (col < f) {
            c0[((int64_t)g * d + m) * f + col] = f2bf(acc[i][j][v]);
          } else {
            c1[((int64_t)g * d + m) * f + (col - f)] = f2bf(acc[i][j][v]);
          }
        }
    }
    if (colsum) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float v = bsum[j];
        v += __shfl_xor(v, 16, 64);
        v += __shfl_xor(v, 32, 64);
        const int col = tl.n0 + wn * 64 + j * 16 + r16;
        if (lane < 16 && col < N) {
          if (MODE == G_WGRAD_DOWN) {
            reinterpret_cast<bf16_t*>(a.db0)[(int64_t)g * d + col] = f2bf(v);
          } else if (col < f) {
            reinterpret_cast<bf16_t*>(a.db0)[(int64_t)g * f + col] = f2bf(v);
          } else {
            reinterpret_cast<bf16_t*>(a.db1)[(int64_t)g * f + col - f] = f2bf(v);
          }
        }
      }
    }
  }
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
    if (MODE == G_WGRAD_DOWN) {
      c0[((int64_t)g * f + m) * d + n] = acc;
      if (colsum) reinterpret_cast<float*>(a.db0)[(int64_t)g * d + n] = bs;
    } else if (n < f) {
      c0[((int64_t)g * d + m) * f + n] = acc;
      if (colsum) reinterpret_cast<float*>(a.db0)[(int64_t)g * f + n] = bs;
    } else {
      c1[((int64_t)g * d + m) * f + n - f] = acc;
      if (colsum) reinterpret_cast<float*>(a.db1)[(int64_t)g * f + n - f] = bs;
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
    reinterpret_cast<float*>(a.c1)[row * f + n] = silu_f(ag) * au;
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
    const float sg = 1.0f / (1.0f + __expf(-gv));
    float* dgu = reinterpret_cast<float*>(a.c0);
    dgu[row * 2 * f + n] = dh * uv * sg * (1.0f + gv * (1.0f - sg));
    dgu[row * 2 * f + f + n] = dh * gv * sg;
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

template <int MODE>
int launch_mode(const GemmArgs& a, hipStream_t s) {
  constexpr bool wgrad = MODE == G_WGRAD_DOWN || MODE == G_WGRAD_GATEUP;
  const int G = a.offsets ? a.ngroups : 1;
  int64_t nb;
  if (a.bf16) {
    if (wgrad) {
      const int Mfix = MODE == G_WGRAD_DOWN ? a.f : a.d;
      const int Nfix = MODE == G_WGRAD_DOWN ? a.d : 2 * a.f;
      nb = (int64_t)G * ((Mfix + BM - 1) / BM) * ((Nfix + BN - 1) / BN);
    } else {
      int ntiles;
      if (MODE == G_FWD_GATEUP) ntiles = a.f / 64;
      else if (MODE == G_FWD_DOWN || MODE == G_DGRAD_GATEUP) ntiles = (a.d + BN - 1) / BN;
      else ntiles = (a.f + BN - 1) / BN;
      const int64_t mt = a.offsets ? (a.max_rows + (int64_t)G * (BM - 1)) / BM : (a.dense_rows + BM - 1) / BM;
      nb = mt * ntiles;
    }
    if (nb <= 0) return MOE_OK;
    return launch(kGemmKernelId[MODE], s, kGemmName[MODE],
                  [&] { gemm_bf16_kernel<MODE><<<(int)nb, 256, 0, s>>>(a); });
  }
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
  return launch(kGemmKernelId[MODE], s, kGemmName[MODE],
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
