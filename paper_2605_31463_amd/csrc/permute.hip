// Token-to-expert permutation: the single-GPU form of the framework's token
// scatter (section 3.2, "fused ... EP token scatter").
//
//   hist     one block per 256 tokens counts how many of its (token, slot)
//            pairs chose each expert;
//   scan     per expert, exclusive prefix of the block counts (each block's
//            base inside the expert) and the exclusive scan over experts
//            (expert_offsets);
//   rank     one block per 256 tokens ranks its pairs inside each expert in
//            ascending token order from per-wave 64-bit membership masks
//            (popcount below the lane) and writes row_of / token_of;
//   copy     one wavefront per token reads its x row once from HBM and writes
//            it to the token's k rows with 16-byte vector loads and stores
//            (rows of the FFN experts only: a zero-computation expert's rows
//            just list its tokens).
// No atomics touch the row layout, so the permutation is the stable counting
// sort by (expert, token) on every run.
#include <mutex>

#include "common.h"
#include "kernels.h"

namespace moe {

// Scratch of the allocation-free permutation entry point: the per-block
// expert histograms [nblk][E_pool] int32 live in this fixed device array
// instead of a caller's workspace.  Every GPU the library runs on holds its
// own copy until the process ends; calls on one GPU share it (hist_kernel
// writes every entry a call reads, so nothing carries over between calls).
static __device__ __align__(256) int32_t scratch[kPermScratchBytes / sizeof(int32_t)];

int permute_scratch(size_t need, int32_t** out) {
  if (need > kPermScratchBytes)
    return moe_set_error(MOE_ERR_UNSUPPORTED,
                         "the allocation-free permutation needs %zu bytes of scratch, above its fixed %zu "
                         "(per-block histograms: ceil(T/256) * E_pool * 4 bytes)",
                         need, kPermScratchBytes);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return moe_set_error(MOE_ERR_HIP, "permute scratch: no usable current device (%d)", dev);
  // the device address of this GPU's copy of the array, looked up once per
  // device with that device current (the host-side name is not an address)
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return moe_set_error(MOE_ERR_HIP, "permute scratch: hipGetSymbolAddress: %s", hipGetErrorString(e));
    addr[dev] = p;
  }
  *out = static_cast<int32_t*>(addr[dev]);
  return MOE_OK;
}

namespace {

__global__ __launch_bounds__(256) void hist_kernel(const int32_t* __restrict__ idx, int64_t T, int k,
                                                   int E, int32_t* __restrict__ hist) {
  __shared__ int cnt[256];
  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += 256) cnt[e] = 0;
  __syncthreads();
  const int64_t t = (int64_t)blockIdx.x * PERM_TB + tid;
  if (t < T) {
    for (int s = 0; s < k; ++s) {
      const int e = idx[t * k + s];
      if ((unsigned)e < (unsigned)E) atomicAdd(&cnt[e], 1);  // out-of-range ids are dropped
    }
  }
  __syncthreads();
  for (int e = tid; e < E; e += 256) hist[(int64_t)blockIdx.x * E + e] = cnt[e];
}

// One block of 1024 threads: thread (e, p) scans a contiguous range of
// blocks of expert e; the parts are combined through LDS.
__global__ __launch_bounds__(1024) void scan_kernel(int32_t* __restrict__ hist, int64_t nblk, int E,
                                                    int EP, int32_t* __restrict__ offsets) {
  __shared__ int part[1024];
  __shared__ int tot[257];
  const int tid = threadIdx.x;
  const int P = 1024 / EP;
  const int e = tid % EP;
  const int p = tid / EP;
  const int64_t chunk = (nblk + P - 1) / P;
  const int64_t b0 = p * chunk;
  const int64_t b1 = b0 + chunk < nblk ? b0 + chunk : nblk;
  int sum = 0;
  if (e < E) {
    for (int64_t b = b0; b < b1; b += 8) {
      int v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = (b + q < b1) ? hist[(b + q) * E + e] : 0;
#pragma unroll
      for (int q = 0; q < 8; ++q) sum += v[q];
    }
  }
  part[p * EP + e] = sum;
  __syncthreads();
  int pre = 0;
  for (int q = 0; q < p; ++q) pre += part[q * EP + e];
  if (e < E) {
    for (int64_t b = b0; b < b1; b += 8) {
      int v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = (b + q < b1) ? hist[(b + q) * E + e] : 0;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if (b + q < b1) hist[(b + q) * E + e] = pre;
        pre += v[q];
      }
    }
  }
  if (p == 0) {
    int t = 0;
    for (int q = 0; q < P; ++q) t += part[q * EP + e];
    if (e < E) tot[e] = t;
  }
  __syncthreads();
  __shared__ int sbuf[256];
  __shared__ int total;
  const int ex = block_scan_256(tid < E ? tot[tid] : 0, sbuf, &total);
  if (tid < E) offsets[tid] = ex;
  if (tid == 0) offsets[E] = total;
}

// Ranks each (token, slot) pair of a 256-token block inside its expert and
// writes row_of / token_of.
__global__ __launch_bounds__(256) void rank_kernel(PermArgs a) {
  __shared__ unsigned long long mask[4][256];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int E = a.E, k = a.k;
  for (int i = tid; i < 4 * 256; i += 256) (&mask[0][0])[i] = 0ull;
  __syncthreads();
  const int64_t blk = blockIdx.x;
  const int64_t t = blk * PERM_TB + tid;
  const bool live = t < a.T;
  int ex[16];
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    ex[s] = -1;
    if (s < k && live) {
      const int e = a.topk_idx[t * k + s];
      if ((unsigned)e < (unsigned)E) {
        ex[s] = e;
        atomicOr(&mask[wave][e], 1ull << lane);
      }
    }
  }
  __syncthreads();
  const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
  for (int s = 0; s < 16; ++s) {
    if (s < k && live && ex[s] < 0) {
      a.row_of[t * k + s] = -1;
    } else if (s < k && live) {
      const int e = ex[s];
      int rank = __popcll(mask[wave][e] & below);
      for (int w = 0; w < wave; ++w) rank += __popcll(mask[w][e]);
      const int row = a.offsets[e] + a.hist[blk * E + e] + rank;
      a.row_of[t * k + s] = row;
      a.token_of[row] = (int32_t)(t * k + s);
    }
  }
}

// Row copy: one wavefront per token reads the x row once (16-byte vector
// loads, 2 per lane in flight) and writes it to the token's k rows.
template <class XT>
__global__ __launch_bounds__(256) void permute_copy_kernel(PermArgs a) {
  constexpr int V = Vec16<XT>::N;
  constexpr int CPL = 4;
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)__builtin_amdgcn_readfirstlane((int)(blockIdx.x * 4 + (threadIdx.x >> 6)));
  if (t >= a.T) return;
  const int k = a.k;
  const int nch = a.d / V;
  const XT* x = reinterpret_cast<const XT*>(a.x) + t * a.d;
  XT* xp = reinterpret_cast<XT*>(a.x_perm);
  // FP8 forward: the token's E4M3 scale from a first pass over its row
  float inv = 1.f, scale = 1.f;
  if (a.xq) {
    float m = 0.f;
    for (int c = lane; c < nch; c += 64) {
      float v[V];
      Vec16<XT>::load(x + (int64_t)c * V, v);
#pragma unroll
      for (int q = 0; q < V; ++q) m = fmaxf(m, fabsf(v[q]));
    }
    m = wave_max(m);
    inv = e4m3_inv(m);
    scale = e4m3_scale(m);
  }
  // rows at or past the FFN experts' end belong to zero-computation experts
  // (no activations): not written
  const int64_t r_end = a.offsets[a.E_rows];
  // the first chunks' loads are issued before the row look-up, so their
  // latency overlaps its dependent loads
  uint4 v[CPL];
  auto load_chunks = [&](int c0) {
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
      const int c = c0 + j * 64 + lane;
      if (c < nch) v[j] = *reinterpret_cast<const uint4*>(x + (int64_t)c * V);
    }
  };
  load_chunks(0);
  int64_t rows[16];
  if (a.maps_ready) {
    // the slot's row: its expert's offset, the base of its 256-token block,
    // the counts of the block's earlier 16-token selection blocks and its
    // rank inside its own (lane s holds slot s)
    int myrow = -1;
    if (lane < k) {
      const int e = a.topk_idx[t * k + lane];
      if ((unsigned)e < (unsigned)a.E) {
        const int64_t b = t / PERM_TB;
        const int q = (int)((t % PERM_TB) >> 4);
        const int32_t* c16 = a.cnt16 + (b * (PERM_TB / 16)) * a.E + e;
        // all loads issued at once: rows past q repeat row q (it exists) and
        // are not counted
        int cv[PERM_TB / 16 - 1];
#pragma unroll
        for (int u = 0; u < PERM_TB / 16 - 1; ++u) cv[u] = c16[(int64_t)min(u, q) * a.E];
        int pre = 0;
#pragma unroll
        for (int u = 0; u < PERM_TB / 16 - 1; ++u) pre += u < q ? cv[u] : 0;
        myrow = a.offsets[e] + a.hist[b * a.E + e] + pre + a.row_of[t * k + lane];
        a.row_of[t * k + lane] = myrow;
        a.token_of[myrow] = (int32_t)(t * k + lane);
      }
    }
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      rows[s] = s < k ? __builtin_amdgcn_readlane(myrow, s) : -1;
      if (rows[s] >= r_end) rows[s] = -1;
    }
  } else {
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      rows[s] = s < k ? a.row_of[t * k + s] : -1;
      if (rows[s] >= r_end) rows[s] = -1;
    }
  }
  for (int c0 = 0; c0 < nch; c0 += 64 * CPL) {
    if (c0) load_chunks(c0);
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      if (s >= k) break;
      if (rows[s] < 0) continue;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int c = c0 + j * 64 + lane;
        if (c < nch) *reinterpret_cast<uint4*>(xp + rows[s] * a.d + (int64_t)c * V) = v[j];
      }
      if (a.xq) {
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
          const int c = c0 + j * 64 + lane;
          if (c >= nch) continue;
          float f8[V];
          Vec16<XT>::load(reinterpret_cast<const XT*>(&v[j]), f8);
          if constexpr (V == 8) {
            const uint2 codes = make_uint2(e4m3x4(f8[0] * inv, f8[1] * inv, f8[2] * inv, f8[3] * inv),
                                           e4m3x4(f8[4] * inv, f8[5] * inv, f8[6] * inv, f8[7] * inv));
            *reinterpret_cast<uint2*>(a.xq + rows[s] * a.d + (int64_t)c * V) = codes;
          }
        }
        if (lane == 0 && c0 == 0) a.sx[rows[s]] = scale;
      }
    }
  }
}

}  // namespace

int launch_permute(const PermArgs& a, hipStream_t s) {
  const int64_t nblk = perm_blocks(a.T);
  int st;
  if (a.maps_ready) {  // the route's selection built the maps' inputs; the copy finishes them
    if (nblk == 0) return MOE_OK;
    const int ncopy = (int)((a.T + 3) / 4);
    if (a.bf16)
      return launch(K_SCATTER, s, "scatter", [&] { permute_copy_kernel<bf16_t><<<ncopy, 256, 0, s>>>(a); });
    return launch(K_SCATTER, s, "scatter", [&] { permute_copy_kernel<float><<<ncopy, 256, 0, s>>>(a); });
  }
  if (nblk > 0) {
    st = launch(K_HIST, s, "hist", [&] { hist_kernel<<<nblk, 256, 0, s>>>(a.topk_idx, a.T, a.k, a.E, a.hist); });
    if (st) return st;
  }
  int EP = 1;
  while (EP < a.E) EP <<= 1;
  st = launch(K_SCAN, s, "scan", [&] { scan_kernel<<<1, 1024, 0, s>>>(a.hist, nblk, a.E, EP, a.offsets); });
  if (st) return st;
  if (nblk == 0) return MOE_OK;
  st = launch(K_RANK, s, "rank", [&] { rank_kernel<<<nblk, 256, 0, s>>>(a); });
  if (st) return st;
  const int ncopy = (int)((a.T + 3) / 4);
  if (a.bf16)
    return launch(K_SCATTER, s, "scatter", [&] { permute_copy_kernel<bf16_t><<<ncopy, 256, 0, s>>>(a); });
  return launch(K_SCATTER, s, "scatter", [&] { permute_copy_kernel<float><<<ncopy, 256, 0, s>>>(a); });
}

}  // namespace moe
