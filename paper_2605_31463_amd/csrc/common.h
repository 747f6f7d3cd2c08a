// Internal helpers shared by the libmoe kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/moe.h"

namespace moe {

// Kernel numbering for moe_timing_select / moe_kernel_name.
enum KernelId {
  K_ROUTE = 0,
  K_COUNT_ZERO,
  K_HIST,
  K_SCAN,
  K_SCATTER,
  K_GEMM_GATEUP_FWD,
  K_GEMM_DOWN_FWD,
  K_COMBINE_FWD,
  K_COMBINE_BWD,
  K_ROUTE_DL,
  K_ROUTE_DWR_PARTIAL,
  K_ROUTE_DWR_REDUCE,
  K_WR_TRANSPOSE,
  K_ROUTE_DX,
  K_GEMM_DOWN_DGRAD,
  K_GEMM_GATEUP_DGRAD,
  K_GEMM_DOWN_WGRAD,
  K_GEMM_GATEUP_WGRAD,
  K_UNPERMUTE,
  K_RANK,
  K_WR_SPLIT,
  K_ROUTE_SELECT,
  K_AUX_STATS,
  K_AUX_GRAD,
  K_AUX_DWR,
  K_ZC_PARAM_PARTIAL,
  K_ZC_PARAM_REDUCE,
  K_THRESHOLD_GRAD,
  K_AUX_PARTIAL_ROWS,
  K_QUANT_ROWS,
  K_WEIGHT_QUANT,
  // the shared expert's dense passes (same kernels as the routed passes)
  K_GEMM_SH_GATEUP_FWD,
  K_GEMM_SH_DOWN_FWD,
  K_GEMM_SH_DOWN_DGRAD,
  K_GEMM_SH_GATEUP_DGRAD,
  K_GEMM_SH_DOWN_WGRAD,
  K_GEMM_SH_GATEUP_WGRAD,
  // the auxiliary loss's router products (dense dx, chunked dW_r)
  K_GEMM_AUX_DX,
  K_GEMM_AUX_DWR,
  K_NUM_KERNELS
};

const char* kernel_name(int id);

// Records the start / stop events around one launch when that kernel id is
// selected for timing.  Returns true when events were recorded.
void timing_before(int id, hipStream_t s);
void timing_after(int id, hipStream_t s);

// Launch helper: times the launch if selected and checks hipGetLastError.
int check_launch(const char* what);

template <class F>
inline int launch(int id, hipStream_t s, const char* what, F&& f) {
  timing_before(id, s);
  f();
  timing_after(id, s);
  return check_launch(what);
}

// ---------------------------------------------------------------------------
// element helpers
// ---------------------------------------------------------------------------
typedef uint16_t bf16_t;  // bfloat16 bit pattern

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ __forceinline__ bf16_t f2bf(float f) {
  // v_cvt_pk_bf16_f32: round to nearest even
  __bf16 h = (__bf16)f;
  return __builtin_bit_cast(bf16_t, h);
}

template <class T> struct Elem;
template <> struct Elem<float> {
  __device__ __forceinline__ static float load(const float* p, int64_t i) { return p[i]; }
  __device__ __forceinline__ static void store(float* p, int64_t i, float v) { p[i] = v; }
  static constexpr int kVec = 4;  // elements per 16 bytes
};
template <> struct Elem<bf16_t> {
  __device__ __forceinline__ static float load(const bf16_t* p, int64_t i) { return bf2f(p[i]); }
  __device__ __forceinline__ static void store(bf16_t* p, int64_t i, float v) { p[i] = f2bf(v); }
  static constexpr int kVec = 8;
};

// 16-byte vectors of activations as float arrays.
template <class T> struct Vec16;
template <> struct Vec16<float> {
  static constexpr int N = 4;
  __device__ __forceinline__ static void load(const float* p, float* out) {
    float4 v = *reinterpret_cast<const float4*>(p);
    out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
  }
  __device__ __forceinline__ static void store(float* p, const float* in) {
    *reinterpret_cast<float4*>(p) = make_float4(in[0], in[1], in[2], in[3]);
  }
};
template <> struct Vec16<bf16_t> {
  static constexpr int N = 8;
  __device__ __forceinline__ static void load(const bf16_t* p, float* out) {
    uint4 v = *reinterpret_cast<const uint4*>(p);
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      out[2 * i] = __uint_as_float(w[i] << 16);
      out[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  __device__ __forceinline__ static void store(bf16_t* p, const float* in) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (uint32_t)f2bf(in[2 * i]) | ((uint32_t)f2bf(in[2 * i + 1]) << 16);
    *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
  }
};

__device__ __forceinline__ float sigmoidf_(float z) { return 1.0f / (1.0f + __expf(-z)); }

// OCP FP8 E4M3 codes (round to nearest even) of four float32 values, clamped
// to +-448 first, packed little-endian into one dword.
__device__ __forceinline__ float e4m3_clamp(float v) { return fminf(fmaxf(v, -448.f), 448.f); }
__device__ __forceinline__ uint32_t e4m3x4(float a, float b, float c, float d) {
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(a), e4m3_clamp(b), 0, false);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(c), e4m3_clamp(d), lo, true);
}
// Row / column quantisation scale of the largest magnitude amax: values are
// multiplied by 448 / amax before rounding and the products carry amax / 448
// (an all-zero row or column: 1 and 1).
__device__ __forceinline__ float e4m3_inv(float amax) { return amax > 0.f ? 448.f / amax : 1.f; }
__device__ __forceinline__ float e4m3_scale(float amax) { return amax > 0.f ? amax / 448.f : 1.f; }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}

// Wave-wide float sum (64 lanes), result in every lane.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// Exclusive scan of one int per thread over the first 256 threads of the
// block (all threads of the block must call it).  buf: 256 ints of LDS.
// Returns the exclusive prefix; *total (LDS) receives the sum.
__device__ __forceinline__ int block_scan_256(int v, int* buf, int* total) {
  const int tid = threadIdx.x;
  if (tid < 256) buf[tid] = v;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    int t = (tid < 256 && tid >= off) ? buf[tid - off] : 0;
    __syncthreads();
    if (tid < 256) buf[tid] += t;
    __syncthreads();
  }
  const int incl = tid < 256 ? buf[tid] : 0;
  if (tid == 255) *total = incl;
  __syncthreads();
  return incl - v;
}

// Blocks are dealt to the 8 XCDs round-robin (block b on XCD b % 8); give
// each XCD a contiguous range of logical tile ids so that tiles sharing
// operands share that XCD's L2.
__device__ __forceinline__ int xcd_remap(int b, int nblocks) {
  const int xcd = b & 7, idx = b >> 3;
  const int per = nblocks >> 3, rem = nblocks & 7;
  return xcd * per + (xcd < rem ? xcd : rem) + idx;
}

// ---------------------------------------------------------------------------
// Global -> LDS copies without registers (buffer_load_dwordx4 ... lds): one
// instruction moves 64 lanes x 16 bytes into 1 KB of LDS at the wave-uniform
// address in M0.  The copies are issued from inline assembly and counted by
// hand with s_waitcnt vmcnt, so that several stages can be in flight while
// the compiler schedules LDS reads freely.  A buffer descriptor bounds every
// copy: reads past its range return zeros and touch no memory.
// ---------------------------------------------------------------------------
typedef int int32x4_t __attribute__((ext_vector_type(4)));
constexpr int RSRC_FLAGS = 0x00020000;

// Buffer descriptor (raw buffer, no stride) over [p, p + bytes), in SGPRs.
__device__ __forceinline__ int32x4_t make_rsrc(const void* p, int64_t bytes) {
  const uint64_t b = (uint64_t)p;
  int32x4_t r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)b);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(b >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane((int)(uint32_t)bytes);
  r[3] = RSRC_FLAGS;
  return r;
}

template <class T>
__device__ __forceinline__ uint32_t lds_addr(const T* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const __attribute__((address_space(3))) T*)p);
}

__device__ __forceinline__ void dma16(const int32x4_t& r, uint32_t lds, uint32_t voff, uint32_t soff) {
  int32x4_t rs;  // wave-uniform by construction; keeps the operand in SGPRs
#pragma unroll
  for (int q = 0; q < 4; ++q) rs[q] = __builtin_amdgcn_readfirstlane(r[q]);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(rs),
                  "s"(__builtin_amdgcn_readfirstlane(soff)) : "memory");
}

// s_waitcnt vmcnt(n), expcnt and lgkmcnt left free
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (((N >> 4) & 3) << 14) | 0x0F70);
}

}  // namespace moe

// Host-side error reporting (api.hip).
int moe_set_error(int status, const char* fmt, ...);
