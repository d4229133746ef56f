// Shared device/host helpers of the gfx950 speculative-verification kernels.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "specroll.h"

namespace sr {

typedef uint16_t bf16_t;  // bfloat16 storage (bit pattern)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }

// float -> bfloat16 bits, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint32_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// 16 bytes per lane from global memory straight into LDS (global_load_lds_dwordx4): lane l's bytes land at
// ldst + 16 * l, so one wave instruction fills 1 KB; ldst must be the same for every lane of the wave.
__device__ __forceinline__ void lds_dma16(const void* gsrc, unsigned char* ldst) {
  __builtin_amdgcn_global_load_lds((const void*)gsrc, (__attribute__((address_space(3))) void*)ldst, 16, 0, 0);
}

// The same transfer issued as inline assembly, which the compiler does not track: it then inserts no
// waits of its own for it, and the caller must wait (s_waitcnt vmcnt) before the bytes are read.
__device__ __forceinline__ void lds_dma16_manual(const void* gsrc, unsigned char* ldst) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)ldst);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(gsrc), "s"(l)
               : "memory", "m0");
}

// The same transfer from a uniform base (SGPR pair) plus a 32-bit per-lane byte offset; ldst_u32 is the
// wave-uniform LDS byte address of the 1 KB destination.
__device__ __forceinline__ void lds_dma16_sv(uint32_t voff, const void* sbase, uint32_t ldst_u32) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase),
               "s"(ldst_u32)
               : "memory", "m0");
}

// workgroup barrier ordering LDS only: this wave's LDS operations complete, global memory operations may
// still be in flight (unlike __syncthreads, which also waits for them)
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// wait until at most N of this wave's vector memory operations (LDS DMA included) are outstanding
template <int N> __device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Element access for the two storage types.
template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float* p, size_t i) { return p[i]; }
  static __device__ __forceinline__ void store(float* p, size_t i, float v) { p[i] = v; }
};
template <> struct Elem<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t* p, size_t i) { return bf2f(p[i]); }
  static __device__ __forceinline__ void store(bf16_t* p, size_t i, float v) { p[i] = (bf16_t)f2bf(v); }
};

__device__ __forceinline__ float warp_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
// Wave-wide max / sum of fp32 values without LDS traffic: DPP exchanges inside each row of 16 lanes
// (pairs, quads, mirrored halves, mirrored rows), then the four row results are read through scalar
// registers. Every lane receives the result.
template <int CTRL> __device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float wave_max_f32(float v) {
  v = fmaxf(v, dpp_f32<0xB1>(v));     // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp_f32<0x4E>(v));     // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp_f32<0x141>(v));    // row_half_mirror
  v = fmaxf(v, dpp_f32<0x140>(v));    // row_mirror
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fmaxf(fmaxf(a, b), fmaxf(c, d));
}
__device__ __forceinline__ float wave_sum_f32(float v) {
  v += dpp_f32<0xB1>(v);
  v += dpp_f32<0x4E>(v);
  v += dpp_f32<0x141>(v);
  v += dpp_f32<0x140>(v);
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (a + b) + (c + d);
}
// Sums over the wave of N values per lane (N = 4 or 8), reduce-scattered: lane l returns the total of
// value j = l / (64 / N) (set in j), summed as pairs over lanes l ^ 32 (v_permlane32_swap, which trades
// the two 32-lane halves of two registers), l ^ 16 and, for N = 8, l ^ 8 (ds_bpermute), then over the low
// lane bits by DPP. Whole wave active.
template <int N>
__device__ __forceinline__ float wave_sum_scatter(const float (&a)[N], int& j) {
  static_assert(N == 4 || N == 8, "4 or 8 values");
  const int lane = threadIdx.x & 63;
  float b[N / 2];
#pragma unroll
  for (int k = 0; k < N / 2; ++k) {
    // lanes 0-31: value k over l, l+32; lanes 32-63: value k + N/2 over l-32, l
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a[k]), __float_as_uint(a[k + N / 2]), false, false);
    b[k] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  float v;
  {
    const bool hi16 = (lane & 16) != 0;
    float c[N / 4];
#pragma unroll
    for (int k = 0; k < N / 4; ++k) {
      const float keep = hi16 ? b[k + N / 4] : b[k], send = hi16 ? b[k] : b[k + N / 4];
      c[k] = keep + __shfl_xor(send, 16, 64);
    }
    if constexpr (N == 4) {
      v = c[0];
    } else {
      const bool hi8 = (lane & 8) != 0;
      const float keep = hi8 ? c[1] : c[0], send = hi8 ? c[0] : c[1];
      v = keep + __shfl_xor(send, 8, 64);
    }
  }
  // the lanes of one value now differ in their low 6 - log2(N) bits
  v += dpp_f32<0xB1>(v);                         // quad_perm [1,0,3,2]: lanes i, i ^ 1
  v += dpp_f32<0x4E>(v);                         // quad_perm [2,3,0,1]: lanes i, i ^ 2
  v += dpp_f32<0x141>(v);                        // row_half_mirror: quads 0 and 1 of each 8 lanes
  if constexpr (N == 4) v += dpp_f32<0x140>(v);  // row_mirror: halves of each 16 lanes
  j = lane / (64 / N);
  return v;
}
template <int CTRL> __device__ __forceinline__ double dpp_f64(double v) {
  const long long u = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_update_dpp((int)u, (int)u, CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp((int)(u >> 32), (int)(u >> 32), CTRL, 0xf, 0xf, false);
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}
__device__ __forceinline__ double readlane_f64(double v, int l) {
  const long long u = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane((int)u, l), hi = __builtin_amdgcn_readlane((int)(u >> 32), l);
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}
// float64 wave max / sum with the same exchange pattern (whole wave active)
__device__ __forceinline__ double wave_max_f64(double v) {
  v = fmax(v, dpp_f64<0xB1>(v));
  v = fmax(v, dpp_f64<0x4E>(v));
  v = fmax(v, dpp_f64<0x141>(v));
  v = fmax(v, dpp_f64<0x140>(v));
  return fmax(fmax(readlane_f64(v, 0), readlane_f64(v, 16)), fmax(readlane_f64(v, 32), readlane_f64(v, 48)));
}
__device__ __forceinline__ double wave_sum_f64(double v) {
  v += dpp_f64<0xB1>(v);
  v += dpp_f64<0x4E>(v);
  v += dpp_f64<0x141>(v);
  v += dpp_f64<0x140>(v);
  return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}
__device__ __forceinline__ double warp_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double warp_max_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ double warp_min_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmin(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ int warp_min_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ int warp_max_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ int warp_sum_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Topology of one trajectory's tree, held in LDS. Validates parents[0] == -1 and
// 0 <= parents[c] < c; computes depth, child count and slot index (1-based) of every
// node. Must be called by the whole block; returns false (uniformly) when invalid.
template <int MAXT>
struct TreeLds {
  int parent[MAXT];
  int depth[MAXT];
  int nkids[MAXT];
  int slot[MAXT];
  int bad;
};

template <int MAXT>
__device__ bool tree_setup(TreeLds<MAXT>& t, const int32_t* parents_b, int T) {
  const int tid = threadIdx.x;
  // the first parent of each thread is loaded before the barrier, in flight with the caller's own loads
  const int p0 = tid < T ? parents_b[tid] : 0;
  if (tid == 0) t.bad = 0;
  __syncthreads();
  for (int c = tid; c < T; c += blockDim.x) {
    int p = c == tid ? p0 : parents_b[c];
    if ((c == 0 && p != -1) || (c > 0 && (p < 0 || p >= c))) atomicOr(&t.bad, 1);
    t.parent[c] = p;
  }
  __syncthreads();
  if (t.bad) return false;
  for (int c = tid; c < T; c += blockDim.x) {
    int d = 0;
    for (int p = t.parent[c]; p >= 0; p = t.parent[p]) ++d;  // terminates: parents strictly decrease
    t.depth[c] = d;
    int n = 0, s = 0;
    for (int k = 1; k < T; ++k) {
      if (t.parent[k] == c) ++n;
      if (k < c && c > 0 && t.parent[k] == t.parent[c]) ++s;
    }
    t.nkids[c] = n;
    t.slot[c] = (c == 0) ? 0 : s + 1;
  }
  __syncthreads();
  return true;
}

}  // namespace sr

// ----------------------------------------------------------------------------- host side
namespace sr {

void set_error(const char* fmt, ...);
sr_status hip_fail(hipError_t e, const char* what);

// Launch bookkeeping: every kernel launch goes through here so the timing hook can
// bracket it with events and launch errors are reported uniformly.
struct LaunchGuard {
  const char* name;
  hipStream_t stream;
  int slot;                      // >= 0: this launch is timed
  hipEvent_t ev_start, ev_stop;  // recorded by the dispatch itself (no separate event packets)
  LaunchGuard(const char* n, hipStream_t s);
  sr_status done();  // counts the timed launch and checks the launch
};

}  // namespace sr

#define SR_LAUNCH(NAME, KERNEL, GRID, BLOCK, SHMEM, STREAM, ...)                                      \
  do {                                                                                                 \
    ::sr::LaunchGuard _g((NAME), (STREAM));                                                            \
    if (_g.slot >= 0)                                                                                  \
      hipExtLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, _g.ev_start, _g.ev_stop, 0, __VA_ARGS__); \
    else                                                                                               \
      hipLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, __VA_ARGS__);                             \
    sr_status _st = _g.done();                                                                         \
    if (_st != SR_OK) return _st;                                                                      \
  } while (0)
