// Block-wide exact selection helpers shared by the top-M selections (512-thread blocks).
#pragma once

#include "common.hpp"

namespace sr {

__device__ __forceinline__ uint32_t fkey(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int TOPM_NT = 512;
constexpr int TOPM_BINS = 2048;

// Suffix (exclusive, from the top) scan of per-thread counts over the block.
__device__ inline int block_suffix_excl(int v, int* sh) {
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int o = 1; o < TOPM_NT; o <<= 1) {
    int add = (tid + o < TOPM_NT) ? sh[tid + o] : 0;
    __syncthreads();
    sh[tid] += add;
    __syncthreads();
  }
  int incl = sh[tid];
  __syncthreads();
  return incl - v;
}
// Prefix (exclusive) scan of per-thread counts; also returns the total.
__device__ inline int block_prefix_excl(int v, int* sh, int* total) {
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int o = 1; o < TOPM_NT; o <<= 1) {
    int add = (tid >= o) ? sh[tid - o] : 0;
    __syncthreads();
    sh[tid] += add;
    __syncthreads();
  }
  int incl = sh[tid];
  *total = sh[TOPM_NT - 1];
  __syncthreads();
  return incl - v;
}

// Radix select over n order-preserving keys: after it, st.prefix is the key K* of the k-th largest
// element, st.rem the number of elements equal to K* that belong to the top k, st.cnt_eq how many equal
// K* in total. Called by the whole block.
struct RadixState {
  uint32_t prefix, pmask;
  int rem, cnt_eq;
};
template <class KeyAt>
__device__ void radix_kth(KeyAt key_at, int n, int k, int* hist, int* scan, RadixState& st) {
  const int tid = threadIdx.x;
  if (tid == 0) { st.prefix = 0; st.pmask = 0; st.rem = k; st.cnt_eq = 0; }
  const int shifts[3] = {21, 10, 0};
  const int bits[3] = {11, 11, 10};
  for (int pass = 0; pass < 3; ++pass) {
    for (int i = tid; i < TOPM_BINS; i += TOPM_NT) hist[i] = 0;
    __syncthreads();
    const uint32_t prefix = st.prefix, pmask = st.pmask;
    const int sh = shifts[pass];
    const uint32_t dmask = (1u << bits[pass]) - 1u;
    for (int i = tid; i < n; i += TOPM_NT) {
      const uint32_t kk = key_at(i);
      if ((kk & pmask) == prefix) atomicAdd(&hist[(kk >> sh) & dmask], 1);
    }
    __syncthreads();
    // thread t owns bins [nb*t, nb*t + nb); find the bin holding rank st.rem counted from the top
    const int nb = (1 << bits[pass]) / TOPM_NT;
    int local = 0;
    for (int j = 0; j < nb; ++j) local += hist[tid * nb + j];
    const int above = block_suffix_excl(local, scan);
    const int rem = st.rem;
    __syncthreads();
    if (above < rem && rem <= above + local) {
      int a = above;
      for (int j = nb - 1; j >= 0; --j) {
        const int c = hist[tid * nb + j];
        if (rem <= a + c) {
          st.prefix = prefix | ((uint32_t)(tid * nb + j) << sh);
          st.pmask = pmask | (dmask << sh);
          st.rem = rem - a;
          st.cnt_eq = c;
          break;
        }
        a += c;
      }
    }
    __syncthreads();
  }
}

}  // namespace sr
