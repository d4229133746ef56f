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

// Inclusive prefix sum of per-thread counts over the block, and the block total: within each wave by DPP
// (row shifts 1, 2, 4, 8, then the three lower rows' totals), across the waves through sh (one entry per
// wave) and one barrier. Integer sums: the same result in any order. Ends with a barrier, so sh may be
// reused at once.
__device__ inline int block_incl_scan(int v, int* sh, int* total) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int NWV = TOPM_NT / 64;
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, true);   // row_shr:1 (lanes past the row read 0)
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, true);   // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, true);   // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, true);   // row_shr:8
  const int r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31),
            r2 = __builtin_amdgcn_readlane(v, 47), r3 = __builtin_amdgcn_readlane(v, 63);
  const int row = lane >> 4;
  v += (row > 0 ? r0 : 0) + (row > 1 ? r1 : 0) + (row > 2 ? r2 : 0);
  if (lane == 0) sh[wave] = r0 + r1 + r2 + r3;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NWV; ++w) {
    const int t = sh[w];
    before += w < wave ? t : 0;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return before + v;
}
// Suffix (exclusive, from the top) scan of per-thread counts over the block.
__device__ inline int block_suffix_excl(int v, int* sh) {
  int total;
  const int incl = block_incl_scan(v, sh, &total);
  return total - incl;
}
// Prefix (exclusive) scan of per-thread counts; also returns the total.
__device__ inline int block_prefix_excl(int v, int* sh, int* total) {
  return block_incl_scan(v, sh, total) - v;
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
