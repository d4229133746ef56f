// Proposal step on gfx950: Reflex-corrected LayerNorm, the head residual blocks and
// the shared-vocabulary projection as MFMA GEMMs, per-row top-M selection, and the
// ordered without-replacement draft-tree build.
//
// Paper: Sec. 3.2 Eq. (heads); App. C "Future-token proposer" (z = h + SiLU(A LN(h) + b),
// logits through the target's vocabulary projection); App. B.1 Eq. (slotq), Eq. (childlist).
#include <math.h>

#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "select.hpp"

namespace sr {

// ============================================================================ clip + LayerNorm
// One block per trajectory: x = h + corr * min(1, c/||corr||) (active rows), n = LN(x).
constexpr int CLN_MAXE = 32;   // row elements per thread held in registers (d <= 8192)
template <typename T>
__global__ __launch_bounds__(256) void k_clip_ln(const T* __restrict__ hidden, const float* __restrict__ corr,
                                                 const uint8_t* __restrict__ active, int d, float clip_norm,
                                                 float eps, float* __restrict__ x_out, T* __restrict__ n_out) {
  const int b = blockIdx.x, tid = threadIdx.x;
  __shared__ float red[8];
  __shared__ float bc;
  auto block_sum = [&](float v) -> float {
    v = warp_sum(v);
    if ((tid & 63) == 0) red[tid >> 6] = v;
    __syncthreads();
    if (tid == 0) {
      float s = 0.f;
      for (int w = 0; w < (int)(blockDim.x >> 6); ++w) s += red[w];
      bc = s;
    }
    __syncthreads();
    float r = bc;
    __syncthreads();
    return r;
  };
  const size_t row = (size_t)b * d;
  float scale = 0.f;
  bool act = corr != nullptr && (active == nullptr || active[b] != 0);
  if constexpr (sizeof(T) == 2) {
    if (d % 8 == 0 && d <= 256 * CLN_MAXE && blockDim.x == 256) {
      // bf16 rows: 8 consecutive elements per 16-byte access, the row in registers; one reduction for
      // ||corr||^2, sum h and sum corr (the mean of x = h + s corr follows from them), one for the
      // centred squares
      constexpr int NCK = CLN_MAXE / 8;        // 8-element chunks per thread
      float hv[NCK][8], cv[NCK][8];
      __shared__ float red3[8][3];
      float ss = 0.f, sh = 0.f, sc = 0.f;
#pragma unroll
      for (int k = 0; k < NCK; ++k) {
        const int i0 = (tid + k * 256) * 8;
        if (i0 < d) {
          const u32x4 hw = *(const u32x4*)(hidden + row + i0);
#pragma unroll
          for (int e = 0; e < 8; ++e) hv[k][e] = bf2f((e & 1) ? (hw[e >> 1] >> 16) : (hw[e >> 1] & 0xffffu));
          if (act) {
            const f32x4 c0 = *(const f32x4*)(corr + row + i0), c1 = *(const f32x4*)(corr + row + i0 + 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) { cv[k][e] = c0[e]; cv[k][e + 4] = c1[e]; }
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) cv[k][e] = 0.f;
          }
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) hv[k][e] = cv[k][e] = 0.f;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) { ss += cv[k][e] * cv[k][e]; sh += hv[k][e]; sc += cv[k][e]; }
      }
      ss = warp_sum(ss); sh = warp_sum(sh); sc = warp_sum(sc);
      if ((tid & 63) == 0) { red3[tid >> 6][0] = ss; red3[tid >> 6][1] = sh; red3[tid >> 6][2] = sc; }
      __syncthreads();
      float tss = 0.f, tsh = 0.f, tsc = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) { tss += red3[w][0]; tsh += red3[w][1]; tsc += red3[w][2]; }
      if (act) {
        const float nrm = sqrtf(tss);
        scale = nrm > 0.f ? fminf(1.f, clip_norm / nrm) : 0.f;
      }
      const float mean = (tsh + scale * tsc) / (float)d;
      float q = 0.f;
#pragma unroll
      for (int k = 0; k < NCK; ++k) {
        const int i0 = (tid + k * 256) * 8;
        if (i0 < d) {
          f32x4 x0, x1;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            hv[k][e] = hv[k][e] + (act ? scale * cv[k][e] : 0.f);
            const float v = hv[k][e] - mean;
            q += v * v;
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) { x0[e] = hv[k][e]; x1[e] = hv[k][e + 4]; }
          *(f32x4*)(x_out + row + i0) = x0;
          *(f32x4*)(x_out + row + i0 + 4) = x1;
        }
      }
      q = warp_sum(q);
      if ((tid & 63) == 0) red3[4 + (tid >> 6)][0] = q;
      __syncthreads();
      const float var = (red3[4][0] + red3[5][0] + red3[6][0] + red3[7][0]) / (float)d;
      const float rs = 1.f / sqrtf(var + eps);
#pragma unroll
      for (int k = 0; k < NCK; ++k) {
        const int i0 = (tid + k * 256) * 8;
        if (i0 < d) {
          u32x4 nw;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            nw[e] = (uint32_t)f2bf((hv[k][2 * e] - mean) * rs) | ((uint32_t)f2bf((hv[k][2 * e + 1] - mean) * rs) << 16);
          *(u32x4*)(n_out + row + i0) = nw;
        }
      }
      return;
    }
  }
  if (d <= 256 * CLN_MAXE && blockDim.x == 256) {
    // the row stays in registers: one round trip for the loads, the same sums in the same order
    float hv[CLN_MAXE], cv[CLN_MAXE];
#pragma unroll
    for (int k = 0; k < CLN_MAXE; ++k) {
      const int i = tid + k * 256;
      hv[k] = i < d ? Elem<T>::load(hidden, row + i) : 0.f;
      cv[k] = (act && i < d) ? corr[row + i] : 0.f;
    }
    if (act) {
      float ss = 0.f;
#pragma unroll
      for (int k = 0; k < CLN_MAXE; ++k) ss += cv[k] * cv[k];
      const float nrm = sqrtf(block_sum(ss));
      scale = nrm > 0.f ? fminf(1.f, clip_norm / nrm) : 0.f;
    }
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < CLN_MAXE; ++k) {
      const int i = tid + k * 256;
      hv[k] = hv[k] + (act ? scale * cv[k] : 0.f);
      if (i < d) {
        x_out[row + i] = hv[k];
        s += hv[k];
      }
    }
    const float mean = block_sum(s) / (float)d;
    float q = 0.f;
#pragma unroll
    for (int k = 0; k < CLN_MAXE; ++k)
      if (tid + k * 256 < d) { const float v = hv[k] - mean; q += v * v; }
    const float var = block_sum(q) / (float)d;
    const float rs = 1.f / sqrtf(var + eps);
#pragma unroll
    for (int k = 0; k < CLN_MAXE; ++k) {
      const int i = tid + k * 256;
      if (i < d) Elem<T>::store(n_out, row + i, (hv[k] - mean) * rs);
    }
    return;
  }
  if (act) {
    float ss = 0.f;
    for (int i = tid; i < d; i += blockDim.x) { float v = corr[row + i]; ss += v * v; }
    float nrm = sqrtf(block_sum(ss));
    scale = nrm > 0.f ? fminf(1.f, clip_norm / nrm) : 0.f;
  }
  float s = 0.f;
  for (int i = tid; i < d; i += blockDim.x) {
    float v = Elem<T>::load(hidden, row + i) + (act ? scale * corr[row + i] : 0.f);
    x_out[row + i] = v;
    s += v;
  }
  const float mean = block_sum(s) / (float)d;
  float q = 0.f;
  for (int i = tid; i < d; i += blockDim.x) { float v = x_out[row + i] - mean; q += v * v; }
  const float var = block_sum(q) / (float)d;
  const float rs = 1.f / sqrtf(var + eps);
  for (int i = tid; i < d; i += blockDim.x) Elem<T>::store(n_out, row + i, (x_out[row + i] - mean) * rs);
}

// ============================================================================ MFMA GEMM
// C[m][n] = sum_k A[m][k] * B[n][k]  (both operands K-contiguous), handed to an epilogue.
// bf16: v_mfma_f32_32x32x16_bf16 (8 elements per lane per slot); fp32: v_mfma_f32_32x32x2_f32.
template <typename T> struct Mma;
template <> struct Mma<bf16_t> {
  static constexpr int KPL = 8;             // k elements a lane supplies per MFMA
  typedef u32x4 frag;                       // 8 x bf16
  static __device__ __forceinline__ frag load(const bf16_t* p) { return *(const u32x4*)p; }
  static __device__ __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                   c, 0, 0, 0);
  }
};
template <> struct Mma<float> {
  static constexpr int KPL = 1;
  typedef float frag;
  static __device__ __forceinline__ frag load(const float* p) { return *p; }
  static __device__ __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

// Epilogue of the head GEMM: z[b][h][j] = x[b][j] + SiLU(acc + bias[h*d + j]), rounded to T.
template <typename T>
struct EpiHead {
  const T* bias; const float* x; T* z; int d, H;
  static constexpr bool kGroupMax = false;
  static constexpr bool kTrans = false;
  __device__ __forceinline__ void group_max(int, int, float) const {}
  __device__ __forceinline__ void store4(int, int, f32x4) const {}
  __device__ __forceinline__ void operator()(int m, int n, float acc) const {
    const int h = n / d, j = n - h * d;
    const float v = acc + Elem<T>::load(bias, n);
    const float sv = v / (1.f + expf(-v));
    Elem<T>::store(z, ((size_t)m * H + h) * d + j, x[(size_t)m * d + j] + sv);
  }
};
// Epilogue of the vocabulary GEMM: fp32 logits[m][n].
struct EpiLogits {
  float* out; int N;
  __device__ __forceinline__ void operator()(int m, int n, float acc) const { out[(size_t)m * N + n] = acc; }
};

template <typename T, int BM, int BN, int BK, int WGM, int WGN, class Epi>
__global__ __launch_bounds__(WGM * WGN * 64) void k_gemm(const T* __restrict__ A, const T* __restrict__ B,
                                                         int M, int N, int K, Epi epi) {
  constexpr int NT = WGM * WGN * 64;
  constexpr int VEC = 16 / sizeof(T);        // elements per 16-byte vector
  constexpr int PAD = VEC;                   // one vector of padding per LDS row
  constexpr int LDK = BK + PAD;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int KPL = Mma<T>::KPL, KSTEP = 2 * KPL;
  constexpr int AV = BM * BK / VEC, BV = BN * BK / VEC;   // vectors per tile
  constexpr int AVT = (AV + NT - 1) / NT, BVT = (BV + NT - 1) / NT;
  static_assert(BK % KSTEP == 0 && BK % VEC == 0, "tile");

  __shared__ __attribute__((aligned(16))) T As[BM * LDK];
  __shared__ __attribute__((aligned(16))) T Bs[BN * LDK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;

  u32x4 ra[AVT], rb[BVT];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < AVT; ++i) {
      int v = tid + i * NT;
      int r = v / (BK / VEC), c = (v % (BK / VEC)) * VEC;
      u32x4 z = {0, 0, 0, 0};
      if (v < AV && m0 + r < M) z = *(const u32x4*)(A + (size_t)(m0 + r) * K + k0 + c);
      ra[i] = z;
    }
#pragma unroll
    for (int i = 0; i < BVT; ++i) {
      int v = tid + i * NT;
      int r = v / (BK / VEC), c = (v % (BK / VEC)) * VEC;
      u32x4 z = {0, 0, 0, 0};
      if (v < BV && n0 + r < N) z = *(const u32x4*)(B + (size_t)(n0 + r) * K + k0 + c);
      rb[i] = z;
    }
  };
  auto lstore = [&]() {
#pragma unroll
    for (int i = 0; i < AVT; ++i) {
      int v = tid + i * NT;
      if (v < AV) *(u32x4*)(As + (v / (BK / VEC)) * LDK + (v % (BK / VEC)) * VEC) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BVT; ++i) {
      int v = tid + i * NT;
      if (v < BV) *(u32x4*)(Bs + (v / (BK / VEC)) * LDK + (v % (BK / VEC)) * VEC) = rb[i];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x16){};

  gload(0);
  for (int k0 = 0; k0 < K; k0 += BK) {
    __syncthreads();
    lstore();
    __syncthreads();
    if (k0 + BK < K) gload(k0 + BK);
#pragma unroll
    for (int ks = 0; ks < BK; ks += KSTEP) {
      const int kk = ks + (lane >> 5) * KPL;
      typename Mma<T>::frag fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) fa[i] = Mma<T>::load(As + (wm * WTM + i * 32 + (lane & 31)) * LDK + kk);
#pragma unroll
      for (int j = 0; j < TN; ++j) fb[j] = Mma<T>::load(Bs + (wn * WTN + j * 32 + (lane & 31)) * LDK + kk);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = Mma<T>::mma(fa[i], fb[j], acc[i][j]);
    }
  }
  // output layout of a 32x32 tile: lane column l%32, register r -> row 8*(r/4) + 4*(l/32) + r%4
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + wn * WTN + j * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * WTM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (m < M && n < N) epi(m, n, acc[i][j][r]);
      }
    }
}

// ============================================================================ bf16 GEMM, direct-to-LDS
// C[m][n] = sum_k A[m][k] * B[n][k] for bf16 operands (both K-contiguous). Tiles stream from global
// memory straight into LDS (global_load_lds_dwordx4) through a STAGES-deep ring: the MFMA operand
// fragments of step ks+1 are read into registers between the two halves of step ks's MFMAs (one barrier
// per K-step), and right after that barrier the slot of step ks (whose fragments are in registers) is
// refilled with step ks+STAGES, so STAGES-1 steps are in flight. In LDS a tile row of
// BK elements is CPR 16-byte chunks; chunk c of row r is stored at position c ^ gemm_swz<CPR>(r): a
// 16-byte LDS read serves eight lanes (128 bytes) per cycle, and the eight rows that one such group of
// the 32x32x16 operand reads touches then fall on distinct 16-byte bank groups. Blocks are mapped so that the
// M-tiles sharing one N-tile of B run on the same XCD at the same time (B is read from HBM once and hits
// in that XCD's L2 for the others).
// Epilogue of the vocabulary GEMM: fp32 logits[m][n] plus, per row, the max over each 64-column group
// (the top-M selection scans only groups whose max can reach the M-th largest value). It takes the
// transposed accumulator layout (a lane owns one row and runs of four consecutive columns), so a group
// max needs one cross-lane exchange; the logits leave through LDS as row-contiguous 16-byte stores.
// Requires N % 4 == 0.
struct EpiLogitsMax {
  float* out; float* gmax; int N, ngroups;
  static constexpr bool kGroupMax = true;
  static constexpr bool kTrans = true;
  __device__ __forceinline__ void store4(int m, int n, f32x4 v) const { *(f32x4*)(out + (size_t)m * N + n) = v; }
  __device__ __forceinline__ void group_max(int m, int grp, float v) const {
    if (grp < ngroups) gmax[(size_t)m * ngroups + grp] = v;   // a tile's last wave may lie past N
  }
};

// wait until at most `ahead` stages of this wave's DMA (LPS transfers each) are outstanding, then meet the
// block; ahead in [0, MAXA] (the vmcnt immediate must be a constant)
template <int LPS, int MAXA>
__device__ __forceinline__ void dma_stage_sync(int ahead) {
  if constexpr (MAXA > 0) {
    if (ahead >= MAXA) {
      asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(MAXA * LPS) : "memory");
      return;
    }
    dma_stage_sync<LPS, MAXA - 1>(ahead);
  } else {
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  }
}

template <int CPR> __device__ __forceinline__ int gemm_swz(int r) {
  static_assert(CPR == 2 || CPR == 4 || CPR == 8, "rows of 32, 64 or 128 bytes");
  constexpr int SH = CPR == 8 ? 0 : CPR == 4 ? 1 : 2;   // rows r and r + 8/CPR share bank groups
  return (r >> SH) & (CPR - 1);
}

// Output of a transposed accumulator block (lane owns row m0w + 32 i + l%32; register r of tile j holds
// column n0w + 32 j + 8 (r/4) + 4 (l/32) + r%4): the 64-column group maxima, then the logits. Stored straight
// from registers, each 16-byte store instruction would touch 64 rows (64 cache lines); instead the wave stages
// its 32 rows of one tile row in its own LDS area stg (32 rows of WTN*4 + 16 bytes: the padding puts the 16
// lanes of a quarter-wave on 16 distinct bank groups) and stores them back with WTN/4 consecutive lanes per
// row. One wave; the caller makes sure no other wave still reads stg.
template <int TM, int TN, int WTN, class Epi>
__device__ __forceinline__ void epi_trans(const f32x16 (&acc)[TM][TN], unsigned char* stg, int m0w, int n0w, int M,
                                          int N, const Epi& epi) {
  static_assert(!Epi::kGroupMax || WTN % 64 == 0, "whole 64-column groups per wave");
  constexpr int RS = WTN * 4 + 16;              // staged row stride in bytes
  constexpr int LPR = WTN / 4;                  // lanes per staged row on the way out
  static_assert(64 % LPR == 0, "whole rows per store instruction");
  const int lane = threadIdx.x & 63, fr = lane & 31, fh = lane >> 5;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int mb = m0w + i * 32, m = mb + fr;
#pragma unroll
    for (int g = 0; g < (TN + 1) / 2; ++g) {   // 64-column group g of this wave: tiles 2g, 2g+1
      float gm = -INFINITY;
#pragma unroll
      for (int j = 2 * g; j < 2 * g + 2 && j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = j * 32 + 8 * q + 4 * fh;
          const f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
          *(f32x4*)(stg + fr * RS + c * 4) = v;
          if (n0w + c < N) gm = fmaxf(gm, fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])));
        }
      if constexpr (Epi::kGroupMax) {
        gm = fmaxf(gm, __shfl_xor(gm, 32, 64));
        if (fh == 0 && m < M) epi.group_max(m, n0w / 64 + g, gm);
      }
    }
    // this wave's own LDS writes above precede its reads below (one wave, in order)
#pragma unroll
    for (int rr = 0; rr < 32; rr += 64 / LPR) {
      const int row = rr + lane / LPR, c = (lane % LPR) * 4;
      const f32x4 v = *(const f32x4*)(stg + row * RS + c * 4);
      const int n = n0w + c;
      if (mb + row < M && n < N) epi.store4(mb + row, n, v);
    }
  }
}

template <int BM, int BN, int BK, int WGM, int WGN, int STAGES, class Epi>
__global__ __launch_bounds__(WGM * WGN * 64) void k_gemm_dl(const bf16_t* __restrict__ A,
                                                            const bf16_t* __restrict__ B, int M, int N, int K,
                                                            int tiles_m, int tiles_n, Epi epi) {
  constexpr int NW = WGM * WGN;
  constexpr int ROWB = BK * 2;                 // bytes per LDS row
  constexpr int CPR = ROWB / 16;               // 16-byte chunks per row
  constexpr int RPB = 1024 / ROWB;             // rows per 1 KB DMA block
  constexpr int A_BYTES = BM * ROWB, B_BYTES = BN * ROWB;
  constexpr int A_BLK = A_BYTES / 1024, B_BLK = B_BYTES / 1024;
  constexpr int LPS = (A_BLK + B_BLK) / NW;    // DMA instructions per wave per K-step
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  static_assert((A_BLK + B_BLK) % NW == 0 && A_BLK % NW == 0, "DMA blocks must split evenly over the waves");
  static_assert(BK == 32 || BK == 64, "tile");
  static_assert(STAGES >= 3, "ring of at least three stages");
  static_assert((STAGES - 1) * LPS <= 63, "the stages in flight must fit the vmcnt counter");
  __shared__ __attribute__((aligned(1024))) unsigned char lds[STAGES][A_BYTES + B_BYTES];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  // XCD-aware block -> (mt, nt)
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int mt = local % tiles_m, nt = (local / tiles_m) * 8 + xcd;
  if (nt >= tiles_n) return;
  const int m0 = mt * BM, n0 = nt * BN;
  const int nk = K / BK;

  // per-lane DMA source pointers for this wave's blocks (rows past M or N re-read the last row)
  const unsigned char* srcA[A_BLK / NW];
  const unsigned char* srcB[B_BLK / NW];
#pragma unroll
  for (int j = 0; j < A_BLK / NW; ++j) {
    const int blk = wave + j * NW;
    const int r = blk * RPB + lane / CPR, pos = lane % CPR;
    const int c = pos ^ gemm_swz<CPR>(r);
    srcA[j] = (const unsigned char*)(A + (size_t)min(m0 + r, M - 1) * K) + c * 16;
  }
#pragma unroll
  for (int j = 0; j < B_BLK / NW; ++j) {
    const int blk = wave + j * NW;
    const int r = blk * RPB + lane / CPR, pos = lane % CPR;
    const int c = pos ^ gemm_swz<CPR>(r);
    srcB[j] = (const unsigned char*)(B + (size_t)min(n0 + r, N - 1) * K) + c * 16;
  }
  // the transfers are untracked by the compiler: every wait on them below is explicit
  auto issue = [&](int ks) {
    unsigned char* dst = lds[ks % STAGES];
    const size_t koff = (size_t)ks * ROWB;
#pragma unroll
    for (int j = 0; j < A_BLK / NW; ++j) lds_dma16_manual(srcA[j] + koff, dst + (wave + j * NW) * 1024);
#pragma unroll
    for (int j = 0; j < B_BLK / NW; ++j) lds_dma16_manual(srcB[j] + koff, dst + A_BYTES + (wave + j * NW) * 1024);
  };
  // stage ks has landed for the whole block (the stages issued after it, up to ks+STAGES-2, may still be in
  // flight) and every wave's LDS reads are done
  auto sync = [&](int ks) { dma_stage_sync<LPS, STAGES - 2>(min(STAGES - 2, nk - 1 - ks)); };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x16){};

  // fragments: lane reads row (l%32) of a 32-row group at chunk 2*kk + l/32 (swizzled)
  const int fr = lane & 31, fh = lane >> 5;
  struct Frags { u32x4 a[BK / 16][TM], b[BK / 16][TN]; };
  auto load = [&](int ks, Frags& f) {
    const unsigned char* As = lds[ks % STAGES];
    const unsigned char* Bs = As + A_BYTES;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int c = 2 * kk + fh;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * WTM + i * 32 + fr;
        f.a[kk][i] = *(const u32x4*)(As + r * ROWB + ((c ^ gemm_swz<CPR>(r)) * 16));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * WTN + j * 32 + fr;
        f.b[kk][j] = *(const u32x4*)(Bs + r * ROWB + ((c ^ gemm_swz<CPR>(r)) * 16));
      }
    }
  };
  auto mma = [&](const Frags& f, int kk) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        if constexpr (Epi::kTrans)   // C^T tile: lane <-> row m, registers <-> columns n
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, f.b[kk][j]),
                                                              __builtin_bit_cast(bf16x8, f.a[kk][i]), acc[i][j], 0, 0, 0);
        else                         // C tile: lane <-> column n, registers <-> rows m
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, f.a[kk][i]),
                                                              __builtin_bit_cast(bf16x8, f.b[kk][j]), acc[i][j], 0, 0, 0);
  };
  // K-step ks: half of its MFMAs; wait for stage ks+1 and meet the block (every wave is done reading stage
  // ks); refill stage ks's slot with step ks+STAGES; read step ks+1's fragments; the other half
  auto step = [&](int ks, const Frags& cur, Frags& nxt) {
#pragma unroll
    for (int kk = 0; kk < BK / 32; ++kk) mma(cur, kk);
    if (ks + 1 < nk) {
      sync(ks + 1);
      if (ks + STAGES < nk) issue(ks + STAGES);
      load(ks + 1, nxt);
    }
#pragma unroll
    for (int kk = BK / 32; kk < BK / 16; ++kk) mma(cur, kk);
  };
#pragma unroll
  for (int t = 0; t < STAGES; ++t)
    if (t < nk) issue(t);
  dma_stage_sync<LPS, STAGES - 1>(min(STAGES - 1, nk - 1));   // stage 0 landed
  Frags fa_, fb_;
  load(0, fa_);
  for (int ks = 0; ks < nk; ks += 2) {
    step(ks, fa_, fb_);
    if (ks + 1 < nk) step(ks + 1, fb_, fa_);
  }

  if constexpr (Epi::kTrans) {
    static_assert(NW * 32 * (WTN * 4 + 16) <= STAGES * (A_BYTES + B_BYTES), "staging fits the ring");
    __syncthreads();                              // every wave has read its last fragments from the ring
    epi_trans<TM, TN, WTN>(acc, &lds[0][0] + wave * 32 * (WTN * 4 + 16), m0 + wm * WTM, n0 + wn * WTN, M, N, epi);
  } else {
    // element stores (lane column l%32, register r -> row 8*(r/4) + 4*(l/32) + r%4)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = n0 + wn * WTN + j * 32 + fr;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + wm * WTM + i * 32 + 8 * (r >> 2) + 4 * fh + (r & 3);
          if (m < M && n < N) epi(m, n, acc[i][j][r]);
        }
      }
  }
}

// ============================================================================ bf16 GEMM, quarter tiles
// C^T tiles of 256 x 256 for the vocabulary projection (M = B*H > 128), four waves in 2 x 2, each owning a
// 128 x 128 quarter as 4 x 4 MFMA tiles of 32 x 32: half the LDS operand reads per MFMA of the 128 x 64
// quarters of eight waves, with the 256 accumulator registers of a wave in AGPRs (one wave per SIMD). The
// operands stream into a STAGES-deep ring of 32-element K-steps (direct-to-LDS, as k_gemm_dl); the fragments
// of one 16-deep K-slice are read while the MFMAs of the previous slice run, and each wave's eight DMA
// transfers per step are spread one per four MFMAs over two slices. One barrier per K-step, between its two
// slices. Per-phase cycle counts (s_memtime) of a 7B-shaped run: 719 cycles for the first slice, 79 at the
// barrier, 599 for the second, against 512 per slice of MFMA work; issued back to back after the barrier the
// transfers had cost ~600 cycles per step.
// ring depth of the quarter-tile GEMM: 4 (128 KB) measured within 2 % of 3 and 5 at the 7B shape
#ifndef SR_GQ_STAGES
#define SR_GQ_STAGES 4
#endif
template <int STAGES, class Epi>
__global__ __launch_bounds__(256, 1) void k_gemm_q(const bf16_t* __restrict__ A, const bf16_t* __restrict__ B, int M,
                                                   int N, int K, int tiles_m, int tiles_n, Epi epi) {
  static_assert(Epi::kTrans, "transposed accumulators (lane <-> row)");
  constexpr int BM = 256, BN = 256, BK = 32, NW = 4, WT = 128, T4 = 4;
  constexpr int ROWB = BK * 2, CPR = ROWB / 16, RPB = 1024 / ROWB;   // 64-byte rows, 4 chunks, 16 rows per KB
  constexpr int A_BYTES = BM * ROWB, B_BYTES = BN * ROWB, SLOT = A_BYTES + B_BYTES;
  constexpr int A_BLK = A_BYTES / 1024, B_BLK = B_BYTES / 1024;
  constexpr int DPW = (A_BLK + B_BLK) / NW;      // DMA instructions per wave per K-step
  static_assert((STAGES - 2) * DPW <= 63 && STAGES >= 3, "stages in flight fit the vmcnt counter");
  static_assert(NW * 32 * (WT * 4 + 16) <= STAGES * SLOT, "epilogue staging fits the ring");
  __shared__ __attribute__((aligned(1024))) unsigned char lds[STAGES][SLOT];

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int fr = lane & 31, fh = lane >> 5;
  // XCD-aware block -> (mt, nt): the M tiles of one N tile run on one XCD at the same time
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int mt = local % tiles_m, nt = (local / tiles_m) * 8 + xcd;
  if (nt >= tiles_n) return;
  const int m0 = mt * BM, n0 = nt * BN;
  const int nk = K / BK;

  // per-lane 32-bit source offsets of this wave's DMA blocks (rows past M or N re-read the last row)
  uint32_t offA[A_BLK / NW], offB[B_BLK / NW];
#pragma unroll
  for (int j = 0; j < A_BLK / NW; ++j) {
    const int r = (wave + j * NW) * RPB + lane / CPR, c = (lane % CPR) ^ gemm_swz<CPR>(r);
    offA[j] = (uint32_t)min(m0 + r, M - 1) * (uint32_t)K * 2u + c * 16;
  }
#pragma unroll
  for (int j = 0; j < B_BLK / NW; ++j) {
    const int r = (wave + j * NW) * RPB + lane / CPR, c = (lane % CPR) ^ gemm_swz<CPR>(r);
    offB[j] = (uint32_t)min(n0 + r, N - 1) * (uint32_t)K * 2u + c * 16;
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)&lds[0][0];
  // transfer q (0..DPW-1) of this wave for step ks: A blocks first, then B blocks
  auto issue_one = [&](int ks, int q) __attribute__((always_inline)) {
    const uint32_t dst = lds0 + (uint32_t)(ks % STAGES) * SLOT;
    const uint32_t koff = (uint32_t)ks * ROWB;
    if (q < A_BLK / NW) lds_dma16_sv(offA[q] + koff, A, dst + (wave + q * NW) * 1024);
    else lds_dma16_sv(offB[q - A_BLK / NW] + koff, B, dst + A_BYTES + (wave + (q - A_BLK / NW) * NW) * 1024);
  };
  auto issue = [&](int ks) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < DPW; ++q) issue_one(ks, q);
  };

  // fragment of 32 rows x 16 K for row block rb (0..7 over the tile: A rows 32 rb, or B rows 32 (rb - 4)...):
  // lane reads row 32 i + l%32 at chunk 2 kk + l/32 (swizzled; the swizzle depends on l%32 only)
  const int sw = gemm_swz<CPR>(fr);
  const uint32_t a_off[2] = {(uint32_t)((wm * WT + fr) * ROWB + ((0 + fh) ^ sw) * 16),
                             (uint32_t)((wm * WT + fr) * ROWB + ((2 + fh) ^ sw) * 16)};
  const uint32_t b_off[2] = {(uint32_t)(A_BYTES + (wn * WT + fr) * ROWB + ((0 + fh) ^ sw) * 16),
                             (uint32_t)(A_BYTES + (wn * WT + fr) * ROWB + ((2 + fh) ^ sw) * 16)};
  struct Frag { u32x4 a[T4], b[T4]; };
  auto read_a = [&](int ks, int kk, int i) __attribute__((always_inline)) -> u32x4 {
    return *(const u32x4*)(&lds[ks % STAGES][0] + a_off[kk] + i * 32 * ROWB);
  };
  auto read_b = [&](int ks, int kk, int j) __attribute__((always_inline)) -> u32x4 {
    return *(const u32x4*)(&lds[ks % STAGES][0] + b_off[kk] + j * 32 * ROWB);
  };

  f32x16 acc[T4][T4];
#pragma unroll
  for (int i = 0; i < T4; ++i)
#pragma unroll
    for (int j = 0; j < T4; ++j) acc[i][j] = (f32x16){};

  // 16 MFMAs of one slice (fragments f, tile (i, j) at step 4 i + j), with the eight reads of the next slice
  // (ks2, kk2) into g issued after the first eight, in the order the next slice first uses them (b0, a0, b1,
  // b2, b3, a1, a2, a3): every read has at least eight MFMAs to land. dma = 1 or 2: the first or second half of
  // the DMA transfers of step kd, one after every fourth MFMA (issued back to back right after the barrier by
  // all four waves, the transfers queued at the CU's address unit for ~600 cycles per step while no MFMA ran).
  auto slice = [&](const Frag& f, Frag& g, auto more, auto dma, int ks2, int kk2, int kd) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < T4 * T4; ++t) {
      const int i = t / T4, j = t % T4;
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, f.b[j]),
                                                          __builtin_bit_cast(bf16x8, f.a[i]), acc[i][j], 0, 0, 0);
      if (decltype(more)::value && t < 2 * T4) {
        if (t == 0) g.b[0] = read_b(ks2, kk2, 0);
        else if (t == 1) g.a[0] = read_a(ks2, kk2, 0);
        else if (t < 5) g.b[t - 1] = read_b(ks2, kk2, t - 1);
        else g.a[t - 4] = read_a(ks2, kk2, t - 4);
      }
      if (decltype(dma)::value != 0 && (t % 4) == 3) issue_one(kd, (decltype(dma)::value - 1) * (DPW / 2) + t / 4);
      __builtin_amdgcn_sched_barrier(0);        // keep the MFMA / read / DMA order as written
    }
  };
  static_assert(DPW == 8, "half a step's transfers per slice, one per four MFMAs");

#pragma unroll
  for (int t = 0; t < STAGES; ++t)
    if (t < nk) issue(t);
  dma_stage_sync<DPW, STAGES - 1>(min(STAGES - 1, nk - 1));   // stage 0 landed
  Frag f0, f1;
#pragma unroll
  for (int i = 0; i < T4; ++i) { f0.a[i] = read_a(0, 0, i); f0.b[i] = read_b(0, 0, i); }
  using yes = std::integral_constant<bool, true>;
  using no = std::integral_constant<bool, false>;
  // slice 0 of step ks reads slice 1 of the same slot; then stage ks+1 has landed (the stages issued after it
  // may still be in flight) and every wave is done with slot ks (its fragments of both slices are in
  // registers), so slice 1 reads slice 0 of step ks+1 and refills slot ks with step ks+STAGES
  // registers), so slice 1 reads slice 0 of step ks+1 and starts refilling slot ks with step ks+STAGES; slice
  // 0 of step ks+1 finishes that refill (the slot has been free since this barrier). Every transfer of stage
  // s is issued before any of stage s+1, so a vmcnt bound of (STAGES-2) stages still means "stage ks+1 landed".
  using none = std::integral_constant<int, 0>;
  using half0 = std::integral_constant<int, 1>;
  using half1 = std::integral_constant<int, 2>;
  // (straight-line loop segments, not branches inside one loop: those made the register allocator move the
  // accumulators through scratch)
  int ks = 0;
  if (STAGES < nk) {
    slice(f0, f1, yes{}, none{}, 0, 1, 0);
    dma_stage_sync<DPW, STAGES - 2>(STAGES - 2);
    slice(f1, f0, yes{}, half0{}, 1, 0, STAGES);
    for (ks = 1; ks + STAGES < nk; ++ks) {
      slice(f0, f1, yes{}, half1{}, ks, 1, ks - 1 + STAGES);
      dma_stage_sync<DPW, STAGES - 2>(STAGES - 2);
      slice(f1, f0, yes{}, half0{}, ks + 1, 0, ks + STAGES);
    }
    // ks = nk - STAGES: the second half of the last stage
    slice(f0, f1, yes{}, half1{}, ks, 1, ks - 1 + STAGES);
    dma_stage_sync<DPW, STAGES - 2>(min(STAGES - 2, nk - 2 - ks));
    slice(f1, f0, yes{}, none{}, ks + 1, 0, 0);
    ++ks;
  }
  for (; ks + 1 < nk; ++ks) {
    slice(f0, f1, yes{}, none{}, ks, 1, 0);
    dma_stage_sync<DPW, STAGES - 2>(min(STAGES - 2, nk - 2 - ks));
    slice(f1, f0, yes{}, none{}, ks + 1, 0, 0);
  }
  slice(f0, f1, yes{}, none{}, nk - 1, 1, 0);   // the last step
  slice(f1, f0, no{}, none{}, 0, 0, 0);

  __syncthreads();                              // every wave has read its last fragments from the ring
  epi_trans<T4, T4, WT>(acc, &lds[0][0] + wave * 32 * (WT * 4 + 16), m0 + wm * WT, n0 + wn * WT, M, N, epi);
}

// ============================================================================ top-M per row
// Exact selection of the M largest entries of each fp32 row, ordered by (value desc, id asc),
// by a three-digit radix select on order-preserving keys (select.hpp) followed by an id-ordered tie
// pass.
//
// Exact top-M of a whole row (radix select + id-ordered tie pass). Used directly by the tree build on
// caller logits, and by the grouped selection for a row whose candidates overflow.
// Exact top-M of one row (whole block): ids and values in (value desc, id asc) order into out_id / out_val.
// ck / cid hold at least SR_MAX_TREE entries.
__device__ void topm_row(const float* __restrict__ row, int V, int M, int32_t* __restrict__ out_id,
                         float* __restrict__ out_val, int* hist, int* scan, RadixState& st, int& s_n, uint32_t* ck,
                         int* cid) {
  const int tid = threadIdx.x;
  if (tid == 0) s_n = 0;
  radix_kth([&](int i) { return fkey(row[i]); }, V, M, hist, scan, st);
  const uint32_t kstar = st.prefix;
  const int need_eq = st.rem, cnt_eq = st.cnt_eq;
  if (cnt_eq == need_eq) {
    for (int i = tid; i < V; i += TOPM_NT) {
      uint32_t k = fkey(row[i]);
      if (k >= kstar) { int p = atomicAdd(&s_n, 1); if (p < SR_MAX_TREE) { ck[p] = k; cid[p] = i; } }
    }
  } else {
    int taken = 0;
    for (int base = 0; base < V; base += TOPM_NT) {
      const int i = base + tid;
      uint32_t k = i < V ? fkey(row[i]) : 0u;
      if (i < V && k > kstar) { int p = atomicAdd(&s_n, 1); if (p < SR_MAX_TREE) { ck[p] = k; cid[p] = i; } }
      int tot;
      int r = block_prefix_excl((i < V && k == kstar) ? 1 : 0, scan, &tot);
      if (i < V && k == kstar && taken + r < need_eq) { int p = atomicAdd(&s_n, 1); if (p < SR_MAX_TREE) { ck[p] = k; cid[p] = i; } }
      taken += tot;
      if (taken >= need_eq) {
        // the remaining equal keys are not needed; keys above the threshold may still follow
        for (int j = base + TOPM_NT + tid; j < V; j += TOPM_NT) {
          uint32_t kk = fkey(row[j]);
          if (kk > kstar) { int p = atomicAdd(&s_n, 1); if (p < SR_MAX_TREE) { ck[p] = kk; cid[p] = j; } }
        }
        break;
      }
    }
  }
  __syncthreads();
  if (tid < M && s_n == M) {
    const uint32_t k = ck[tid];
    const int id = cid[tid];
    int rank = 0;
    for (int j = 0; j < M; ++j) rank += (ck[j] > k) || (ck[j] == k && cid[j] < id);
    out_id[rank] = id;
    out_val[rank] = row[id];
  }
}

__global__ __launch_bounds__(TOPM_NT) void k_topm(const float* __restrict__ logits, int V, int M,
                                                  int32_t* __restrict__ top_id, float* __restrict__ top_val) {
  __shared__ int hist[TOPM_BINS];
  __shared__ int scan[TOPM_NT];
  __shared__ RadixState st;
  __shared__ int s_n;
  __shared__ uint32_t ck[SR_MAX_TREE];
  __shared__ int cid[SR_MAX_TREE];
  const size_t r = blockIdx.x;
  topm_row(logits + r * V, V, M, top_id + r * M, top_val + r * M, hist, scan, st, s_n, ck, cid);
}

// Max of every 64-column group of each row (for logits that did not come from the vocabulary GEMM).
__global__ __launch_bounds__(256) void k_group_max(const float* __restrict__ logits, int V, int ngroups,
                                                   float* __restrict__ gmax) {
  const int row = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = blockIdx.x * 4 + wave;
  if (g >= ngroups) return;
  const int i = g * 64 + lane;
  float v = i < V ? logits[(size_t)row * V + i] : -INFINITY;
  v = warp_max(v);
  if (lane == 0) gmax[(size_t)row * ngroups + g] = v;
}

// Exact top-M of each row using its 64-column group maxima: tau = the M-th largest group max is a lower
// bound of the M-th largest value (the top M groups each hold an element >= tau), so every top-M element
// lies in a group whose max is >= tau and is itself >= tau. Only those groups are read. If more than
// TOPM_CAP elements qualify (heavy ties), the same block runs the full selection of the row.
constexpr int TOPM_MAXG = 4096;     // V <= 262144
constexpr int TOPM_CAP = 2048;
__global__ __launch_bounds__(TOPM_NT) void k_topm_grouped(const float* __restrict__ logits,
                                                          const float* __restrict__ gmax, int V, int ngroups, int M,
                                                          int32_t* __restrict__ top_id, float* __restrict__ top_val) {
  __shared__ uint32_t gk[TOPM_MAXG];
  __shared__ int glist[TOPM_MAXG];
  __shared__ int hist[TOPM_BINS];
  __shared__ int scan[TOPM_NT];
  __shared__ RadixState st;
  __shared__ int s_ng, s_n;
  __shared__ uint32_t ck[TOPM_CAP];
  __shared__ int cid[TOPM_CAP];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = blockIdx.x;
  const float* lrow = logits + (size_t)row * V;
  for (int g = tid; g < ngroups; g += TOPM_NT) gk[g] = fkey(gmax[(size_t)row * ngroups + g]);
  if (tid == 0) { s_ng = 0; s_n = 0; }
  __syncthreads();
  radix_kth([&](int i) { return gk[i]; }, ngroups, M, hist, scan, st);
  const uint32_t tau = st.prefix;
  for (int g = tid; g < ngroups; g += TOPM_NT)
    if (gk[g] >= tau) glist[atomicAdd(&s_ng, 1)] = g;
  __syncthreads();
  const int ng = s_ng;
  for (int q = wave; q < ng; q += TOPM_NT / 64) {
    const int i = glist[q] * 64 + lane;
    if (i < V) {
      const uint32_t k = fkey(lrow[i]);
      if (k >= tau) {
        const int p = atomicAdd(&s_n, 1);
        if (p < TOPM_CAP) { ck[p] = k; cid[p] = i; }
      }
    }
  }
  __syncthreads();
  const int n = s_n;
  if (n > TOPM_CAP) {                          // uniform: every thread has read s_n before it is reused
    __syncthreads();
    topm_row(lrow, V, M, top_id + (size_t)row * M, top_val + (size_t)row * M, hist, scan, st, s_n, ck, cid);
    return;
  }
  for (int t = tid; t < n; t += TOPM_NT) {
    const uint32_t k = ck[t];
    const int id = cid[t];
    int rank = 0;
    for (int j = 0; j < n; ++j) rank += (ck[j] > k) || (ck[j] == k && cid[j] < id);
    if (rank < M) {
      top_id[(size_t)row * M + rank] = id;
      top_val[(size_t)row * M + rank] = lrow[id];
    }
  }
}

// ============================================================================ tree build
// One block per trajectory, one wave per node with children: node u draws the ordered list of its
// m_u children from C_u = top-m_u of head min(depth(u)+1, H), without replacement (Eq. (slotq)).
// The wave holds C_u across its lanes, so each draw's float64 weights, their sum and the cumulative
// weights in C_u's order are computed in parallel.
constexpr int TB_NT = 1024;           // 16 waves: one node with children per wave at a time

// a float64 moved across the lanes of each 16-lane row by the DPP control CTRL (lanes whose source lies
// outside the row read 0)
template <int CTRL>
__device__ __forceinline__ double dpp0_f64(double v) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, 0xf, 0xf, true);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, 0xf, 0xf, true);
  return __hiloint2double(hi, lo);
}
__global__ __launch_bounds__(TB_NT) void k_tree_build(const int32_t* __restrict__ top_id,
                                                     const float* __restrict__ top_val, int H, int M, int T,
                                                     const int32_t* __restrict__ parents,
                                                     const int32_t* __restrict__ root_token,
                                                     const float* __restrict__ u_tree,
                                                     int32_t* __restrict__ tokens,
                                                     float* __restrict__ child_logit) {
  __shared__ TreeLds<SR_MAX_TREE> t;
  __shared__ int too_many;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  bool ok = tree_setup<SR_MAX_TREE>(t, parents + (size_t)b * T, T);
  if (ok) {
    if (tid == 0) too_many = 0;
    __syncthreads();
    if (tid < T && t.nkids[tid] > M) atomicOr(&too_many, 1);
    __syncthreads();
    ok = !too_many;
  }
  int32_t* tok_b = tokens + (size_t)b * T;
  float* cl_b = child_logit + (size_t)b * T;
  if (!ok) {
    for (int u = tid; u < T; u += TB_NT) {
      tok_b[u] = u == 0 ? root_token[b] : -1;
      cl_b[u] = u == 0 ? 0.f : __uint_as_float(0x7fc00000u);
    }
    return;
  }
  if (tid == 0) { tok_b[0] = root_token[b]; cl_b[0] = 0.f; }
  // one wave per node with children; lane i holds candidates i and i + 64 of C_u (the second only when
  // m_u > 64: with fewer candidates every second slot is empty and its weights, sums and ballots are zero)
  // NS = 0: at most 16 candidates, all in the first 16-lane row: the max, the prefix sums and the total
  // move by DPP within that row. The sums are the same additions in the same order as the wave-wide scan
  // (whose further steps only add zeros there), so the draws are identical.
  auto draws = [&](int u, int m, auto ns_) __attribute__((always_inline)) {
    constexpr bool R16 = decltype(ns_)::value == 0;
    constexpr int NS = R16 ? 1 : decltype(ns_)::value;
    const int k = min(t.depth[u] + 1, H);                      // proposing head, 1-based
    const size_t rbase = ((size_t)b * H + (k - 1)) * M;
    double l[NS];
    bool live[NS];
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) {
      const int i = lane + 64 * s2;
      live[s2] = i < m;
      l[s2] = live[s2] ? (double)top_val[rbase + i] : -INFINITY;
    }
    int c = u + 1;
    for (int j = 0; j < m; ++j) {
      while (t.parent[c] != u) ++c;                            // j-th child of u in index order
      // weights exp(l - max over the remaining candidates), float64, in C_u's order
      double lm = -INFINITY;
#pragma unroll
      for (int s2 = 0; s2 < NS; ++s2) lm = fmax(lm, live[s2] ? l[s2] : -INFINITY);
      double mx;
      if constexpr (R16) {
        mx = fmax(lm, dpp_f64<0xb1>(lm));         // quad_perm [1,0,3,2]
        mx = fmax(mx, dpp_f64<0x4e>(mx));         // quad_perm [2,3,0,1]
        mx = fmax(mx, dpp_f64<0x141>(mx));        // row_half_mirror
        mx = fmax(mx, dpp_f64<0x140>(mx));        // row_mirror
      } else {
        mx = wave_max_f64(lm);
      }
      double w[NS];
#pragma unroll
      for (int s2 = 0; s2 < NS; ++s2) w[s2] = live[s2] ? exp(l[s2] - mx) : 0.0;
      // inclusive prefix sums over candidates 0..63, then 64..127
      double cum[NS];
#pragma unroll
      for (int s2 = 0; s2 < NS; ++s2) {
        double v = w[s2];
        if constexpr (R16) {
          v += dpp0_f64<0x111>(v);                 // row_shr:1, 2, 4, 8
          v += dpp0_f64<0x112>(v);
          v += dpp0_f64<0x114>(v);
          v += dpp0_f64<0x118>(v);
        } else {
#pragma unroll
          for (int o = 1; o < 64; o <<= 1) {
            const double y = __shfl_up(v, o, 64);
            if (lane >= o) v += y;
          }
        }
        cum[s2] = v;
      }
      if constexpr (NS == 2) cum[1] += __shfl(cum[0], 63, 64);
      double S;
      if constexpr (R16)
        S = __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(cum[0]), 15),
                             __builtin_amdgcn_readlane(__double2loint(cum[0]), 15));
      else
        S = __shfl(cum[NS - 1], 63, 64);
      const double target = (double)u_tree[(size_t)b * T + c] * S;
      // first candidate whose cumulative weight exceeds the target; the last live one on rounding
      int pick = -1;
#pragma unroll
      for (int s2 = 0; s2 < NS; ++s2) {
        const unsigned long long hit = __ballot(live[s2] && target < cum[s2]);
        if (pick < 0 && hit) pick = 64 * s2 + __ffsll((long long)hit) - 1;
      }
      if (pick < 0) {
#pragma unroll
        for (int s2 = NS - 1; s2 >= 0; --s2) {
          const unsigned long long lv = __ballot(live[s2]);
          if (pick < 0 && lv) pick = 64 * s2 + 63 - __clzll((long long)lv);
        }
      }
      if (lane == (pick & 63)) live[pick >> 6] = false;
      if (lane == 0) {
        tok_b[c] = top_id[rbase + pick];
        cl_b[c] = top_val[rbase + pick];
      }
      ++c;
    }
  };
  for (int u = wave; u < T; u += TB_NT / 64) {
    const int m = t.nkids[u];
    if (m == 0) continue;                                      // uniform per wave
    if (m > 64) draws(u, m, std::integral_constant<int, 2>{});
    else if (m > 16) draws(u, m, std::integral_constant<int, 1>{});
    else draws(u, m, std::integral_constant<int, 0>{});
  }
}

// ============================================================================ launchers
template <typename T>
static sr_status launch_heads_z_t(const sr_heads_desc& d, const void* hidden, const float* corr,
                                  const uint8_t* active, const void* A, const void* bias, float* x, void* n, void* z,
                                  hipStream_t s) {
  SR_LAUNCH("sr_clip_ln", (k_clip_ln<T>), dim3(d.B), dim3(256), 0, s, (const T*)hidden, corr, active, d.d,
            d.clip_norm, d.ln_eps, x, (T*)n);
  if constexpr (sizeof(T) == 2) {
    constexpr int BM = 64, BN = 64, BK = 64;
    EpiHead<T> epi{(const T*)bias, x, (T*)z, d.d, d.H};
    if (d.B <= 32 && (d.H * d.d + BN - 1) / BN < 256) {
      // the rows fit one 32-row tile and 64 x 64 tiles would leave CUs without a block: the GEMM streams the
      // weights, and 32 x 32 one-wave tiles (four times the blocks) keep every CU streaming to the end; with
      // two row tiles they would read the weights twice
      const int tn = (d.H * d.d + 31) / 32;
      SR_LAUNCH("sr_head_gemm", (k_gemm_dl<32, 32, BK, 1, 1, 4, EpiHead<T>>), dim3(((tn + 7) / 8) * 8), dim3(64), 0, s,
                (const T*)n, (const T*)A, d.B, d.H * d.d, d.d, 1, tn, epi);
      return SR_OK;
    }
    const int tm = (d.B + BM - 1) / BM, tn = (d.H * d.d + BN - 1) / BN;
    dim3 grid(((tn + 7) / 8) * 8 * tm);
    SR_LAUNCH("sr_head_gemm", (k_gemm_dl<BM, BN, BK, 2, 2, 4, EpiHead<T>>), grid, dim3(256), 0, s, (const T*)n,
              (const T*)A, d.B, d.H * d.d, d.d, tm, tn, epi);
  } else {
    constexpr int BM = 64, BN = 128, BK = 32;
    EpiHead<T> epi{(const T*)bias, x, (T*)z, d.d, d.H};
    dim3 grid((d.H * d.d + BN - 1) / BN, (d.B + BM - 1) / BM);
    SR_LAUNCH("sr_head_gemm", (k_gemm<T, BM, BN, BK, 2, 2, EpiHead<T>>), grid, dim3(256), 0, s, (const T*)n,
              (const T*)A, d.B, d.H * d.d, d.d, epi);
  }
  return SR_OK;
}

template <typename T>
static sr_status launch_vocab_t(const sr_heads_desc& d, const void* z, const void* W, float* logits, float* gmax,
                                hipStream_t s) {
  const int M = d.B * d.H;
  if constexpr (sizeof(T) == 2) {
    // M = B*H rows: 256 x 256 quarter tiles (k_gemm_q) when there are enough rows to fill them. At small
    // batches the GEMM is a stream of W: 64- or 128-row tiles by 128 columns (four waves of 32 or 64 rows by
    // 64 columns; a 60 or 64 KB ring, two blocks per CU), so that the vocabulary splits into enough tiles
    // to keep every CU streaming to the end (256-column tiles at one block per CU left the last of three
    // rounds two-thirds empty)
    constexpr int BK = 32;
    EpiLogitsMax epi{logits, gmax, d.V, (d.V + 63) / 64};
    if (M <= 64) {
      constexpr int BM = 64;
      const int tm = (M + BM - 1) / BM, tn = (d.V + 127) / 128;
      SR_LAUNCH("sr_vocab_gemm", (k_gemm_dl<BM, 128, BK, 2, 2, 5, EpiLogitsMax>), dim3(((tn + 7) / 8) * 8 * tm),
                dim3(256), 0, s, (const T*)z, (const T*)W, M, d.V, d.d, tm, tn, epi);
    } else if (M <= 128) {
      constexpr int BM = 128;
      const int tm = (M + BM - 1) / BM, tn = (d.V + 127) / 128;
      SR_LAUNCH("sr_vocab_gemm", (k_gemm_dl<BM, 128, BK, 2, 2, 4, EpiLogitsMax>), dim3(((tn + 7) / 8) * 8 * tm),
                dim3(256), 0, s, (const T*)z, (const T*)W, M, d.V, d.d, tm, tn, epi);
    } else {
      constexpr int BM = 256, BN = 256;
      const int tm = (M + BM - 1) / BM, tn = (d.V + BN - 1) / BN;
      SR_LAUNCH("sr_vocab_gemm", (k_gemm_q<SR_GQ_STAGES, EpiLogitsMax>), dim3(((tn + 7) / 8) * 8 * tm), dim3(256), 0,
                s, (const T*)z, (const T*)W, M, d.V, d.d, tm, tn, epi);
    }
  } else {
    constexpr int BM = 128, BN = 128, BK = 32;
    EpiLogits epi{logits, d.V};
    dim3 grid((d.V + BN - 1) / BN, (M + BM - 1) / BM);
    SR_LAUNCH("sr_vocab_gemm", (k_gemm<T, BM, BN, BK, 2, 2, EpiLogits>), grid, dim3(256), 0, s, (const T*)z,
              (const T*)W, M, d.V, d.d, epi);
    const int ng = (d.V + 63) / 64;
    SR_LAUNCH("sr_group_max", k_group_max, dim3((ng + 3) / 4, M), dim3(256), 0, s, logits, d.V, ng, gmax);
  }
  return SR_OK;
}

sr_status launch_heads_z(const sr_heads_desc& d, const void* hidden, const float* corr, const uint8_t* active,
                         const void* A, const void* bias, float* x, void* n, void* z, hipStream_t s) {
  if (d.dtype == SR_BF16) return launch_heads_z_t<bf16_t>(d, hidden, corr, active, A, bias, x, n, z, s);
  return launch_heads_z_t<float>(d, hidden, corr, active, A, bias, x, n, z, s);
}

sr_status launch_vocab(const sr_heads_desc& d, const void* z, const void* W, float* logits, float* gmax,
                       hipStream_t s) {
  if (d.dtype == SR_BF16) return launch_vocab_t<bf16_t>(d, z, W, logits, gmax, s);
  return launch_vocab_t<float>(d, z, W, logits, gmax, s);
}

sr_status launch_heads(const sr_heads_desc& d, const void* hidden, const float* corr, const uint8_t* active,
                       const void* A, const void* bias, const void* W, float* x, void* n, void* z,
                       float* logits, float* gmax, hipStream_t s) {
  sr_status st = launch_heads_z(d, hidden, corr, active, A, bias, x, n, z, s);
  if (st != SR_OK) return st;
  return launch_vocab(d, z, W, logits, gmax, s);
}

sr_status launch_tree_build(const sr_heads_desc& d, const float* logits, const float* gmax,
                            const int32_t* parents, const int32_t* root_token, const float* u_tree,
                            int32_t* tokens, float* child_logit, int32_t* top_id, float* top_val, hipStream_t s) {
  const int M = d.max_children;
  const int rows = d.B * d.H;
  if (M > 0) {
    const int ng = (d.V + 63) / 64;
    if (gmax != nullptr && ng <= TOPM_MAXG && M <= ng) {
      SR_LAUNCH("sr_topm", k_topm_grouped, dim3(rows), dim3(TOPM_NT), 0, s, logits, gmax, d.V, ng, M, top_id,
                top_val);
    } else {
      SR_LAUNCH("sr_topm_full", k_topm, dim3(rows), dim3(TOPM_NT), 0, s, logits, d.V, M, top_id, top_val);
    }
  }
  SR_LAUNCH("sr_tree_build", k_tree_build, dim3(d.B), dim3(TB_NT), 0, s, top_id, top_val, d.H, M, d.T,
            parents, root_token, u_tree, tokens, child_logit);
  return SR_OK;
}

size_t group_max_count(const sr_heads_desc& d) { return (size_t)d.B * d.H * ((d.V + 63) / 64); }

sr_status launch_group_max(const sr_heads_desc& d, const float* logits, float* gmax, hipStream_t s) {
  const int ng = (d.V + 63) / 64;
  SR_LAUNCH("sr_group_max", k_group_max, dim3((ng + 3) / 4, d.B * d.H), dim3(256), 0, s, logits, d.V, ng, gmax);
  return SR_OK;
}

}  // namespace sr
