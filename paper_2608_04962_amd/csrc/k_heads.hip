// Proposal step on gfx950: Reflex-corrected LayerNorm, the head residual blocks and
// the shared-vocabulary projection as MFMA GEMMs, per-row top-M selection, and the
// ordered without-replacement draft-tree build.
//
// Paper: Sec. 3.2 Eq. (heads); App. C "Future-token proposer" (z = h + SiLU(A LN(h) + b),
// logits through the target's vocabulary projection); App. B.1 Eq. (slotq), Eq. (childlist).
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace sr {

// ============================================================================ clip + LayerNorm
// One block per trajectory: x = h + corr * min(1, c/||corr||) (active rows), n = LN(x).
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

// ============================================================================ top-M per row
// Exact selection of the M largest entries of each fp32 row, ordered by (value desc, id asc),
// by a three-digit radix select on order-preserving keys followed by an id-ordered tie pass.
__device__ __forceinline__ uint32_t fkey(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int TOPM_NT = 512;
constexpr int TOPM_BINS = 2048;

// Suffix (exclusive, from the top) scan of per-thread counts over the block.
__device__ int block_suffix_excl(int v, int* sh) {
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
__device__ int block_prefix_excl(int v, int* sh, int* total) {
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

__global__ __launch_bounds__(TOPM_NT) void k_topm(const float* __restrict__ logits, int V, int M,
                                                  int32_t* __restrict__ top_id, float* __restrict__ top_val) {
  __shared__ int hist[TOPM_BINS];
  __shared__ int scan[TOPM_NT];
  __shared__ uint32_t s_prefix, s_pmask;
  __shared__ int s_rem, s_cnt_eq, s_n;
  __shared__ uint32_t ck[SR_MAX_TREE];
  __shared__ int cid[SR_MAX_TREE];
  const int tid = threadIdx.x;
  const float* row = logits + (size_t)blockIdx.x * V;
  if (tid == 0) { s_prefix = 0; s_pmask = 0; s_rem = M; s_n = 0; }
  const int shifts[3] = {21, 10, 0};
  const int bits[3] = {11, 11, 10};
  for (int pass = 0; pass < 3; ++pass) {
    for (int i = tid; i < TOPM_BINS; i += TOPM_NT) hist[i] = 0;
    __syncthreads();
    const uint32_t prefix = s_prefix, pmask = s_pmask;
    const int sh = shifts[pass];
    const uint32_t dmask = (1u << bits[pass]) - 1u;
    for (int i = tid; i < V; i += TOPM_NT) {
      uint32_t k = fkey(row[i]);
      if ((k & pmask) == prefix) atomicAdd(&hist[(k >> sh) & dmask], 1);
    }
    __syncthreads();
    // thread t owns bins [4t, 4t+4); find the bin holding rank s_rem counted from the top
    const int nb = (1 << bits[pass]) / TOPM_NT;    // 4 or 2
    int local = 0;
    for (int j = 0; j < nb; ++j) local += hist[tid * nb + j];
    const int above = block_suffix_excl(local, scan);
    const int rem = s_rem;
    __syncthreads();
    if (above < rem && rem <= above + local) {
      int a = above;
      for (int j = nb - 1; j >= 0; --j) {
        int c = hist[tid * nb + j];
        if (rem <= a + c) {
          s_prefix = prefix | ((uint32_t)(tid * nb + j) << sh);
          s_pmask = pmask | (dmask << sh);
          s_rem = rem - a;
          s_cnt_eq = c;
          break;
        }
        a += c;
      }
    }
    __syncthreads();
  }
  const uint32_t kstar = s_prefix;
  const int need_eq = s_rem, cnt_eq = s_cnt_eq;
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
    top_id[(size_t)blockIdx.x * M + rank] = id;
    top_val[(size_t)blockIdx.x * M + rank] = row[id];
  }
}

// ============================================================================ tree build
// One block per trajectory, one thread per node: node u draws the ordered list of its m_u
// children from C_u = top-m_u of head min(depth(u)+1, H), without replacement (Eq. (slotq)).
__global__ __launch_bounds__(SR_MAX_TREE) void k_tree_build(const int32_t* __restrict__ top_id,
                                                            const float* __restrict__ top_val, int H, int M, int T,
                                                            const int32_t* __restrict__ parents,
                                                            const int32_t* __restrict__ root_token,
                                                            const float* __restrict__ u_tree,
                                                            int32_t* __restrict__ tokens,
                                                            float* __restrict__ child_logit) {
  __shared__ TreeLds<SR_MAX_TREE> t;
  __shared__ int too_many;
  const int b = blockIdx.x, u = threadIdx.x;
  bool ok = tree_setup<SR_MAX_TREE>(t, parents + (size_t)b * T, T);
  if (ok) {
    if (u == 0) too_many = 0;
    __syncthreads();
    if (u < T && t.nkids[u] > M) atomicOr(&too_many, 1);
    __syncthreads();
    ok = !too_many;
  }
  int32_t* tok_b = tokens + (size_t)b * T;
  float* cl_b = child_logit + (size_t)b * T;
  if (!ok) {
    if (u < T) {
      tok_b[u] = u == 0 ? root_token[b] : -1;
      cl_b[u] = u == 0 ? 0.f : __uint_as_float(0x7fc00000u);
    }
    return;
  }
  if (u == 0) { tok_b[0] = root_token[b]; cl_b[0] = 0.f; }
  if (u >= T) return;
  const int m = t.nkids[u];
  if (m == 0) return;
  const int k = min(t.depth[u] + 1, H);                       // proposing head, 1-based
  const size_t rbase = ((size_t)b * H + (k - 1)) * M;
  uint32_t used[SR_MAX_TREE / 32] = {0, 0, 0, 0};
  int c = u + 1;
  for (int j = 0; j < m; ++j) {
    while (t.parent[c] != u) ++c;                              // j-th child of u in index order
    // weights exp(l - max over the remaining candidates), float64, in C_u's order
    double mx = -INFINITY;
    for (int i = 0; i < m; ++i)
      if (!((used[i >> 5] >> (i & 31)) & 1u)) mx = fmax(mx, (double)top_val[rbase + i]);
    double S = 0.0;
    for (int i = 0; i < m; ++i)
      if (!((used[i >> 5] >> (i & 31)) & 1u)) S += exp((double)top_val[rbase + i] - mx);
    const double target = (double)u_tree[(size_t)b * T + c] * S;
    double cum = 0.0;
    int pick = -1, last = -1;
    for (int i = 0; i < m; ++i) {
      if ((used[i >> 5] >> (i & 31)) & 1u) continue;
      cum += exp((double)top_val[rbase + i] - mx);
      last = i;
      if (target < cum) { pick = i; break; }
    }
    if (pick < 0) pick = last;                                 // rounding guard: U*S at the very top
    used[pick >> 5] |= 1u << (pick & 31);
    tok_b[c] = top_id[rbase + pick];
    cl_b[c] = top_val[rbase + pick];
    ++c;
  }
}

// ============================================================================ launchers
template <typename T>
static sr_status launch_heads_t(const sr_heads_desc& d, const void* hidden, const float* corr,
                                const uint8_t* active, const void* A, const void* bias, const void* W,
                                float* x, void* n, void* z, float* logits, hipStream_t s) {
  SR_LAUNCH("sr_clip_ln", (k_clip_ln<T>), dim3(d.B), dim3(256), 0, s, (const T*)hidden, corr, active, d.d,
            d.clip_norm, d.ln_eps, x, (T*)n);
  {
    constexpr int BM = 64, BN = 128, BK = (sizeof(T) == 2 ? 64 : 32);
    EpiHead<T> epi{(const T*)bias, x, (T*)z, d.d, d.H};
    dim3 grid((d.H * d.d + BN - 1) / BN, (d.B + BM - 1) / BM);
    SR_LAUNCH("sr_head_gemm", (k_gemm<T, BM, BN, BK, 2, 2, EpiHead<T>>), grid, dim3(256), 0, s, (const T*)n,
              (const T*)A, d.B, d.H * d.d, d.d, epi);
  }
  {
    constexpr int BM = 128, BN = 128, BK = (sizeof(T) == 2 ? 64 : 32);
    EpiLogits epi{logits, d.V};
    const int M = d.B * d.H;
    dim3 grid((d.V + BN - 1) / BN, (M + BM - 1) / BM);
    SR_LAUNCH("sr_vocab_gemm", (k_gemm<T, BM, BN, BK, 2, 2, EpiLogits>), grid, dim3(256), 0, s, (const T*)z,
              (const T*)W, M, d.V, d.d, epi);
  }
  return SR_OK;
}

sr_status launch_heads(const sr_heads_desc& d, const void* hidden, const float* corr, const uint8_t* active,
                       const void* A, const void* bias, const void* W, float* x, void* n, void* z,
                       float* logits, hipStream_t s) {
  if (d.dtype == SR_BF16) return launch_heads_t<bf16_t>(d, hidden, corr, active, A, bias, W, x, n, z, logits, s);
  return launch_heads_t<float>(d, hidden, corr, active, A, bias, W, x, n, z, logits, s);
}

sr_status launch_tree_build(const sr_heads_desc& d, const float* logits, const int32_t* parents,
                            const int32_t* root_token, const float* u_tree, int32_t* tokens, float* child_logit,
                            int32_t* top_id, float* top_val, hipStream_t s) {
  const int M = d.max_children;
  if (M > 0) {
    SR_LAUNCH("sr_topm", k_topm, dim3(d.B * d.H), dim3(TOPM_NT), 0, s, logits, d.V, M, top_id, top_val);
  }
  SR_LAUNCH("sr_tree_build", k_tree_build, dim3(d.B), dim3(SR_MAX_TREE), 0, s, top_id, top_val, d.H, M, d.T,
            parents, root_token, u_tree, tokens, child_logit);
  return SR_OK;
}

}  // namespace sr
