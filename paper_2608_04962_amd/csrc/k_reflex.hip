// Reflex verifier feedback: one matured proposal record per block.
//
// Paper: Sec. 3.3 -- the distribution and coverage errors of a candidate set C, Eq. (optimal-candidates),
// Eq. (conditional-distributions), Eq. (conditional-overlap), Eq. (acceptance-gap-decomposition);
// Sec. 3.4 -- the sparse support S (Eq. (support)), the directions W_S^T (p_S - q_S) (Eq. (distdir)) and
// sum_{y in O} p_S(y) (W_y - W_B) (Eq. (covdir)), their RMS-normalised combination (Eq. (unified-feedback))
// and the memory EMA (Eq. (ema)); App. A.1 for the coverage direction over a weighted boundary set;
// App. C "Verifier-derived feedback" for the support budget, weights, severity and gate.
//
// A block (8 waves) reads the record's target row and proposal row once each: every wave reduces
// 512-token chunks to (chunk max, sum of exp) in fp32 and writes the 64-token group maxima as
// order-preserving keys. The top lists come from those group maxima (the k-th largest group max bounds
// the k-th largest value, so only the groups at or above it are read again); a row whose groups cannot
// separate the top k (fewer than k groups, or more than RF_CAP tied candidates) takes the full radix
// select instead. Wave 0 then builds the support and every per-record scalar in float64, and the whole
// block gathers the support's rows of W into the two d-vectors, normalises and folds them into the
// memory row.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"
#include "select.hpp"

namespace sr {

constexpr int RF_NT = TOPM_NT;            // 512 threads
constexpr int RF_NW = RF_NT / 64;
constexpr int RF_CH = 512;                // tokens per wave chunk (64 lanes x 8)
constexpr int RF_MAXCH = 512;             // V <= 262144
constexpr int RF_MAXG = 4096;             // 64-token groups
constexpr int RF_CAP = 2048;              // candidates of the grouped selection
constexpr int RF_MAXS = 64;               // support, top lists and candidates
constexpr int RF_SEQ = 4 * RF_MAXS + 1;   // support sequence before de-duplication
constexpr int RF_CG = 2;                  // 8-column groups of W per thread: d <= 8 * RF_NT * RF_CG
constexpr int RF_GROUP = 4;               // row chunks whose loads a wave issues together

template <typename T> struct RfRow;
template <> struct RfRow<bf16_t> {
  static __device__ __forceinline__ void load8(const bf16_t* p, float* x) {
    const u32x4 w = *(const u32x4*)p;
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = bf2f((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xffffu));
  }
  static __device__ __forceinline__ float load1(const bf16_t* p) { return bf2f(*p); }
};
template <> struct RfRow<float> {
  static __device__ __forceinline__ void load8(const float* p, float* x) {
    const f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) { x[e] = a[e]; x[e + 4] = b[e]; }
  }
  static __device__ __forceinline__ float load1(const float* p) { return *p; }
};

struct RfSmem {
  uint32_t gk[RF_MAXG];
  int glist[RF_MAXG];
  uint32_t ck[RF_CAP];
  int cid[RF_CAP];
  int hist[TOPM_BINS];
  int scan[RF_NT];
  float cmax[RF_MAXCH / RF_GROUP];   // per group of RF_GROUP chunks: reference max and sum
  float csum[RF_MAXCH / RF_GROUP];
  RadixState st;
  int s_ng, s_n;
  int top_p[RF_MAXS], top_q[RF_MAXS];
  int seq[RF_SEQ];
  int S[RF_MAXS];
  float ca[RF_MAXS], cb[RF_MAXS];   // coefficients of the support rows in r_dist and r_cov
  double red[RF_NW][2];
  double xr[RF_NW][RF_MAXS];      // per-wave partial sketch projections
  float Mrow;
  double Zrow;
  int nS, bad;
  double dd, dc, tvs, sev, pC, pstar;
};

// exp(y - m) with y = x * invtau (m finite), as 2^(x (invtau log2 e) - m log2 e): one fused
// multiply-add with both factors rounded to fp32 first, the same wherever it is evaluated
__device__ __forceinline__ float rf_tilt(float x, float invtau, float m) {
  return __builtin_amdgcn_exp2f(__builtin_fmaf(x, __fmul_rn(invtau, kLog2e), -__fmul_rn(m, kLog2e)));
}

// One pass over a row: group-max keys, the row max M of x * invtau and Z = sum exp(x * invtau - M).
template <typename T>
__device__ void rf_row_pass(RfSmem& sm, const T* __restrict__ row, int V, float invtau) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nch = (V + RF_CH - 1) / RF_CH;
  // RF_GROUP chunks per wave at a time, their loads issued together
  for (int c0 = wave * RF_GROUP; c0 < nch; c0 += RF_NW * RF_GROUP) {
    float x[RF_GROUP][8];
#pragma unroll
    for (int gi = 0; gi < RF_GROUP; ++gi) {
      const int base = (c0 + gi) * RF_CH + lane * 8;
      if (c0 + gi < nch && base < V) {
        RfRow<T>::load8(row + base, x[gi]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[gi][e] = -INFINITY;
      }
    }
    // 64-token group maxima (lanes 8j .. 8j+7 of a chunk, by DPP), then one reference max and one sum
    // for the whole group of chunks: only the row's max and sum are kept
    float ml = -INFINITY;
#pragma unroll
    for (int gi = 0; gi < RF_GROUP; ++gi) {
      const int c = c0 + gi;
      const int base = c * RF_CH + lane * 8;
      float gm = x[gi][0];
#pragma unroll
      for (int e = 1; e < 8; ++e) gm = fmaxf(gm, x[gi][e]);
      gm = fmaxf(gm, dpp_f32<0xB1>(gm));        // lanes i, i ^ 1
      gm = fmaxf(gm, dpp_f32<0x4E>(gm));        // lanes i, i ^ 2
      gm = fmaxf(gm, dpp_f32<0x141>(gm));       // quads 0 and 1 of each 8 lanes
      if (c < nch && (lane & 7) == 0 && base < V) sm.gk[c * 8 + (lane >> 3)] = fkey(gm);
      ml = fmaxf(ml, gm);
    }
    // max of x * invtau from the raw maxima (rounding is monotone and invtau > 0)
    const float m = __fmul_rn(wave_max_f32(ml), invtau);
    float sl = 0.f;                             // at most 32 terms per lane in (0, 1]
    if (m != -INFINITY) {                       // uniform; a -inf token then weighs 2^-inf = 0
#pragma unroll
      for (int gi = 0; gi < RF_GROUP; ++gi)
#pragma unroll
        for (int e = 0; e < 8; ++e) sl += rf_tilt(x[gi][e], invtau, m);
    }
    const float s = wave_sum_f32(sl);
    if (lane == 0) { sm.cmax[c0 / RF_GROUP] = m; sm.csum[c0 / RF_GROUP] = s; }
  }
  __syncthreads();
  if (wave == 0) {
    const int ng = (nch + RF_GROUP - 1) / RF_GROUP;
    float ml = -INFINITY;
    for (int g = lane; g < ng; g += 64) ml = fmaxf(ml, sm.cmax[g]);
    const float M = wave_max_f32(ml);
    double sl = 0.0;
    for (int g = lane; g < ng; g += 64) sl += (double)sm.csum[g] * exp((double)sm.cmax[g] - (double)M);
    const double Z = wave_sum_f64(sl);
    if (lane == 0) { sm.Mrow = M; sm.Zrow = Z; }
  }
  __syncthreads();
}

// Rank the n collected (key, id) pairs by (key desc, id asc) and keep the first k ids in out[].
__device__ void rf_rank_out(RfSmem& sm, int n, int k, int* out) {
  for (int t = threadIdx.x; t < n; t += RF_NT) {
    const uint32_t key = sm.ck[t];
    const int id = sm.cid[t];
    int rank = 0;
    for (int j = 0; j < n; ++j) rank += (sm.ck[j] > key) || (sm.ck[j] == key && sm.cid[j] < id);
    if (rank < k) out[rank] = id;
  }
  __syncthreads();
}

// Exact top-k of a row by a radix select over the whole row (any k <= V, any number of ties).
template <typename T>
__device__ void rf_topk_full(RfSmem& sm, const T* __restrict__ row, int V, int k, int* out) {
  const int tid = threadIdx.x;
  radix_kth([&](int i) { return fkey(RfRow<T>::load1(row + i)); }, V, k, sm.hist, sm.scan, sm.st);
  const uint32_t kstar = sm.st.prefix;
  const int need_eq = sm.st.rem;
  if (tid == 0) sm.s_n = 0;
  __syncthreads();
  // keys above the k-th: at most k - need_eq of them
  for (int i = tid; i < V; i += RF_NT) {
    const uint32_t key = fkey(RfRow<T>::load1(row + i));
    if (key > kstar) {
      const int p = atomicAdd(&sm.s_n, 1);
      if (p < RF_CAP) { sm.ck[p] = key; sm.cid[p] = i; }
    }
  }
  __syncthreads();
  // the first need_eq keys equal to the k-th, in id order, one 512-token block at a time
  int taken = 0;
  for (int base = 0; base < V && taken < need_eq; base += RF_NT) {
    const int i = base + tid;
    const bool eq = i < V && fkey(RfRow<T>::load1(row + i)) == kstar;
    int tot;
    const int r = block_prefix_excl(eq ? 1 : 0, sm.scan, &tot);
    if (eq && taken + r < need_eq) {
      const int p = atomicAdd(&sm.s_n, 1);
      if (p < RF_CAP) { sm.ck[p] = kstar; sm.cid[p] = i; }
    }
    taken += tot;
  }
  __syncthreads();
  rf_rank_out(sm, min(sm.s_n, RF_CAP), k, out);
}

// Exact top-k from the group-max keys written by rf_row_pass; falls back to rf_topk_full.
template <typename T>
__device__ void rf_topk(RfSmem& sm, const T* __restrict__ row, int V, int k, int* out) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ng = (V + 63) / 64;
  if (k > ng) {
    rf_topk_full<T>(sm, row, V, k, out);
    return;
  }
  if (tid == 0) { sm.s_ng = 0; sm.s_n = 0; }
  radix_kth([&](int i) { return sm.gk[i]; }, ng, k, sm.hist, sm.scan, sm.st);
  const uint32_t tau = sm.st.prefix;
  for (int g = tid; g < ng; g += RF_NT)
    if (sm.gk[g] >= tau) sm.glist[atomicAdd(&sm.s_ng, 1)] = g;
  __syncthreads();
  const int nsel = sm.s_ng;
  for (int q = wave; q < nsel; q += RF_NW) {
    const int i = sm.glist[q] * 64 + lane;
    if (i < V) {
      const uint32_t key = fkey(RfRow<T>::load1(row + i));
      if (key >= tau) {
        const int p = atomicAdd(&sm.s_n, 1);
        if (p < RF_CAP) { sm.ck[p] = key; sm.cid[p] = i; }
      }
    }
  }
  __syncthreads();
  const int n = sm.s_n;
  __syncthreads();
  if (n > RF_CAP) {
    rf_topk_full<T>(sm, row, V, k, out);
    return;
  }
  rf_rank_out(sm, n, k, out);
}

// block-wide sums of two per-thread float64 values; every thread receives them
__device__ __forceinline__ void rf_block_sum2(RfSmem& sm, double& a, double& b) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  a = wave_sum_f64(a);
  b = wave_sum_f64(b);
  if (lane == 0) { sm.red[wave][0] = a; sm.red[wave][1] = b; }
  __syncthreads();
  a = 0.0;
  b = 0.0;
  for (int w = 0; w < RF_NW; ++w) { a += sm.red[w][0]; b += sm.red[w][1]; }
  __syncthreads();
}

template <typename TP, typename TW>
__global__ __launch_bounds__(RF_NT) void k_reflex_feedback(
    const TP* __restrict__ plog, const int32_t* __restrict__ p_row, const float* __restrict__ qlog,
    const int32_t* __restrict__ q_row, const int32_t* __restrict__ cand, const int32_t* __restrict__ y_star,
    const int32_t* __restrict__ traj, const int32_t* __restrict__ horizon, const TW* __restrict__ W,
    float* __restrict__ memory, float* __restrict__ stats, float* __restrict__ e_out, const float* __restrict__ P,
    const float* __restrict__ rec_sketch, float* __restrict__ align, sr_reflex_desc d) {
  __shared__ RfSmem sm;
  const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int V = d.V, KS = d.support, MC = d.max_cand;
  const float invtau = 1.0f / d.temperature;
  float* st_out = stats + (size_t)r * 8;

  // ---- validation (uniform over the block)
  const int pr = p_row[r], qr = q_row[r], ti = traj[r], hz = horizon[r], ys = y_star[r];
  bool bad = pr < 0 || pr >= d.n_p_rows || qr < 0 || qr >= d.n_q_rows || ti < 0 || ti >= d.B || hz < 1 ||
             hz > d.H || ys < 0 || ys >= V;
  bool dup = false;
  for (int j = tid; j < r; j += RF_NT) dup |= traj[j] == ti && horizon[j] == hz;
  dup = __syncthreads_or(dup);
  if (tid == 0) sm.bad = 0;
  __syncthreads();
  int K = 0;
  if (!bad && !dup) {
    // candidates: a non-empty prefix of in-range, distinct ids followed by -1 padding
    const int32_t* cr = cand + (size_t)r * MC;
    for (int j = tid; j < MC; j += RF_NT) {
      const int c = cr[j];
      if (c >= V || c < -1) atomicOr(&sm.bad, 1);
      if (c == -1) continue;
      if (j > 0 && cr[j - 1] == -1) atomicOr(&sm.bad, 1);
      for (int i = 0; i < j; ++i)
        if (cr[i] == c) atomicOr(&sm.bad, 1);
    }
    __syncthreads();
    for (int j = 0; j < MC && cr[j] >= 0; ++j) ++K;
    bad = sm.bad != 0 || K == 0;
  }
  if (bad || dup) {
    if (tid < 8) st_out[tid] = tid == 5 ? (dup ? -1.f : -2.f) : __uint_as_float(0x7fc00000u);
    if (e_out)
      for (int c = tid; c < d.d; c += RF_NT) e_out[(size_t)r * d.d + c] = __uint_as_float(0x7fc00000u);
    return;
  }
  const int32_t* cr = cand + (size_t)r * MC;
  const TP* prow = plog + (size_t)pr * V;
  const float* qrow = qlog + (size_t)qr * V;
  const int KP = max(KS, K);

  // ---- the two rows: statistics and top lists
  rf_row_pass<TP>(sm, prow, V, invtau);
  const float Mp = sm.Mrow;
  const double Zp = sm.Zrow;
  rf_topk<TP>(sm, prow, V, KP, sm.top_p);
  rf_row_pass<float>(sm, qrow, V, invtau);
  const float Mq = sm.Mrow;
  const double Zq = sm.Zrow;
  rf_topk<float>(sm, qrow, V, KS, sm.top_q);

  // ---- support sequence: C, Top_K(p), y*, then the rest of Top_k(p) and Top_k(q) alternately
  if (tid == 0) {
    int L = 0;
    for (int j = 0; j < K; ++j) sm.seq[L++] = cr[j];
    for (int j = 0; j < K; ++j) sm.seq[L++] = sm.top_p[j];
    sm.seq[L++] = ys;
    const int np = KP - K, nq = KS;
    for (int i = 0; i < max(np, nq); ++i) {
      if (i < np) sm.seq[L++] = sm.top_p[K + i];
      if (i < nq) sm.seq[L++] = sm.top_q[i];
    }
    sm.nS = L;
  }
  __syncthreads();
  // ---- support: first occurrences in sequence order, at most KS entries (wave 0)
  if (wave == 0) {
    const int L = sm.nS;
    int nS = 0;
    for (int b0 = 0; b0 < L && nS < KS; b0 += 64) {
      const int i = b0 + lane;
      bool first = false;
      int v = -1;
      if (i < L) {
        v = sm.seq[i];
        first = true;
        for (int j = 0; j < i; ++j)
          if (sm.seq[j] == v) { first = false; break; }
      }
      const unsigned long long m = __ballot(first);
      const int pos = nS + __popcll(m & ((1ull << lane) - 1ull));
      if (first && pos < KS) sm.S[pos] = v;
      nS = min(KS, nS + __popcll(m));
    }
    if (lane == 0) sm.nS = nS;
  }
  __syncthreads();
  // ---- per-record scalars and the support coefficients (wave 0, float64)
  if (wave == 0) {
    const int nS = sm.nS;
    // p and q of the candidates and of Top_K(p)
    double pc = 0.0, qc = 0.0, qlc = -INFINITY, ptop = 0.0;
    int cid = -1;
    if (lane < K) {
      cid = cr[lane];
      pc = exp((double)__fmul_rn(RfRow<TP>::load1(prow + cid), invtau) - (double)Mp) / Zp;
      qlc = (double)qrow[cid];
      qc = exp((double)__fmul_rn((float)qlc, invtau) - (double)Mq) / Zq;
      ptop = exp((double)__fmul_rn(RfRow<TP>::load1(prow + sm.top_p[lane]), invtau) - (double)Mp) / Zp;
    }
    const double pC = wave_sum_f64(pc), qC = wave_sum_f64(qc), pstar = wave_sum_f64(ptop);
    const double tvc = 0.5 * wave_sum_f64(lane < K ? fabs(pc / pC - qc / qC) : 0.0);
    // boundary set: the n_boundary candidates of lowest head logit (ties to the lower id)
    int brank = 1 << 30;
    if (lane < K) {
      brank = 0;
      for (int j = 0; j < K; ++j) {
        const int oj = cr[j];
        const double qj = (double)qrow[oj];
        brank += (qj < qlc) || (qj == qlc && oj < cid);
      }
    }
    const int nb = min(d.n_boundary, K);
    // support distributions; O = Top_K(p) outside C
    double ps = 0.0, qs = 0.0;
    int sv = -1;
    bool inO = false, inB = false;
    if (lane < nS) {
      sv = sm.S[lane];
      ps = exp((double)__fmul_rn(RfRow<TP>::load1(prow + sv), invtau) - (double)Mp) / Zp;
      qs = exp((double)__fmul_rn(qrow[sv], invtau) - (double)Mq) / Zq;
      bool inC = false, inTop = false;
      for (int j = 0; j < K; ++j) {
        inC |= cr[j] == sv;
        inTop |= sm.top_p[j] == sv;
      }
      inO = inTop && !inC;
    }
    // B membership of support entry sv: the candidate lane holding sv has brank < nb
    for (int j = 0; j < K; ++j) {
      const int cj = __shfl(cid, j, 64);
      const int bj = __shfl(brank, j, 64);
      if (lane < nS && sv == cj && bj < nb) inB = true;
    }
    const double sp = wave_sum_f64(ps), sq = wave_sum_f64(qs);
    const double pS = lane < nS ? ps / sp : 0.0, qS = lane < nS ? qs / sq : 0.0;
    const double tvs = 0.5 * wave_sum_f64(fabs(pS - qS));
    const double sumO = wave_sum_f64(inO ? pS : 0.0);
    if (lane < nS) {
      sm.ca[lane] = (float)(pS - qS);
      sm.cb[lane] = (float)((inO ? pS : 0.0) - (inB ? sumO / nb : 0.0));
    }
    if (lane == 0) {
      sm.nS = nS;
      sm.pC = pC;
      sm.pstar = pstar;
      sm.dd = pC * tvc;
      sm.dc = pstar - pC;
      sm.tvs = tvs;
      sm.sev = fmin(fmax((double)d.sev_tv * tvs + (double)d.sev_out * (1.0 - pC), 0.0), 1.0);
    }
  }
  __syncthreads();

  // ---- d-vectors: r_dist and r_cov from the support rows of W (8 consecutive columns per lane)
  const int nS = sm.nS;
  const int dcols = d.d;
  float rd[RF_CG][8], rc[RF_CG][8];
#pragma unroll
  for (int gi = 0; gi < RF_CG; ++gi)
#pragma unroll
    for (int e = 0; e < 8; ++e) { rd[gi][e] = 0.f; rc[gi][e] = 0.f; }
#pragma unroll 4
  for (int j = 0; j < nS; ++j) {
    const float a = sm.ca[j], b = sm.cb[j];
    const TW* wr = W + (size_t)sm.S[j] * dcols;
#pragma unroll
    for (int gi = 0; gi < RF_CG; ++gi) {
      const int c0 = (tid + gi * RF_NT) * 8;
      if (c0 < dcols) {
        float w[8];
        RfRow<TW>::load8(wr + c0, w);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          rd[gi][e] = fmaf(a, w[e], rd[gi][e]);
          rc[gi][e] = fmaf(b, w[e], rc[gi][e]);
        }
      }
    }
  }
  double s2d = 0.0, s2c = 0.0;
#pragma unroll
  for (int gi = 0; gi < RF_CG; ++gi)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      s2d += (double)rd[gi][e] * rd[gi][e];
      s2c += (double)rc[gi][e] * rc[gi][e];
    }
  rf_block_sum2(sm, s2d, s2c);
  const double dd = sm.dd, dc = sm.dc, eps = (double)d.eps;
  const double kd = (double)d.w_dist * dd / (sqrt(s2d / dcols) + eps);
  const double kc = (double)d.w_cov * dc / (sqrt(s2c / dcols) + eps);
  float g[RF_CG][8];
  double s2g = 0.0, unused = 0.0;
#pragma unroll
  for (int gi = 0; gi < RF_CG; ++gi)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      g[gi][e] = (float)(kd * rd[gi][e] + kc * rc[gi][e]);
      s2g += (double)g[gi][e] * g[gi][e];
    }
  rf_block_sum2(sm, s2g, unused);
  const float ke = (float)((dd + dc) / (sqrt(s2g / dcols) + eps));
  const bool apply = sm.sev >= (double)d.w_min;
  const float rho = d.rho[hz - 1];
  float* mrow = memory + ((size_t)ti * d.H + (hz - 1)) * dcols;
#pragma unroll
  for (int gi = 0; gi < RF_CG; ++gi) {
    const int c0 = (tid + gi * RF_NT) * 8;
    if (c0 < dcols) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float ev = ke * g[gi][e];
        if (e_out) e_out[(size_t)r * dcols + c0 + e] = ev;
        if (apply) mrow[c0 + e] = rho * mrow[c0 + e] + (1.0f - rho) * ev;
      }
    }
  }
  // ---- delayed alignment: the applied record's feedback sketch against the memory sketch stored at
  // proposal time (Sec. 3.4 "Reliability from delayed alignment"), one-pass moments per slot
  if (align != nullptr && apply) {
    float* al = align + ((size_t)ti * d.H + (hz - 1)) * 4;
    const int rk = d.rank;
    if (rk > 0 && P != nullptr && rec_sketch != nullptr) {
      // sixteen rows at a time: their loads first, then one wave reduction per row
      constexpr int JB = 16;
      for (int j0 = 0; j0 < rk; j0 += JB) {
        float part[JB];
#pragma unroll
        for (int jj = 0; jj < JB; ++jj) {
          const int j = j0 + jj;
          part[jj] = 0.f;
          if (j < rk) {
            const float* pj = P + (size_t)j * dcols;
#pragma unroll
            for (int gi = 0; gi < RF_CG; ++gi) {
              const int c0 = (tid + gi * RF_NT) * 8;
              if (c0 < dcols) {
                float pv[8];
                RfRow<float>::load8(pj + c0, pv);
#pragma unroll
                for (int e = 0; e < 8; ++e) part[jj] = fmaf(pv[e], ke * g[gi][e], part[jj]);
              }
            }
          }
        }
#pragma unroll
        for (int jj = 0; jj < JB; ++jj) {
          const int j = j0 + jj;
          if (j < rk) {
            const double v = wave_sum_f64((double)part[jj]);
            if (lane == 0) sm.xr[wave][j] = v;
          }
        }
      }
      __syncthreads();
      if (tid == 0) {
        double nx = 0.0, ns = 0.0, dot = 0.0;
        const float* sr = rec_sketch + (size_t)r * rk;
        for (int j = 0; j < rk; ++j) {
          double x = 0.0;
          for (int w = 0; w < RF_NW; ++w) x += sm.xr[w][j];
          nx += x * x;
          ns += (double)sr[j] * sr[j];
          dot += (double)sr[j] * x;
        }
        if (nx > 0.0 && ns > 0.0) {
          const double a = dot / sqrt(nx);
          const double n1 = (double)al[0] + 1.0, dl = a - (double)al[1];
          const double mean1 = (double)al[1] + dl / n1;
          al[2] = (float)((double)al[2] + dl * (a - mean1));
          al[1] = (float)mean1;
          al[0] = (float)n1;
        }
      }
    }
    if (tid == 0) al[3] += 1.0f;
  }
  if (tid == 0) {
    st_out[0] = (float)sm.dd;
    st_out[1] = (float)sm.dc;
    st_out[2] = (float)sm.tvs;
    st_out[3] = (float)sm.sev;
    st_out[4] = (float)nS;
    st_out[5] = apply ? 1.f : 0.f;
    st_out[6] = (float)sm.pC;
    st_out[7] = (float)sm.pstar;
  }
}

sr_status launch_reflex_feedback(const sr_reflex_desc& d, const void* target_logits, const int32_t* p_row,
                                 const float* head_logits, const int32_t* q_row, const int32_t* cand,
                                 const int32_t* y_star, const int32_t* traj, const int32_t* horizon, const void* W,
                                 float* memory, float* stats, float* e_out, const float* P, const float* rec_sketch,
                                 float* align, hipStream_t s) {
#define SR_RF_LAUNCH(TP, TW)                                                                                   \
  SR_LAUNCH("sr_reflex_feedback", (k_reflex_feedback<TP, TW>), dim3(d.R), dim3(RF_NT), 0, s,                  \
            (const TP*)target_logits, p_row, head_logits, q_row, cand, y_star, traj, horizon, (const TW*)W,     \
            memory, stats, e_out, P, rec_sketch, align, d)
  if (d.p_dtype == SR_BF16 && d.w_dtype == SR_BF16) {
    SR_RF_LAUNCH(bf16_t, bf16_t);
  } else if (d.p_dtype == SR_BF16) {
    SR_RF_LAUNCH(bf16_t, float);
  } else if (d.w_dtype == SR_BF16) {
    SR_RF_LAUNCH(float, bf16_t);
  } else {
    SR_RF_LAUNCH(float, float);
  }
#undef SR_RF_LAUNCH
  return SR_OK;
}

// ============================================================================ gated correction
// One block per (trajectory, head) row: RMS of z and of the memory, the memory sketch, the reliability
// gate from the alignment moments, and z + alpha RMS(z) m / (RMS(m) + eps) in place (rows the gate keeps
// closed are not written).
constexpr int RC_NT = 256;
constexpr int RC_NW = RC_NT / 64;
constexpr int RC_MAXE = 32;               // d <= RC_NT * RC_MAXE

template <typename T>
__global__ __launch_bounds__(RC_NT) void k_reflex_correct(T* __restrict__ z, const float* __restrict__ memory,
                                                          const float* __restrict__ align, const float* __restrict__ P,
                                                          float* __restrict__ sketch_out, float* __restrict__ alpha_out,
                                                          int H, int d, sr_reflex_gate_desc g) {
  __shared__ double red[RC_NW][2];
  __shared__ double tot[RF_MAXS + 2];
  __shared__ __attribute__((aligned(16))) float ms[RC_NT * RC_MAXE];     // the memory row, for the sketch
  const int row = blockIdx.x, h = row % H;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  T* zr = z + (size_t)row * d;
  const float* mr = memory + (size_t)row * d;
  float zv[RC_MAXE], mv[RC_MAXE];
  double sz = 0.0, sm2 = 0.0;
#pragma unroll
  for (int k = 0; k < RC_MAXE; ++k) {
    const int c = tid + k * RC_NT;
    zv[k] = 0.f;
    mv[k] = 0.f;
    if (c < d) {
      zv[k] = Elem<T>::load(zr, c);
      mv[k] = mr[c];
      ms[c] = mv[k];
    }
    sz += (double)zv[k] * zv[k];
    sm2 += (double)mv[k] * mv[k];
  }
  sz = wave_sum_f64(sz);
  sm2 = wave_sum_f64(sm2);
  if (lane == 0) { red[wave][0] = sz; red[wave][1] = sm2; }
  __syncthreads();
  // sketch rows j = wave, wave + RC_NW, ...: each lane walks the row with all of its wave's rows at once
  const int rk = g.rank;
  constexpr int JPW = (RF_MAXS + RC_NW - 1) / RC_NW;
  float acc[JPW];
#pragma unroll
  for (int jj = 0; jj < JPW; ++jj) acc[jj] = 0.f;
  // four consecutive columns per lane and step, several steps' loads in flight (d is a multiple of 8)
#pragma unroll 4
  for (int c = 4 * lane; c < d; c += 256) {
    const f32x4 mc = *(const f32x4*)(ms + c);
#pragma unroll
    for (int jj = 0; jj < JPW; ++jj) {
      const int j = wave + jj * RC_NW;
      if (j < rk) {
        const f32x4 pv = *(const f32x4*)(P + (size_t)j * d + c);
        acc[jj] = fmaf(pv[0], mc[0], fmaf(pv[1], mc[1], fmaf(pv[2], mc[2], fmaf(pv[3], mc[3], acc[jj]))));
      }
    }
  }
#pragma unroll
  for (int jj = 0; jj < JPW; ++jj) {
    const int j = wave + jj * RC_NW;
    if (j < rk) {                               // uniform over the wave
      const double v = wave_sum_f64((double)acc[jj]);
      if (lane == 0) tot[2 + j] = v;
    }
  }
  if (tid < 2) {
    double a = 0.0;
    for (int w = 0; w < RC_NW; ++w) a += red[w][tid];
    tot[tid] = a;
  }
  __syncthreads();
  const double rms_z = sqrt(tot[0] / d), rms_m = sqrt(tot[1] / d);
  const float* al = align + (size_t)row * 4;
  const double n = al[0], mean = al[1], m2 = al[2], nfb = al[3];
  bool gate = n >= 2.0 && n >= (double)g.n_align_min[h] && nfb >= (double)g.n_fb_min[h] && rms_m > (double)g.m_floor;
  double rel = 0.0;
  if (gate) {
    rel = mean - (double)g.z_delta * sqrt(m2 / (n - 1.0)) / sqrt(n);
    gate = rel > 0.0;
  }
  const double alpha = gate ? (double)g.alpha_min[h] + ((double)g.alpha_max[h] - (double)g.alpha_min[h]) * fmin(rel, 1.0)
                            : 0.0;
  if (gate) {
    const double coef = alpha * rms_z / (rms_m + (double)g.eps);
#pragma unroll
    for (int k = 0; k < RC_MAXE; ++k) {
      const int c = tid + k * RC_NT;
      if (c < d) Elem<T>::store(zr, c, (float)((double)zv[k] + coef * (double)mv[k]));
    }
  }
  if (tid == 0 && alpha_out != nullptr) alpha_out[row] = (float)alpha;
  if (sketch_out != nullptr && rk > 0) {
    double nrm = 0.0;
    for (int j = 0; j < rk; ++j) nrm += tot[2 + j] * tot[2 + j];
    nrm = sqrt(nrm);
    for (int j = tid; j < rk; j += RC_NT) sketch_out[(size_t)row * rk + j] = nrm > 0.0 ? (float)(tot[2 + j] / nrm) : 0.f;
  }
}

sr_status launch_reflex_correct(const sr_heads_desc& d, const sr_reflex_gate_desc& g, void* z, const float* memory,
                                const float* align, const float* P, float* sketch_out, float* alpha_out,
                                hipStream_t s) {
  if (d.dtype == SR_BF16) {
    SR_LAUNCH("sr_reflex_correct", k_reflex_correct<bf16_t>, dim3(d.B * d.H), dim3(RC_NT), 0, s, (bf16_t*)z, memory,
              align, P, sketch_out, alpha_out, d.H, d.d, g);
  } else {
    SR_LAUNCH("sr_reflex_correct", k_reflex_correct<float>, dim3(d.B * d.H), dim3(RC_NT), 0, s, (float*)z, memory,
              align, P, sketch_out, alpha_out, d.H, d.d, g);
  }
  return SR_OK;
}

}  // namespace sr
