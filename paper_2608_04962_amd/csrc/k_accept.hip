// Exact node-wise acceptance walk on gfx950.
//
// Paper: App. B.2 -- Eq. (nodeaccept): candidate y at slot j is accepted with probability
// min(1, r(y)/q_{u,j}(y)); Eq. (noderesidual): after a rejection r <- [r - q_{u,j}]_+ / Z;
// Alg. "Exact node-wise tree verification": an accepted child with children is visited, an
// accepted leaf adds a bonus token from its own target distribution, and a node whose
// children are all rejected ends the round with a fallback token from the final residual.
//
// One block (16 waves) walks one trajectory. At each visited node the block makes a single
// pass over the target-logit row: every wave reduces 512-token chunks to (chunk max, sum of
// exp(logit - chunk max)) in fp32; the chunk sums are combined in float64. The residual is only
// ever different from p on the node's children, so wave 0 keeps it explicitly on the
// children (float64) plus one scalar for the mass outside them; the slot tests and the
// normaliser Z are exact restatements of the full-vocabulary update. Terminal draws walk the
// chunk sums, then one chunk, in token-id order.
//
// With nucleus truncation (top_p < 1) each target row is cut to the smallest prefix, in (logit desc, id
// asc) order, whose mass reaches top_p: a radix select over the order-preserving keys of the logits with
// histograms of the tokens' masses in 40-bit fixed point (integer sums: the same on every run), two
// passes of 11 and 5 bits for bf16 rows and three of 11, 11 and 10 bits for fp32 rows, each counting only
// tokens inside the bin chosen so far. All tokens of the final bin share one logit, so the number of
// them that stay follows from their common mass; when the cut falls inside them, one more pass finds the
// id of the last one kept. The walk then treats every token outside the nucleus as having zero mass; a
// terminal draw first recomputes the chunk sums over the nucleus.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace sr {

constexpr int ACC_NW = 16;
constexpr int ACC_NT = ACC_NW * 64;
constexpr int ACC_CH = 512;                  // tokens per chunk = 64 lanes x 8
constexpr int ACC_MAX_CHUNKS = 512;          // V <= 262144
static_assert(SR_MAX_TREE <= ACC_NT, "one tree node per thread at set-up");
// Row access. A lane's 8 consecutive tokens load as one Raw value (kept packed while in flight: bf16
// rows take half the registers, so a wave keeps GROUP = 8 chunks' loads in flight instead of 4) and
// unpack to fp32 when used; ninf() unpacks to eight -inf (lanes past the row).
template <typename T> struct RowLoad;
template <> struct RowLoad<bf16_t> {
  using Raw = u32x4;
  static constexpr int GROUP = 8;
  static __device__ __forceinline__ Raw raw(const bf16_t* p) { return *(const u32x4*)p; }
  static __device__ __forceinline__ Raw ninf() { return (u32x4){0xff80ff80u, 0xff80ff80u, 0xff80ff80u, 0xff80ff80u}; }
  static __device__ __forceinline__ void unpack(const Raw& w, float* x) {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = bf2f((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xffffu));
  }
  static __device__ __forceinline__ void load8(const bf16_t* p, float* x) { unpack(raw(p), x); }
  static __device__ __forceinline__ float load1(const bf16_t* p) { return bf2f(*p); }
};
template <> struct RowLoad<float> {
  struct Raw { f32x4 a, b; };
  static constexpr int GROUP = 4;
  static __device__ __forceinline__ Raw raw(const float* p) { return Raw{*(const f32x4*)p, *(const f32x4*)(p + 4)}; }
  static __device__ __forceinline__ Raw ninf() {
    const f32x4 n = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    return Raw{n, n};
  }
  static __device__ __forceinline__ void unpack(const Raw& w, float* x) {
#pragma unroll
    for (int e = 0; e < 4; ++e) { x[e] = w.a[e]; x[e + 4] = w.b[e]; }
  }
  static __device__ __forceinline__ void load8(const float* p, float* x) { unpack(raw(p), x); }
  static __device__ __forceinline__ float load1(const float* p) { return *p; }
};

constexpr int NUC_NB = 2048;                 // bins of the first (widest) radix digit
constexpr double NUC_FP = 1099511627776.0;   // 2^40: fixed-point scale of a token's mass (<= 1)

struct AccSmem {
  unsigned long long nh[NUC_NB];             // nucleus radix histogram (fixed-point masses)
  int tie_cnt[ACC_MAX_CHUNKS];
  TreeLds<SR_MAX_TREE> tree;
  int tok[SR_MAX_TREE];
  float cl[SR_MAX_TREE];
  float ua[SR_MAX_TREE];
  float cmax[ACC_MAX_CHUNKS];
  double csum[ACC_MAX_CHUNKS];
  double cscale[ACC_MAX_CHUNKS];
  int kids[SR_MAX_TREE];
  double kpt[SR_MAX_TREE];   // unnormalised target weight of each child's token at the current node
  float kx[SR_MAX_TREE];     // plain walk: each child's logit, taken from the row pass
  int ktok[SR_MAX_TREE];     // the current node's children's tokens (kids order)
  double xsum[ACC_MAX_CHUNKS];         // chunks holding a child: the weight of their other tokens
  unsigned char xflag[ACC_MAX_CHUNKS]; // the chunk holds a child of the current node
  double S;
  double S_out;      // weight of the row outside the current node's children
  int bad;
  int nkid;
  int accepted;      // slot index (0-based) accepted at the current node, -1 = all rejected
  int draw_tok;
  double draw_margin;
  float M;           // row max of logit / temperature
  int nk_on;         // the nucleus cut is active for the current row
  uint32_t nk_key;   // last kept key ...
  int nk_idcut;      // ... and, among the tokens with that key, the last kept id
  double nk_margin;
  unsigned long long nk_above, nk_bin;
  int nk_b;
  int nk_found;
  unsigned long long wtot[ACC_NW];   // per-wave totals of a block scan
  float wred[ACC_NW];        // per-wave partial of a block reduction
};

__device__ __forceinline__ uint32_t acc_key(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ bool nuc_member(const AccSmem& sm, float x, int v) {
  if (!sm.nk_on) return true;
  const uint32_t k = acc_key(x);
  return k > sm.nk_key || (k == sm.nk_key && v <= sm.nk_idcut);
}

// exp(y - m) with y = x * invtau (m finite), as 2^(x (invtau log2 e) - m log2 e) on the hardware
// exponential: one fused multiply-add with both factors rounded to fp32 first, the same at every call
// site, so a token's weight is identical wherever it is recomputed
__device__ __forceinline__ float tilt(float x, float invtau, float m) {
  return __builtin_amdgcn_exp2f(__builtin_fmaf(x, __fmul_rn(invtau, kLog2e), -__fmul_rn(m, kLog2e)));
}

// Row pass of the plain walk. With m > 0 (the node's children in sm.kids, their chunks flagged in xflag)
// the same pass also sums each flagged chunk over its tokens other than the children -- exactly what
// outside_mass would sum, from the same loaded values -- and keeps the children's logits in sm.kx; the
// final combine then sets xsum (scaled) and S_out as outside_mass does.
template <typename T>
__device__ void row_stats(AccSmem& sm, const T* __restrict__ row, int V, float invtau, int m_kids) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nch = (V + ACC_CH - 1) / ACC_CH;
  constexpr int GRP = RowLoad<T>::GROUP;
  for (int c0 = wave * GRP; c0 < nch; c0 += ACC_NW * GRP) {
    typename RowLoad<T>::Raw w[GRP];
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) {
      const int base = (c0 + gi) * ACC_CH + lane * 8;
      w[gi] = (c0 + gi < nch && base < V) ? RowLoad<T>::raw(row + base) : RowLoad<T>::ninf();
    }
    // the group's chunk flags in one LDS read (byte gi: chunk c0 + gi holds a child; entries past nch are
    // never tested)
    unsigned long long gflags = 0;
    if (m_kids > 0) {
      if constexpr (GRP == 8) gflags = *(const unsigned long long*)&sm.xflag[c0];
      else gflags = *(const uint32_t*)&sm.xflag[c0];
    }
    // One reference max for the GRP chunks of this group: their max of x * invtau (rounding is monotone,
    // so the max of the raw logits times invtau > 0 is the max of the products). Every consumer weighs a
    // token of chunk c against cmax[c], so a shared reference only has to be stored per chunk; a token
    // more than ~87 below it (probability < 1e-37) underflows to weight 0.
    float ml = -INFINITY;
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) {
      float x[8];
      RowLoad<T>::unpack(w[gi], x);
#pragma unroll
      for (int e = 0; e < 8; ++e) ml = fmaxf(ml, x[e]);
    }
    const float m = __fmul_rn(wave_max_f32(ml), invtau);
    float a[GRP];                               // this lane's part of each chunk sum: 8 terms in (0, 1]
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) a[gi] = 0.f;
    if (m != -INFINITY) {                       // uniform; a -inf token then weighs 2^-inf = 0
#pragma unroll
      for (int gi = 0; gi < GRP; ++gi) {
        float x[8];
        RowLoad<T>::unpack(w[gi], x);
#pragma unroll
        for (int e = 0; e < 8; ++e) a[gi] += tilt(x[e], invtau, m);
      }
    }
    // the GRP chunk sums over the wave at once: each exchange halves the values a lane holds, then the
    // lanes that share a chunk finish with a plain butterfly; chunk j's total lands in lanes 64/GRP j ..
    int j;
    const float s = wave_sum_scatter<GRP>(a, j);
    if ((lane & (64 / GRP - 1)) == 0 && c0 + j < nch) { sm.cmax[c0 + j] = m; sm.csum[c0 + j] = (double)s; }
    if (m_kids > 0 && gflags != 0) {
#pragma unroll
      for (int gi = 0; gi < GRP; ++gi) {
        const int c = c0 + gi;
        if (c >= nch || ((gflags >> (8 * gi)) & 0xffu) == 0) continue;   // uniform per wave
        const int base = c * ACC_CH + lane * 8;
        float x[8];
        RowLoad<T>::unpack(w[gi], x);
        unsigned excl = 0;                        // this lane's tokens that are children
        for (int k = 0; k < m_kids; ++k) {
          const int v = sm.ktok[k];
          if (v >= base && v < base + 8) {
            excl |= 1u << (v - base);
            sm.kx[k] = x[v - base];
          }
        }
        double xs = 0.0;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (!((excl >> e) & 1u) && x[e] != -INFINITY) xs += (double)tilt(x[e], invtau, m);
        xs = wave_sum_f64(xs);
        if (lane == 0) sm.xsum[c] = xs;           // scaled by cscale[c] below
      }
    }
  }
  __syncthreads();
  if (wave == 0) {
    float ml = -INFINITY;
    for (int c = lane; c < nch; c += 64) ml = fmaxf(ml, sm.cmax[c]);
    const float M = wave_max_f32(ml);
    double sl = 0.0, so = 0.0;
    for (int c = lane; c < nch; c += 64) {
      const double sc = exp((double)sm.cmax[c] - (double)M);
      sm.cscale[c] = sc;
      const double a = sm.csum[c] * sc;
      sl += a;
      if (m_kids > 0 && sm.xflag[c]) {
        const double xs = sm.xsum[c] * sc;
        sm.xsum[c] = xs;
        so += xs;
      } else {
        so += a;
      }
    }
    const double S = wave_sum_f64(sl);
    const double So = wave_sum_f64(so);
    if (lane == 0) { sm.S = S; sm.S_out = So; sm.M = M; sm.nk_on = 0; }
  }
  __syncthreads();
}

// unnormalised target weight of token v under the current row statistics
template <typename T>
__device__ __forceinline__ double ptilde(const AccSmem& sm, const T* row, int v, float invtau) {
  const int c = v / ACC_CH;
  const float x = RowLoad<T>::load1(row + v);
  if (x == -INFINITY || !nuc_member(sm, x, v)) return 0.0;
  return (double)tilt(x, invtau, sm.cmax[c]) * sm.cscale[c];
}

// ---- nucleus truncation
// floor(w 2^40) for a weight w in [0, 1], from the float's bits: w 2^40 = m 2^e with m the 24-bit significand
// (the same value as the float64 product truncated, without the conversions)
__device__ __forceinline__ unsigned long long nuc_fixed(float w) {
  const uint32_t u = __float_as_uint(w);
  const int e = (int)(u >> 23) - 110;
  const unsigned long long m = (unsigned long long)((u & 0x7fffffu) | 0x800000u);
  return e >= 0 ? (m << e) : (e > -24 ? (m >> -e) : 0ull);
}

// Histogram of the fixed-point masses of the tokens whose key matches prefix under pmask, by key digit
// (key >> sh) & dmask. Whole block.
template <typename T>
__device__ void nuc_hist(AccSmem& sm, const T* __restrict__ row, int V, float invtau, uint32_t prefix,
                         uint32_t pmask, int sh, uint32_t dmask) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nch = (V + ACC_CH - 1) / ACC_CH;
  const float M = sm.M;
  for (int i = tid; i < NUC_NB; i += ACC_NT) sm.nh[i] = 0ull;
  __syncthreads();
  constexpr int GRP = RowLoad<T>::GROUP;
  for (int c0 = wave * GRP; c0 < nch; c0 += ACC_NW * GRP) {
    typename RowLoad<T>::Raw w[GRP];
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) {
      const int base = (c0 + gi) * ACC_CH + lane * 8;
      w[gi] = (c0 + gi < nch && base < V) ? RowLoad<T>::raw(row + base) : RowLoad<T>::ninf();
    }
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) {
      float x[8];
      RowLoad<T>::unpack(w[gi], x);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float xv = x[e];
        const uint32_t k = acc_key(xv);
        if (xv != -INFINITY && (k & pmask) == prefix)
          atomicAdd(&sm.nh[(k >> sh) & dmask], nuc_fixed(tilt(xv, invtau, M)));
      }
    }
  }
  __syncthreads();
}

// Wave 0: among bins [0, nb) in descending order, the bin b with above + (bins > b) < target <=
// above + (bins >= b); sets sm.nk_b, sm.nk_above (mass ranked before the bin) and sm.nk_bin (its mass).
__device__ void nuc_find(AccSmem& sm, int nb, unsigned long long above, unsigned long long target) {
  const int lane = threadIdx.x & 63;
  const int per = (nb + 63) / 64;                 // lane l owns bins nb-1-l*per down to nb-(l+1)*per
  unsigned long long ls = 0;
  for (int j = 0; j < per; ++j) {
    const int b = nb - 1 - lane * per - j;
    if (b >= 0) ls += sm.nh[b];
  }
  // exclusive prefix over lanes (lane 0 holds the top bins)
  unsigned long long incl = ls;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const unsigned long long t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  const unsigned long long before = above + (incl - ls);
  const bool mine = before < target && target <= before + ls;
  const unsigned long long bal = __ballot(mine);
  const int owner = bal ? __ffsll((long long)bal) - 1 : 63;
  if (lane == owner) {
    unsigned long long cum = before;
    int bsel = max(0, nb - 1 - lane * per - (per - 1));
    unsigned long long msel = 0, asel = cum;
    for (int j = 0; j < per; ++j) {
      const int b = nb - 1 - lane * per - j;
      if (b < 0) break;
      const unsigned long long m = sm.nh[b];
      if (cum < target && target <= cum + m) { bsel = b; msel = m; asel = cum; break; }
      cum += m;
    }
    sm.nk_b = bsel;
    sm.nk_above = asel;
    sm.nk_bin = msel;
  }
}

// The first `want` tokens (in id order) whose key equals kstar: the id of the last of them. Whole block;
// the result is in sm.nk_idcut.
template <typename T>
__device__ void nuc_tie_cut(AccSmem& sm, const T* __restrict__ row, int V, uint32_t kstar, int want) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nch = (V + ACC_CH - 1) / ACC_CH;
  for (int c = wave; c < nch; c += ACC_NW) {
    const int base = c * ACC_CH + lane * 8;
    int n = 0;
    if (base < V) {
      float x[8];
      RowLoad<T>::load8(row + base, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) n += (x[e] != -INFINITY && acc_key(x[e]) == kstar) ? 1 : 0;
    }
    n = warp_sum_i(n);
    if (lane == 0) sm.tie_cnt[c] = n;
  }
  __syncthreads();
  if (wave == 0) {
    constexpr int CPL = ACC_MAX_CHUNKS / 64;
    int cnt[CPL], ls = 0;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = lane * CPL + i;
      cnt[i] = c < nch ? sm.tie_cnt[c] : 0;
      ls += cnt[i];
    }
    int incl = ls;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(incl, o, 64);
      if (lane >= o) incl += t;
    }
    int before = incl - ls, cstar = -1, cbefore = 0;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      if (cstar < 0 && before < want && want <= before + cnt[i]) { cstar = lane * CPL + i; cbefore = before; }
      before += cnt[i];
    }
    const unsigned long long bal = __ballot(cstar >= 0);
    const int owner = bal ? __ffsll((long long)bal) - 1 : 0;
    cstar = max(0, __shfl(cstar, owner, 64));
    cbefore = __shfl(cbefore, owner, 64);
    // scan the chunk: 8 tokens per lane
    const int base = cstar * ACC_CH + lane * 8;
    float x[8];
    int n = 0;
    if (base < V) {
      RowLoad<T>::load8(row + base, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) n += (x[e] != -INFINITY && acc_key(x[e]) == kstar) ? 1 : 0;
    }
    int li = n;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(li, o, 64);
      if (lane >= o) li += t;
    }
    int cum = cbefore + li - n, id = -1;
    if (base < V) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (x[e] != -INFINITY && acc_key(x[e]) == kstar) {
          ++cum;
          if (cum == want && id < 0) id = base + e;
        }
      }
    }
    const unsigned long long b2 = __ballot(id >= 0);
    const int idv = __shfl(id, b2 ? __ffsll((long long)b2) - 1 : 0, 64);
    if (lane == 0 && b2) sm.nk_idcut = idv;
  }
  __syncthreads();
}

// Row statistics for the nucleus path, relative to the row max itself: a first pass takes the max, a
// second computes each token's weight once, for both the chunk sums (cmax[c] = M, cscale[c] = 1) and the
// first digit of the nucleus histogram (the masses nuc_hist's first pass adds, in the same fixed point).
// Leaves what row_stats leaves, plus that histogram. Whole block.
// hc: NUC_HC copies of the first digit's histogram, lane l adding to copy l mod NUC_HC (a quarter of the
// same-address collisions of one atomic instruction), summed into sm.nh at the end; null: sm.nh directly
constexpr int NUC_HC = 4;
template <typename T>
__device__ __attribute__((noinline)) void row_stats_nuc(AccSmem& sm, const T* __restrict__ row, int V, float invtau,
                                                        unsigned long long* __restrict__ hc) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nch = (V + ACC_CH - 1) / ACC_CH;
  constexpr int GRP = RowLoad<T>::GROUP;
  if (hc != nullptr) {
    for (int i = tid; i < NUC_HC * NUC_NB; i += ACC_NT) hc[i] = 0ull;
  } else {
    for (int i = tid; i < NUC_NB; i += ACC_NT) sm.nh[i] = 0ull;
  }
  unsigned long long* hist = hc != nullptr ? hc + (lane & (NUC_HC - 1)) * NUC_NB : sm.nh;
  auto load_group = [&](int c0, typename RowLoad<T>::Raw (&w)[GRP]) {
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) {
      const int base = (c0 + gi) * ACC_CH + lane * 8;
      w[gi] = (c0 + gi < nch && base < V) ? RowLoad<T>::raw(row + base) : RowLoad<T>::ninf();
    }
  };
  float ml = -INFINITY;
  for (int c0 = wave * GRP; c0 < nch; c0 += ACC_NW * GRP) {
    typename RowLoad<T>::Raw w[GRP];
    load_group(c0, w);
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) {
      float x[8];
      RowLoad<T>::unpack(w[gi], x);
#pragma unroll
      for (int e = 0; e < 8; ++e) ml = fmaxf(ml, x[e]);
    }
  }
  ml = wave_max_f32(ml);
  if (lane == 0) sm.wred[wave] = ml;
  __syncthreads();
  float mx = -INFINITY;
#pragma unroll
  for (int w = 0; w < ACC_NW; ++w) mx = fmaxf(mx, sm.wred[w]);
  const float M = __fmul_rn(mx, invtau);         // the max of x * invtau (rounding is monotone)
  for (int c0 = wave * GRP; c0 < nch; c0 += ACC_NW * GRP) {
    typename RowLoad<T>::Raw w[GRP];
    load_group(c0, w);
    float a[GRP];
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) a[gi] = 0.f;
    if (M != -INFINITY) {                        // uniform
#pragma unroll
      for (int gi = 0; gi < GRP; ++gi) {
        float x[8];
        RowLoad<T>::unpack(w[gi], x);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float wt = tilt(x[e], invtau, M);
          a[gi] += wt;
          if (x[e] != -INFINITY) atomicAdd(&hist[acc_key(x[e]) >> 21], nuc_fixed(wt));
        }
      }
    }
    int j;
    const float sc = wave_sum_scatter<GRP>(a, j);
    if ((lane & (64 / GRP - 1)) == 0 && c0 + j < nch) { sm.cmax[c0 + j] = M; sm.csum[c0 + j] = (double)sc; }
  }
  __syncthreads();
  if (hc != nullptr) {                          // integer sums: the copies add up exactly
    for (int i = tid; i < NUC_NB; i += ACC_NT) {
      unsigned long long t = 0;
#pragma unroll
      for (int k = 0; k < NUC_HC; ++k) t += hc[k * NUC_NB + i];
      sm.nh[i] = t;
    }
  }
  if (wave == 0) {
    double sl = 0.0;
    for (int c = lane; c < nch; c += 64) {
      sm.cscale[c] = 1.0;
      sl += sm.csum[c];
    }
    const double S = wave_sum_f64(sl);
    if (lane == 0) { sm.S = S; sm.M = M; sm.nk_on = 0; }
  }
  __syncthreads();
}

// Nucleus cut of the current row (after row_stats_nuc): membership fields of sm, sm.S = the nucleus mass
// and sm.nk_margin. Whole block.
template <typename T>
__device__ __attribute__((noinline)) void nucleus(AccSmem& sm, const T* __restrict__ row, int V, float invtau, float top_p) {
  // the first digit's histogram comes from row_stats_nuc
  const int tid = threadIdx.x, wave = tid >> 6;
  constexpr bool BF = sizeof(T) == 2;
  constexpr int NP = BF ? 2 : 3;
  const int shs[3] = {21, BF ? 16 : 10, 0};
  const int bits[3] = {11, BF ? 5 : 11, 10};
  uint32_t prefix = 0, pmask = 0;
  unsigned long long above = 0, target = 0, total = 0;
  for (int pass = 0; pass < NP; ++pass) {
    const uint32_t dmask = (1u << bits[pass]) - 1u;
    if (pass > 0) nuc_hist<T>(sm, row, V, invtau, prefix, pmask, shs[pass], dmask);
    if (pass == 0) {
      // total mass and the integer target: a token stays iff the mass ranked before it is < top_p * total
      if (wave == 0) {
        unsigned long long ls = 0;
        for (int b = threadIdx.x; b < NUC_NB; b += 64) ls += sm.nh[b];
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) ls += __shfl_xor(ls, o, 64);
        if (threadIdx.x == 0) {
          sm.nk_above = ls;                       // stash the total
        }
      }
      __syncthreads();
      total = sm.nk_above;
      target = (unsigned long long)ceil((double)top_p * (double)total);
      __syncthreads();
    }
    if (wave == 0) nuc_find(sm, 1 << bits[pass], above, target);
    __syncthreads();
    above = sm.nk_above;
    prefix |= (uint32_t)sm.nk_b << shs[pass];
    pmask |= dmask << shs[pass];
    __syncthreads();
  }
  // every token of the final bin has one key and the same mass q. A bf16 value widened to fp32 has 16 zero
  // low bits, so its key's low bits are all zero (positive) or all one (negative): complete the key.
  if (BF && !(prefix & 0x80000000u)) prefix |= 0xffffu;
  const unsigned long long bin_mass = sm.nk_bin;
  // the mass of one such token, recomputed from its value
  const uint32_t u = (prefix & 0x80000000u) ? (prefix & 0x7fffffffu) : ~prefix;
  const float xk = __uint_as_float(u);
  const unsigned long long q = nuc_fixed(tilt(xk, invtau, sm.M));
  const unsigned long long n_tie = q > 0 ? bin_mass / q : 1;
  // tokens t = 0.. of the bin stay while above + t q < target
  const unsigned long long need = q > 0 ? (target - above + q - 1) / q : n_tie;
  const unsigned long long kt = need < n_tie ? need : n_tie;
  if (tid == 0) {
    sm.nk_key = prefix;
    sm.nk_idcut = 0x7fffffff;
    const double bl = (double)(above + (kt - 1) * q), bh = bl + (double)q, tg = (double)top_p * (double)total;
    sm.nk_margin = fmin(tg - bl, bh - tg) / (double)total;
    sm.S = (double)(above + kt * q) / NUC_FP;
  }
  __syncthreads();
  if (kt < n_tie) nuc_tie_cut<T>(sm, row, V, prefix, (int)kt);
  if (tid == 0) sm.nk_on = 1;
  __syncthreads();
}

// Boundary-bin tallies of the fused nucleus pass (bf16 rows): per chunk and second key digit, the summed
// weight (fp32; every cell is updated by the one wave that owns its chunk) and the token count (two 16-bit
// counts per word; a chunk holds at most 512 tokens).
constexpr int NUC_D2 = 32;                   // values of the second digit of a bf16 key (bits 16..20)
struct alignas(16) NucBins {
  float bm[ACC_MAX_CHUNKS * NUC_D2];
  uint32_t bc[ACC_MAX_CHUNKS * NUC_D2 / 2];
};
static_assert(sizeof(NucBins) >= NUC_HC * NUC_NB * sizeof(unsigned long long), "histogram copies fit the bins");
// the bf16 nucleus pass's bins, which also hold the histogram copies of row_stats_nuc (used one after the other)
__device__ __forceinline__ NucBins& nuc_bins() {
  __shared__ NucBins nb;
  return nb;
}
__device__ __forceinline__ int nuc_bcount(const NucBins& nb, int c, int d) {
  return (int)((nb.bc[c * (NUC_D2 / 2) + (d >> 1)] >> (16 * (d & 1))) & 0xffffu);
}

// The nucleus cut of a bf16 row and its masked chunk sums in one pass over the row (after row_stats_nuc),
// in place of nucleus + nuc_masked_sums. A bf16 key is fixed by its top 16 bits: the first digit (bits
// 21..31) comes from row_stats_nuc's histogram, the second (bits 16..20) from this pass. Knowing the first
// digit's cut bin b1, the pass sums per chunk the weights of the tokens above b1 (members whatever the
// second digit), and tallies the tokens of bin b1 by chunk and second digit (weight and count) beside the
// second digit's histogram. Once the second digit d2 is found, a chunk's nucleus sum is its sum above b1,
// plus its bin-b1 weight of digits above d2, plus its kept tokens of the cut key (all of one weight).
// The cut itself (key, id cut, mass, margin) is computed exactly as nucleus computes it.
__device__ __attribute__((noinline)) void nucleus_bf16(AccSmem& sm, NucBins& nb, const bf16_t* __restrict__ row, int V, float invtau,
                             float top_p) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nch = (V + ACC_CH - 1) / ACC_CH;
  // total mass, target and the first digit's cut bin, from row_stats_nuc's histogram: one block scan with
  // the bins in descending order (thread t holds bins NUC_NB-1-2t and NUC_NB-2-2t); the bin found is the one
  // nuc_find would find over all NUC_NB bins
  static_assert(NUC_NB == 2 * ACC_NT, "two bins per thread");
  const int bhi = NUC_NB - 1 - 2 * tid;
  const unsigned long long m0 = sm.nh[bhi], m1 = sm.nh[bhi - 1], v01 = m0 + m1;
  unsigned long long incl = v01;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const unsigned long long t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  if (lane == 63) sm.wtot[wave] = incl;
  if (tid == 0) sm.nk_found = 0;
  __syncthreads();
  unsigned long long total = 0, wbefore = 0;
#pragma unroll
  for (int w = 0; w < ACC_NW; ++w) {
    const unsigned long long t = sm.wtot[w];
    total += t;
    wbefore += w < wave ? t : 0ull;
  }
  const unsigned long long target = (unsigned long long)ceil((double)top_p * (double)total);
  {
    const unsigned long long before = wbefore + incl - v01;   // mass of the bins above bhi
    if (before < target && target <= before + m0) {
      sm.nk_b = bhi; sm.nk_above = before; sm.nk_bin = m0; sm.nk_found = 1;
    } else if (before + m0 < target && target <= before + v01) {
      sm.nk_b = bhi - 1; sm.nk_above = before + m0; sm.nk_bin = m1; sm.nk_found = 1;
    }
  }
  __syncthreads();
  if (tid == 0 && !sm.nk_found) { sm.nk_b = 0; sm.nk_above = 0ull; sm.nk_bin = 0ull; }   // an empty row
  __syncthreads();
  const uint32_t b1 = (uint32_t)sm.nk_b;
  const unsigned long long above1 = sm.nk_above;
  for (int i = tid; i < nch * NUC_D2; i += ACC_NT) nb.bm[i] = 0.f;
  for (int i = tid; i < nch * (NUC_D2 / 2); i += ACC_NT) nb.bc[i] = 0u;
  __syncthreads();                            // every thread has read nk_b / nk_above before nh is reused
  for (int i = tid; i < NUC_D2; i += ACC_NT) sm.nh[i] = 0ull;
  __syncthreads();
  const float M = sm.M;
  constexpr int GRP = RowLoad<bf16_t>::GROUP;
  for (int c0 = wave * GRP; c0 < nch; c0 += ACC_NW * GRP) {
    RowLoad<bf16_t>::Raw w[GRP];
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) {
      const int base = (c0 + gi) * ACC_CH + lane * 8;
      w[gi] = (c0 + gi < nch && base < V) ? RowLoad<bf16_t>::raw(row + base) : RowLoad<bf16_t>::ninf();
    }
    float a[GRP];                              // this lane's weight above bin b1, per chunk
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) {
      a[gi] = 0.f;
      const int c = min(c0 + gi, nch - 1);     // past the row every token is -inf and tallies nothing
      float x[8];
      RowLoad<bf16_t>::unpack(w[gi], x);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t k = acc_key(x[e]);
        const uint32_t d1 = k >> 21;
        if (x[e] != -INFINITY && d1 >= b1) {
          const float wt = tilt(x[e], invtau, M);
          if (d1 > b1) {
            a[gi] += wt;
          } else {
            const int d = (int)((k >> 16) & (NUC_D2 - 1));
            atomicAdd(&nb.bm[c * NUC_D2 + d], wt);
            atomicAdd(&nb.bc[c * (NUC_D2 / 2) + (d >> 1)], 1u << (16 * (d & 1)));
            atomicAdd(&sm.nh[d], nuc_fixed(wt));
          }
        }
      }
    }
    int j;
    const float sc = wave_sum_scatter<GRP>(a, j);
    if ((lane & (64 / GRP - 1)) == 0 && c0 + j < nch) sm.csum[c0 + j] = (double)sc;
  }
  __syncthreads();
  if (wave == 0) nuc_find(sm, NUC_D2, above1, target);
  __syncthreads();
  const int d2 = sm.nk_b;
  const unsigned long long above = sm.nk_above, bin_mass = sm.nk_bin;
  uint32_t prefix = (b1 << 21) | ((uint32_t)d2 << 16);
  // a bf16 value widened to fp32 has 16 zero low bits: the key's low bits are all zero (positive) or all one
  // (negative)
  if (!(prefix & 0x80000000u)) prefix |= 0xffffu;
  const uint32_t u = (prefix & 0x80000000u) ? (prefix & 0x7fffffffu) : ~prefix;
  const float xk = __uint_as_float(u);
  const float wk = tilt(xk, invtau, M);       // the weight of every token with the cut key
  const unsigned long long q = nuc_fixed(wk);
  const unsigned long long n_tie = q > 0 ? bin_mass / q : 1;
  const unsigned long long need = q > 0 ? (target - above + q - 1) / q : n_tie;
  const unsigned long long kt = need < n_tie ? need : n_tie;
  if (tid == 0) {
    sm.nk_key = prefix;
    sm.nk_idcut = 0x7fffffff;
    const double bl = (double)(above + (kt - 1) * q), bh = bl + (double)q, tg = (double)top_p * (double)total;
    sm.nk_margin = fmin(tg - bl, bh - tg) / (double)total;
    sm.S = (double)(above + kt * q) / NUC_FP;
  }
  // chunk holding the last kept token of the cut key and the kept ones before it, from the tallies (wave 0)
  int cstar = nch, cbefore = 0;
  if (kt < n_tie && wave == 0) {
    constexpr int CPL = ACC_MAX_CHUNKS / 64;
    const int want = (int)kt;
    int cnt[CPL], ls = 0;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = lane * CPL + i;
      cnt[i] = c < nch ? nuc_bcount(nb, c, d2) : 0;
      ls += cnt[i];
    }
    int incl = ls;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(incl, o, 64);
      if (lane >= o) incl += t;
    }
    int before = incl - ls, cs = -1, cb = 0;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      if (cs < 0 && before < want && want <= before + cnt[i]) { cs = lane * CPL + i; cb = before; }
      before += cnt[i];
    }
    const unsigned long long bal = __ballot(cs >= 0);
    const int owner = bal ? __ffsll((long long)bal) - 1 : 0;
    cstar = max(0, __shfl(cs, owner, 64));
    cbefore = __shfl(cb, owner, 64);
    // the id of the want-th token of the cut key: scan chunk cstar, 8 tokens per lane
    const int base = cstar * ACC_CH + lane * 8;
    float x[8];
    int n = 0;
    if (base < V) {
      RowLoad<bf16_t>::load8(row + base, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) n += (x[e] != -INFINITY && acc_key(x[e]) == prefix) ? 1 : 0;
    }
    int li = n;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(li, o, 64);
      if (lane >= o) li += t;
    }
    int cum = cbefore + li - n, id = -1;
    if (base < V) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (x[e] != -INFINITY && acc_key(x[e]) == prefix) {
          ++cum;
          if (cum == want && id < 0) id = base + e;
        }
      }
    }
    const unsigned long long b2 = __ballot(id >= 0);
    const int idv = __shfl(id, b2 ? __ffsll((long long)b2) - 1 : 0, 64);
    if (lane == 0) {
      if (b2) sm.nk_idcut = idv;
      sm.nk_b = cstar;                          // handed to the masked sums below
      sm.nk_bin = (unsigned long long)cbefore;
    }
  }
  __syncthreads();
  if (kt < n_tie) { cstar = sm.nk_b; cbefore = (int)sm.nk_bin; }
  // masked chunk sums: above b1, plus bin b1's digits above d2, plus the kept tokens of the cut key
  for (int c = tid; c < nch; c += ACC_NT) {
    double sum = sm.csum[c];
    for (int d = d2 + 1; d < NUC_D2; ++d) sum += (double)nb.bm[c * NUC_D2 + d];
    const int nt = nuc_bcount(nb, c, d2);
    const int kept = c < cstar ? nt : (c == cstar ? (int)kt - cbefore : 0);
    sm.csum[c] = sum + (double)kept * (double)wk;
  }
  if (tid == 0) sm.nk_on = 1;
  __syncthreads();
}

// chunk sums restricted to the nucleus (for the terminal draws), relative to the chunks' reference
// maxima; the same chunk groups and exchanges as row_stats
template <typename T>
__device__ __attribute__((noinline)) void nuc_masked_sums(AccSmem& sm, const T* __restrict__ row, int V, float invtau) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nch = (V + ACC_CH - 1) / ACC_CH;
  constexpr int GRP = RowLoad<T>::GROUP;
  for (int c0 = wave * GRP; c0 < nch; c0 += ACC_NW * GRP) {
    typename RowLoad<T>::Raw w[GRP];
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) {
      const int base = (c0 + gi) * ACC_CH + lane * 8;
      w[gi] = (c0 + gi < nch && base < V) ? RowLoad<T>::raw(row + base) : RowLoad<T>::ninf();
    }
    float a[GRP];
#pragma unroll
    for (int gi = 0; gi < GRP; ++gi) {
      a[gi] = 0.f;
      if (c0 + gi < nch) {                      // uniform
        const int base = (c0 + gi) * ACC_CH + lane * 8;
        const float m = sm.cmax[c0 + gi];
        float x[8];
        RowLoad<T>::unpack(w[gi], x);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (x[e] != -INFINITY && nuc_member(sm, x[e], base + e)) a[gi] += tilt(x[e], invtau, m);
      }
    }
    int j;
    const float s = wave_sum_scatter<GRP>(a, j);
    if ((lane & (64 / GRP - 1)) == 0 && c0 + j < nch) sm.csum[c0 + j] = (double)s;
  }
  __syncthreads();
}

// Weight of the current row outside the node's m children (sm.kids), chunk by chunk. A chunk that holds a
// child is summed again over its other tokens: its chunk sum minus the children's weights would keep only
// fp32 rounding of the remainder when the children hold most of the chunk (peaked rows). Sets xflag and
// xsum of those chunks and sm.S_out; with the nucleus cut also sm.S, the sum of the (nucleus-masked) chunk
// sums. Whole block.
template <typename T, bool NUC>
__device__ void outside_mass(AccSmem& sm, const T* __restrict__ row, int V, float invtau, int m) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nch = (V + ACC_CH - 1) / ACC_CH;
  for (int c = tid; c < nch; c += ACC_NT) sm.xflag[c] = 0;
  __syncthreads();
  for (int k = tid; k < m; k += ACC_NT) sm.xflag[sm.tok[sm.kids[k]] / ACC_CH] = 1;
  __syncthreads();
  for (int k = wave; k < m; k += ACC_NW) {
    const int c = sm.tok[sm.kids[k]] / ACC_CH;
    bool first = true;                           // the first child of its chunk sums it
    for (int k2 = 0; k2 < k; ++k2)
      if (sm.tok[sm.kids[k2]] / ACC_CH == c) { first = false; break; }
    if (!first) continue;                        // uniform per wave
    const int base = c * ACC_CH + lane * 8;
    unsigned excl = 0;                           // this lane's tokens that are children
    for (int k2 = 0; k2 < m; ++k2) {
      const int v = sm.tok[sm.kids[k2]];
      if (v >= base && v < base + 8) excl |= 1u << (v - base);
    }
    double s = 0.0;
    if (base < V) {                              // V is a multiple of 8: all 8 tokens are in the row
      float x[8];
      RowLoad<T>::load8(row + base, x);
      const float cm = sm.cmax[c];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (!((excl >> e) & 1u) && x[e] != -INFINITY && nuc_member(sm, x[e], base + e))
          s += (double)tilt(x[e], invtau, cm);
    }
    s = wave_sum_f64(s);
    if (lane == 0) sm.xsum[c] = s * sm.cscale[c];
  }
  __syncthreads();
  if (wave == 0) {
    double so = 0.0, st = 0.0;
    for (int c = lane; c < nch; c += 64) {
      const double a = sm.csum[c] * sm.cscale[c];
      st += a;
      so += sm.xflag[c] ? sm.xsum[c] : a;
    }
    so = wave_sum_f64(so);
    st = wave_sum_f64(st);
    if (lane == 0) {
      sm.S_out = so;
      if (NUC) sm.S = st;
    }
  }
  __syncthreads();
}

// Inverse-CDF draw over the current row, token-id order, excluding the tokens of
// sm.kids[0..n_excl) (whose chunks' remaining weights outside_mass left in xsum). Run by wave 0; result in
// sm.draw_tok / sm.draw_margin.
template <typename T>
__device__ void draw(AccSmem& sm, const T* __restrict__ row, int V, float invtau, int n_excl, float U) {
  const int lane = threadIdx.x & 63;
  const int nch = (V + ACC_CH - 1) / ACC_CH;
  // excluded mass per chunk is subtracted from that chunk's sum
  constexpr int CPL = ACC_MAX_CHUNKS / 64;     // chunks per lane, consecutive
  double adj[CPL];
  double lsum = 0.0;
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int c = lane * CPL + i;
    double a = 0.0;
    if (c < nch) a = (n_excl > 0 && sm.xflag[c]) ? sm.xsum[c] : sm.csum[c] * sm.cscale[c];
    adj[i] = a;
    lsum += a;
  }
  // exclusive prefix over lanes
  double incl = lsum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  const double Sp = __shfl(incl, 63, 64);
  double before = incl - lsum;
  const double target = (double)U * Sp;
  // first chunk whose cumulative sum exceeds the target
  int cstar = 1 << 30;
  double cbefore = 0.0;
  {
    double cum = before;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = lane * CPL + i;
      if (c < nch && cstar == (1 << 30) && target < cum + adj[i]) { cstar = c; cbefore = cum; }
      cum += adj[i];
    }
  }
  int cfirst = warp_min_i(cstar);
  if (cfirst == (1 << 30)) {                  // rounding at the very top: last chunk with mass
    int lastc = -1;
#pragma unroll
    for (int i = 0; i < CPL; ++i)
      if (lane * CPL + i < nch && adj[i] > 0.0) lastc = lane * CPL + i;
    for (int o = 32; o > 0; o >>= 1) lastc = max(lastc, __shfl_xor(lastc, o, 64));
    cfirst = max(lastc, 0);
    // cumulative mass before that chunk
    double cb = 0.0;
    double cum = before;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      if (lane * CPL + i == cfirst) cb = cum;
      cum += adj[i];
    }
    cstar = (lane * CPL <= cfirst && cfirst < lane * CPL + CPL) ? cfirst : (1 << 30);
    cbefore = cb;
  }
  // broadcast the cumulative mass before the chosen chunk from its owner lane
  const int owner = cfirst / CPL;
  const double cb = __shfl(cbefore, owner, 64);
  // scan the chosen chunk: 8 tokens per lane
  double w[8];
  double wl = 0.0;
  const int base = cfirst * ACC_CH + lane * 8;
  unsigned excl = 0;                            // this lane's tokens that are excluded children
  for (int k = 0; k < n_excl; ++k) {
    const int v = sm.tok[sm.kids[k]];
    if (v >= base && v < base + 8) excl |= 1u << (v - base);
  }
  float xs[8];
  if (base < V) {
    RowLoad<T>::load8(row + base, xs);          // V is a multiple of 8: all 8 tokens are in the row
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) xs[e] = -INFINITY;
  }
  const float cm = sm.cmax[cfirst];
  const double csc = sm.cscale[cfirst];
#pragma unroll
  for (int e = 0; e < 8; ++e) {               // ptilde of token base + e, from the loaded values
    const int v = base + e;
    double pv = 0.0;
    if (!((excl >> e) & 1u) && xs[e] != -INFINITY && nuc_member(sm, xs[e], v))
      pv = (double)tilt(xs[e], invtau, cm) * csc;
    w[e] = pv;
    wl += pv;
  }
  double li = wl;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double t = __shfl_up(li, o, 64);
    if (lane >= o) li += t;
  }
  double cum = cb + (li - wl);
  int pick = 1 << 30;
  double lo = 0.0, hi = 0.0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const double nx = cum + w[e];
    if (pick == (1 << 30) && w[e] > 0.0 && target < nx) { pick = base + e; lo = cum; hi = nx; }
    cum = nx;
  }
  int first = warp_min_i(pick);
  double margin;
  if (first == (1 << 30)) {                   // rounding guard: last token of the chunk with mass
    int lastv = -1;
    double llo = 0.0, lhi = 0.0;
    double c2 = cb + (li - wl);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (w[e] > 0.0) { lastv = base + e; llo = c2; lhi = c2 + w[e]; }
      c2 += w[e];
    }
    int lv = lastv;
    for (int o = 32; o > 0; o >>= 1) lv = max(lv, __shfl_xor(lv, o, 64));
    first = max(lv, 0);
    const int ol = (first - cfirst * ACC_CH) / 8;
    lo = __shfl(llo, ol, 64);
    hi = __shfl(lhi, ol, 64);
    margin = 0.0;
    (void)hi;
  } else {
    const int ol = (first - cfirst * ACC_CH) / 8;
    lo = __shfl(lo, ol, 64);
    hi = __shfl(hi, ol, 64);
    margin = Sp > 0.0 ? fmin(target - lo, hi - target) / Sp : 0.0;
  }
  if (lane == 0) { sm.draw_tok = first; sm.draw_margin = margin; }
}

template <typename T, bool NUC>   // NUC: the nucleus cut (top_p < 1) is compiled in
__global__ __launch_bounds__(ACC_NT) void k_tree_accept(const T* __restrict__ logits,
                                                        const float* __restrict__ child_logit,
                                                        const int32_t* __restrict__ tokens,
                                                        const int32_t* __restrict__ parents,
                                                        const float* __restrict__ u_acc,
                                                        const float* __restrict__ u_fin, int T_, int V,
                                                        int max_depth, float invtau, float top_p,
                                                        int32_t* __restrict__ acc_nodes,
                                                        int32_t* __restrict__ out_tokens,
                                                        int32_t* __restrict__ out_len, uint8_t* __restrict__ kind,
                                                        float* __restrict__ min_margin) {
  __shared__ AccSmem sm;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int32_t* an = acc_nodes + (size_t)b * max_depth;
  int32_t* ot = out_tokens + (size_t)b * (max_depth + 1);

  // the node inputs are loaded before the topology is checked, so their latency overlaps it (T <= the
  // block size: one node per thread)
  int v_in = 0;
  float cl_in = 0.f, ua_in = 0.f;
  if (tid < T_) {
    v_in = tokens[(size_t)b * T_ + tid];
    cl_in = child_logit[(size_t)b * T_ + tid];
    ua_in = u_acc[(size_t)b * T_ + tid];
  }
  bool ok = tree_setup<SR_MAX_TREE>(sm.tree, parents + (size_t)b * T_, T_);
  if (ok) {
    if (tid < T_) {
      const int c = tid, v = v_in;
      sm.tok[c] = v;
      sm.cl[c] = cl_in;
      sm.ua[c] = ua_in;
      if (c > 0 && (v < 0 || v >= V)) atomicOr(&sm.tree.bad, 1);
      if (sm.tree.depth[c] > max_depth) atomicOr(&sm.tree.bad, 1);
    }
    __syncthreads();
    for (int c = 1 + tid; c < T_; c += ACC_NT)
      for (int k = 1; k < c; ++k)
        if (sm.tree.parent[k] == sm.tree.parent[c] && sm.tok[k] == sm.tok[c]) atomicOr(&sm.tree.bad, 1);
    __syncthreads();
    ok = sm.tree.bad == 0;
  }
  for (int i = tid; i < max_depth; i += ACC_NT) an[i] = -1;
  for (int i = tid; i <= max_depth; i += ACC_NT) ot[i] = -1;
  if (!ok) {
    if (tid == 0) {
      out_len[b] = 0;
      kind[b] = 255;
      if (min_margin) min_margin[b] = __uint_as_float(0x7fc00000u);
    }
    return;
  }
  __syncthreads();

  const T* base = logits + (size_t)b * T_ * V;
  double margin = INFINITY;                   // kept by thread 0
  int n_acc = 0;
  int u = 0;
  const float Ufin = u_fin[b];
  const int nch = (V + ACC_CH - 1) / ACC_CH;
  // nucleus cut of a row and its masked chunk sums: one fused pass for bf16 rows, two (plus the tie count
  // when the cut splits a key) for fp32 rows, whose keys take three digits
  // weights and the first digit's histogram of a nucleus row (bf16: in copies held by the cut's bins)
  auto nuc_stats = [&](const T* r) __attribute__((always_inline)) {
    if constexpr (sizeof(T) == 2) row_stats_nuc<T>(sm, r, V, invtau, (unsigned long long*)&nuc_bins());
    else row_stats_nuc<T>(sm, r, V, invtau, nullptr);
  };
  auto nuc_cut = [&](const T* r) __attribute__((always_inline)) {
    if constexpr (NUC && sizeof(T) == 2) {
      nucleus_bf16(sm, nuc_bins(), r, V, invtau, top_p);
    } else {
      nucleus<T>(sm, r, V, invtau, top_p);
      nuc_masked_sums<T>(sm, r, V, invtau);
    }
  };
  while (true) {
    const T* row = base + (size_t)u * V;
    // the node's children in node order (ballot compaction) and, for the plain walk, the chunks that
    // hold them
    if (wave == 0) {
      if (!NUC) {                                // cleared before the children set theirs (one wave's LDS
        for (int c = lane; c < nch; c += 64) sm.xflag[c] = 0;   // writes complete in order)
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      }
      int n = 0;
      for (int c0 = 0; c0 < T_; c0 += 64) {
        const int c = c0 + lane;
        const bool kid = c > u && c < T_ && sm.tree.parent[c] == u;
        const unsigned long long bal = __ballot(kid);
        if (kid) {
          const int slot = n + __popcll(bal & ((1ull << lane) - 1ull));
          const int v = sm.tok[c];
          sm.kids[slot] = c;
          sm.ktok[slot] = v;
          if (!NUC) sm.xflag[v / ACC_CH] = 1;
        }
        n += __popcll(bal);
      }
      if (lane == 0) sm.nkid = n;
    }
    __syncthreads();
    const int m = sm.nkid;
    if constexpr (NUC) {
      nuc_stats(row);
      nuc_cut(row);                             // and the chunk sums over the nucleus
      if (tid == 0) margin = fmin(margin, sm.nk_margin);
      outside_mass<T, NUC>(sm, row, V, invtau, m);   // sums the masked chunk sums to S
    } else {
      row_stats<T>(sm, row, V, invtau, m);     // with the children's chunks and logits
    }
    if (wave == 0) {
      // residual on the children (2 per lane) and the mass outside them, float64
      double r[2], lg[2];
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int k = lane + 64 * s;
        r[s] = 0.0;
        lg[s] = -INFINITY;
        if (k < m) {
          double pt;
          if constexpr (NUC) {
            pt = ptilde(sm, row, sm.tok[sm.kids[k]], invtau);
          } else {                              // ptilde of the logit the row pass kept
            const float x = sm.kx[k];
            const int c = sm.tok[sm.kids[k]] / ACC_CH;
            pt = x == -INFINITY ? 0.0 : (double)tilt(x, invtau, sm.cmax[c]) * sm.cscale[c];
          }
          sm.kpt[k] = pt;
          r[s] = pt / sm.S;
          lg[s] = (double)sm.cl[sm.kids[k]];
        }
      }
      double rest = sm.S_out / sm.S;
      int acc = -1;
      for (int j = 0; j < m; ++j) {
        // q_{u,j}: softmax of the draft logits over children j..m-1
        double mx = -INFINITY;
#pragma unroll
        for (int s = 0; s < 2; ++s)
          if (lane + 64 * s >= j) mx = fmax(mx, lg[s]);
        mx = wave_max_f64(mx);
        double w[2];
        double ql = 0.0;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const int k = lane + 64 * s;
          w[s] = (k >= j && k < m) ? exp(lg[s] - mx) : 0.0;
          ql += w[s];
        }
        const double Q = wave_sum_f64(ql);
        const double rj = __shfl((j >> 6) ? r[1] : r[0], j & 63, 64);
        const double qj = __shfl((j >> 6) ? w[1] : w[0], j & 63, 64) / Q;
        const double A = fmin(1.0, rj / qj);
        const double U = (double)sm.ua[sm.kids[j]];
        margin = fmin(margin, fabs(A - U));
        if (U <= A) { acc = j; break; }
        // Eq. (noderesidual) restricted to where q is non-zero; Z = sum over the vocabulary
        double zl = 0.0;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const int k = lane + 64 * s;
          if (k >= j && k < m) r[s] = fmax(r[s] - w[s] / Q, 0.0);
          zl += (k < m) ? r[s] : 0.0;
        }
        const double Z = rest + wave_sum_f64(zl);
        rest /= Z;
#pragma unroll
        for (int s = 0; s < 2; ++s) r[s] /= Z;
      }
      if (lane == 0) sm.accepted = acc;
    }
    __syncthreads();
    const int acc = sm.accepted;
    if (acc < 0) {
      // every child rejected: fallback from the final residual = p outside the children
      if (wave == 0) draw<T>(sm, row, V, invtau, m, Ufin);
      __syncthreads();
      if (tid == 0) {
        ot[n_acc] = sm.draw_tok;
        out_len[b] = n_acc + 1;
        kind[b] = 0;
        margin = fmin(margin, sm.draw_margin);
        if (min_margin) min_margin[b] = (float)margin;
      }
      return;
    }
    const int c = sm.kids[acc];
    if (tid == 0) { an[n_acc] = c; ot[n_acc] = sm.tok[c]; }
    ++n_acc;
    __syncthreads();
    if (sm.tree.nkids[c] > 0) { u = c; continue; }
    // accepted leaf: bonus token from its own target distribution
    const T* lrow = base + (size_t)c * V;
    if constexpr (NUC) {
      nuc_stats(lrow);
      nuc_cut(lrow);
      if (tid == 0) margin = fmin(margin, sm.nk_margin);
    } else {
      row_stats<T>(sm, lrow, V, invtau, 0);
    }
    if (wave == 0) draw<T>(sm, lrow, V, invtau, 0, Ufin);
    __syncthreads();
    if (tid == 0) {
      ot[n_acc] = sm.draw_tok;
      out_len[b] = n_acc + 1;
      kind[b] = 1;
      margin = fmin(margin, sm.draw_margin);
      if (min_margin) min_margin[b] = (float)margin;
    }
    return;
  }
}

sr_status launch_tree_accept(const sr_accept_desc& d, const void* target_logits, const float* child_logit,
                             const int32_t* tokens, const int32_t* parents, const float* u_acc,
                             const float* u_fin, int32_t* acc_nodes, int32_t* out_tokens, int32_t* out_len,
                             uint8_t* final_kind, float* min_margin, hipStream_t s) {
  const float invtau = 1.0f / d.temperature;
  const bool nuc = d.top_p < 1.f;
  if (d.logit_dtype == SR_BF16) {
    const bf16_t* lg = (const bf16_t*)target_logits;
    if (nuc)
      SR_LAUNCH("sr_tree_accept", (k_tree_accept<bf16_t, true>), dim3(d.B), dim3(ACC_NT), 0, s, lg, child_logit,
                tokens, parents, u_acc, u_fin, d.T, d.V, d.max_depth, invtau, d.top_p, acc_nodes, out_tokens,
                out_len, final_kind, min_margin);
    else
      SR_LAUNCH("sr_tree_accept", (k_tree_accept<bf16_t, false>), dim3(d.B), dim3(ACC_NT), 0, s, lg, child_logit,
                tokens, parents, u_acc, u_fin, d.T, d.V, d.max_depth, invtau, d.top_p, acc_nodes, out_tokens,
                out_len, final_kind, min_margin);
  } else {
    const float* lg = (const float*)target_logits;
    if (nuc)
      SR_LAUNCH("sr_tree_accept", (k_tree_accept<float, true>), dim3(d.B), dim3(ACC_NT), 0, s, lg, child_logit,
                tokens, parents, u_acc, u_fin, d.T, d.V, d.max_depth, invtau, d.top_p, acc_nodes, out_tokens,
                out_len, final_kind, min_margin);
    else
      SR_LAUNCH("sr_tree_accept", (k_tree_accept<float, false>), dim3(d.B), dim3(ACC_NT), 0, s, lg, child_logit,
                tokens, parents, u_acc, u_fin, d.T, d.V, d.max_depth, invtau, d.top_p, acc_nodes, out_tokens,
                out_len, final_kind, min_margin);
  }
  return SR_OK;
}

}  // namespace sr
