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
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace sr {

constexpr int ACC_NW = 16;
constexpr int ACC_NT = ACC_NW * 64;
constexpr int ACC_CH = 512;                  // tokens per chunk = 64 lanes x 8
constexpr int ACC_MAX_CHUNKS = 512;          // V <= 262144
constexpr int ACC_GROUP = 4;                 // chunks whose loads a wave issues together

template <typename T> struct RowLoad;
template <> struct RowLoad<bf16_t> {
  static __device__ __forceinline__ void load8(const bf16_t* p, float* x) {
    const u32x4 w = *(const u32x4*)p;
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = bf2f((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xffffu));
  }
  static __device__ __forceinline__ float load1(const bf16_t* p) { return bf2f(*p); }
};
template <> struct RowLoad<float> {
  static __device__ __forceinline__ void load8(const float* p, float* x) {
    const f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) { x[e] = a[e]; x[e + 4] = b[e]; }
  }
  static __device__ __forceinline__ float load1(const float* p) { return *p; }
};

struct AccSmem {
  TreeLds<SR_MAX_TREE> tree;
  int tok[SR_MAX_TREE];
  float cl[SR_MAX_TREE];
  float ua[SR_MAX_TREE];
  float cmax[ACC_MAX_CHUNKS];
  double csum[ACC_MAX_CHUNKS];
  double cscale[ACC_MAX_CHUNKS];
  int kids[SR_MAX_TREE];
  double S;
  int bad;
  int nkid;
  int accepted;      // slot index (0-based) accepted at the current node, -1 = all rejected
  int draw_tok;
  double draw_margin;
};

// exp(y - m) with y = x * invtau, as 2^((y - m) log2 e) on the hardware exponential; every step is
// rounded separately, so the value is identical wherever it is recomputed
__device__ __forceinline__ float tilt(float x, float invtau, float m) {
  return __builtin_amdgcn_exp2f(__fmul_rn(__fsub_rn(__fmul_rn(x, invtau), m), kLog2e));
}

template <typename T>
__device__ void row_stats(AccSmem& sm, const T* __restrict__ row, int V, float invtau) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nch = (V + ACC_CH - 1) / ACC_CH;
  for (int c0 = wave * ACC_GROUP; c0 < nch; c0 += ACC_NW * ACC_GROUP) {
    float x[ACC_GROUP][8];
#pragma unroll
    for (int gi = 0; gi < ACC_GROUP; ++gi) {
      const int base = (c0 + gi) * ACC_CH + lane * 8;
      if (c0 + gi < nch && base < V) {
        RowLoad<T>::load8(row + base, x[gi]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[gi][e] = -INFINITY;
      }
    }
#pragma unroll
    for (int gi = 0; gi < ACC_GROUP; ++gi) {
      if (c0 + gi >= nch) break;
      float ml = -INFINITY;
#pragma unroll
      for (int e = 0; e < 8; ++e) ml = fmaxf(ml, __fmul_rn(x[gi][e], invtau));
      const float m = wave_max_f32(ml);
      float sl = 0.f;                           // at most 512 terms in (0, 1]: fp32 suffices
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (x[gi][e] != -INFINITY) sl += tilt(x[gi][e], invtau, m);
      const float s = wave_sum_f32(sl);
      if (lane == 0) { sm.cmax[c0 + gi] = m; sm.csum[c0 + gi] = (double)s; }
    }
  }
  __syncthreads();
  if (wave == 0) {
    float ml = -INFINITY;
    for (int c = lane; c < nch; c += 64) ml = fmaxf(ml, sm.cmax[c]);
    const float M = wave_max_f32(ml);
    double sl = 0.0;
    for (int c = lane; c < nch; c += 64) {
      const double sc = exp((double)sm.cmax[c] - (double)M);
      sm.cscale[c] = sc;
      sl += sm.csum[c] * sc;
    }
    const double S = wave_sum_f64(sl);
    if (lane == 0) sm.S = S;
  }
  __syncthreads();
}

// unnormalised target weight of token v under the current row statistics
template <typename T>
__device__ __forceinline__ double ptilde(const AccSmem& sm, const T* row, int v, float invtau) {
  const int c = v / ACC_CH;
  const float x = RowLoad<T>::load1(row + v);
  if (x == -INFINITY) return 0.0;
  return (double)tilt(x, invtau, sm.cmax[c]) * sm.cscale[c];
}

// Inverse-CDF draw over the current row, token-id order, excluding the tokens of
// sm.kids[0..n_excl). Run by wave 0; result in sm.draw_tok / sm.draw_margin.
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
    if (c < nch) {
      a = sm.csum[c] * sm.cscale[c];
      for (int k = 0; k < n_excl; ++k) {
        const int v = sm.tok[sm.kids[k]];
        if (v / ACC_CH == c) a -= ptilde(sm, row, v, invtau);
      }
      a = fmax(a, 0.0);
    }
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
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int v = base + e;
    double pv = 0.0;
    if (v < V) {
      bool ex = false;
      for (int k = 0; k < n_excl; ++k) ex |= sm.tok[sm.kids[k]] == v;
      if (!ex) pv = ptilde(sm, row, v, invtau);
    }
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

template <typename T>
__global__ __launch_bounds__(ACC_NT) void k_tree_accept(const T* __restrict__ logits,
                                                        const float* __restrict__ child_logit,
                                                        const int32_t* __restrict__ tokens,
                                                        const int32_t* __restrict__ parents,
                                                        const float* __restrict__ u_acc,
                                                        const float* __restrict__ u_fin, int T_, int V,
                                                        int max_depth, float invtau, int32_t* __restrict__ acc_nodes,
                                                        int32_t* __restrict__ out_tokens,
                                                        int32_t* __restrict__ out_len, uint8_t* __restrict__ kind,
                                                        float* __restrict__ min_margin) {
  __shared__ AccSmem sm;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int32_t* an = acc_nodes + (size_t)b * max_depth;
  int32_t* ot = out_tokens + (size_t)b * (max_depth + 1);

  bool ok = tree_setup<SR_MAX_TREE>(sm.tree, parents + (size_t)b * T_, T_);
  if (ok) {
    for (int c = tid; c < T_; c += ACC_NT) {
      const int v = tokens[(size_t)b * T_ + c];
      sm.tok[c] = v;
      sm.cl[c] = child_logit[(size_t)b * T_ + c];
      sm.ua[c] = u_acc[(size_t)b * T_ + c];
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
  while (true) {
    const T* row = base + (size_t)u * V;
    row_stats<T>(sm, row, V, invtau);
    if (tid == 0) {
      int n = 0;
      for (int c = u + 1; c < T_; ++c)
        if (sm.tree.parent[c] == u) sm.kids[n++] = c;
      sm.nkid = n;
    }
    __syncthreads();
    const int m = sm.nkid;
    if (wave == 0) {
      // residual on the children (2 per lane) and the mass outside them, float64
      double r[2], lg[2];
      double out_mass_part = 0.0;
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int k = lane + 64 * s;
        r[s] = 0.0;
        lg[s] = -INFINITY;
        if (k < m) {
          const double pt = ptilde(sm, row, sm.tok[sm.kids[k]], invtau);
          r[s] = pt / sm.S;
          lg[s] = (double)sm.cl[sm.kids[k]];
          out_mass_part += pt;
        }
      }
      double rest = (sm.S - wave_sum_f64(out_mass_part)) / sm.S;
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
    row_stats<T>(sm, lrow, V, invtau);
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
  if (d.logit_dtype == SR_BF16) {
    SR_LAUNCH("sr_tree_accept", k_tree_accept<bf16_t>, dim3(d.B), dim3(ACC_NT), 0, s,
              (const bf16_t*)target_logits, child_logit, tokens, parents, u_acc, u_fin, d.T, d.V, d.max_depth,
              invtau, acc_nodes, out_tokens, out_len, final_kind, min_margin);
  } else {
    SR_LAUNCH("sr_tree_accept", k_tree_accept<float>, dim3(d.B), dim3(ACC_NT), 0, s,
              (const float*)target_logits, child_logit, tokens, parents, u_acc, u_fin, d.T, d.V, d.max_depth,
              invtau, acc_nodes, out_tokens, out_len, final_kind, min_margin);
  }
  return SR_OK;
}

}  // namespace sr
