// Tree-verify attention on gfx950.
//
// Paper: App. B.1 Eq. (nodep) -- the packed verification forward must give every tree node
// the result of an ordinary autoregressive forward at prefix ++ path(u). For one attention
// layer: node u's queries see the whole cached prefix and the tree tokens on u's root path.
//
// Work item = (trajectory b, KV head g, prefix chunk c, row group). The query rows of one
// work item are the T*G (node, head-in-group) pairs sharing KV head g, so every K/V tile
// staged in LDS is reused by all of them (GQA sharing). Each wave owns 32 query rows and
// computes transposed scores S^T = K Q^T on 32x32 MFMA tiles: a lane then holds 16 keys of
// one query row, so the row max needs one cross-half exchange. P stays in registers and
// feeds O^T = V^T P^T; V is transposed into LDS when staged. bf16 scores use
// v_mfma_f32_32x32x16_bf16; the probability-weighted V sum uses v_mfma_f32_32x32x16_f16
// with P and V in fp16 (bf16 P would cost ~3e-3 relative error at 4k-token contexts).
// The last chunk of a trajectory also processes the T tree keys under the ancestor mask.
// Several chunks of one (b, g) are merged by log-sum-exp in k_attn_combine.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace sr {

constexpr int ATT_KT = 64;             // keys per LDS tile
constexpr int ATT_NW = 8;              // waves per block
constexpr int ATT_ROWS = ATT_NW * 32;  // query rows per block
constexpr int ATT_CHUNK_PAGES = 128;   // prefix pages per work item (2048 tokens)
constexpr int ATT_BS = 16;             // tokens per page

template <typename T> struct AttnT;
template <> struct AttnT<bf16_t> {
  static constexpr int KPL = 8;        // elements per lane per MFMA slot
  typedef u32x4 qfrag;                 // 8 x bf16
  typedef _Float16 vt;                 // V^T element in LDS
  typedef f16x8 pfrag;
  static constexpr int PADK = 8, PADV = 4;
  static __device__ __forceinline__ f32x16 mma_qk(qfrag a, qfrag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  }
  static __device__ __forceinline__ f32x16 mma_pv(pfrag a, pfrag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};
template <> struct AttnT<float> {
  static constexpr int KPL = 1;
  typedef float qfrag;
  typedef float vt;
  typedef float pfrag;
  static constexpr int PADK = 4, PADV = 4;
  static __device__ __forceinline__ f32x16 mma_qk(qfrag a, qfrag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ f32x16 mma_pv(pfrag a, pfrag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

// key (within a 32-key subtile) held by register i of a lane in half h of a 32x32 output tile
__device__ __forceinline__ int tile_row(int i, int h) { return 8 * (i >> 2) + 4 * h + (i & 3); }

template <typename T, int D>
struct AttnSmem {
  static constexpr int LDK = D + AttnT<T>::PADK;
  static constexpr int LDV = ATT_KT + AttnT<T>::PADV;
  T ks[ATT_KT * LDK];
  typename AttnT<T>::vt vt[D * LDV];
  int blk[ATT_CHUNK_PAGES];
  uint32_t anc[SR_MAX_TREE][SR_MAX_TREE / 32];
  int parent[SR_MAX_TREE];
  int bad;
};

template <typename T, int D>
__global__ __launch_bounds__(ATT_NW * 64) void k_tree_attn(
    const T* __restrict__ q, const T* __restrict__ k_cache, const T* __restrict__ v_cache,
    const int32_t* __restrict__ block_table, const int32_t* __restrict__ ctx_len, const T* __restrict__ k_tree,
    const T* __restrict__ v_tree, const int32_t* __restrict__ parents, float* __restrict__ out,
    float* __restrict__ lse, float* __restrict__ part_o, float* __restrict__ part_ml, int T_, int Hq, int Hkv,
    int max_blocks, int num_blocks, float scale_log2, int R, int Rpad, int row_groups, int n_chunks_max) {
  using AT = AttnT<T>;
  constexpr int KPL = AT::KPL, KSTEP = 2 * KPL;
  constexpr int VEC = 16 / sizeof(T);
  constexpr int LDK = AttnSmem<T, D>::LDK, LDV = AttnSmem<T, D>::LDV;
  constexpr int NQF = D / KSTEP;      // Q fragments per lane
  constexpr int NDT = D / 32;         // 32-wide output tiles along D
  constexpr int NT = ATT_NW * 64;
  constexpr int TILE_VECS = ATT_KT * D / VEC;
  constexpr int VPT = (TILE_VECS + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) AttnSmem<T, D> sm;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
  const int c = blockIdx.x / row_groups, rg = blockIdx.x % row_groups;
  const int g = blockIdx.y, b = blockIdx.z;
  const int G = Hq / Hkv;
  const int Lraw = ctx_len[b];
  const bool ctx_ok = Lraw >= 0 && Lraw <= max_blocks * ATT_BS;
  const int L = ctx_ok ? Lraw : 0;
  const int pages = (L + ATT_BS - 1) / ATT_BS;
  const int n_chunks = ctx_ok ? max(1, (pages + ATT_CHUNK_PAGES - 1) / ATT_CHUNK_PAGES) : 1;
  if (c >= n_chunks) return;
  const bool last = c == n_chunks - 1;
  const int page0 = c * ATT_CHUNK_PAGES, page1 = min(pages, page0 + ATT_CHUNK_PAGES);
  const int key0 = page0 * ATT_BS, key1 = min(L, page1 * ATT_BS);

  // ---- stage page ids and (last chunk) the ancestor masks; validate what this block reads
  if (tid == 0) sm.bad = ctx_ok ? 0 : 1;
  __syncthreads();
  for (int p = page0 + tid; p < page1; p += NT) {
    int blk = block_table[(size_t)b * max_blocks + p];
    if (blk < 0 || blk >= num_blocks) { atomicOr(&sm.bad, 1); blk = 0; }
    sm.blk[p - page0] = blk;
  }
  if (last) {
    for (int i = tid; i < T_; i += NT) {
      int p = parents[(size_t)b * T_ + i];
      if ((i == 0 && p != -1) || (i > 0 && (p < 0 || p >= i))) atomicOr(&sm.bad, 1);
      sm.parent[i] = p;
    }
    __syncthreads();
    if (!sm.bad)
      for (int i = tid; i < T_; i += NT) {
        uint32_t m[SR_MAX_TREE / 32] = {0, 0, 0, 0};
        for (int a = i; a >= 0; a = sm.parent[a]) m[a >> 5] |= 1u << (a & 31);
#pragma unroll
        for (int w = 0; w < SR_MAX_TREE / 32; ++w) sm.anc[i][w] = m[w];
      }
  }
  __syncthreads();
  const bool bad = sm.bad != 0;

  // ---- this wave's query rows: row r <-> (node t = r / G, head g*G + r % G)
  const int rowbase = rg * ATT_ROWS + wave * 32;
  const int my_r = rowbase + (lane & 31);
  const bool row_ok = my_r < R;
  const int my_t = row_ok ? my_r / G : 0;
  typename AT::qfrag qf[NQF];
  {
    const T* qp = q + (((size_t)b * T_ + my_t) * Hq + g * G + (row_ok ? my_r % G : 0)) * D;
#pragma unroll
    for (int ks = 0; ks < NQF; ++ks) {
      const int dd = ks * KSTEP + half * KPL;
      if constexpr (KPL == 8) {
        u32x4 z = {0, 0, 0, 0};
        if (row_ok) z = *(const u32x4*)(qp + dd);
        qf[ks] = z;
      } else {
        qf[ks] = row_ok ? qp[dd] : 0.f;
      }
    }
  }
  uint32_t my_anc[SR_MAX_TREE / 32] = {0, 0, 0, 0};
  if (last && !bad && row_ok) {
#pragma unroll
    for (int w = 0; w < SR_MAX_TREE / 32; ++w) my_anc[w] = sm.anc[my_t][w];
  }

  f32x16 o[NDT];
#pragma unroll
  for (int i = 0; i < NDT; ++i) o[i] = (f32x16){};
  float m_run = -INFINITY, l_run = 0.f;
  const bool wave_active = rowbase < R && !bad;

  // ---- one K/V tile: keys [t0, t0 + ATT_KT) of the prefix (tree == false) or of the tree
  auto do_tile = [&](int t0, bool tree) {
    __syncthreads();
    // stage K (row-major) and V (transposed) in LDS; keys outside the range are zero
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int v = tid + i * NT;
      if (v >= TILE_VECS) break;
      const int key = v / (D / VEC), col = (v % (D / VEC)) * VEC;
      const int kidx = t0 + key;
      u32x4 kv = {0, 0, 0, 0}, vv = {0, 0, 0, 0};
      if (!bad) {
        size_t off = 0;
        bool ok;
        if (!tree) {
          ok = kidx < key1;
          if (ok) off = (((size_t)sm.blk[(kidx >> 4) - page0] * Hkv + g) * ATT_BS + (kidx & 15)) * D + col;
          if (ok) { kv = *(const u32x4*)(k_cache + off); vv = *(const u32x4*)(v_cache + off); }
        } else {
          ok = kidx < T_;
          if (ok) off = (((size_t)b * T_ + kidx) * Hkv + g) * D + col;
          if (ok) { kv = *(const u32x4*)(k_tree + off); vv = *(const u32x4*)(v_tree + off); }
        }
      }
      *(u32x4*)(sm.ks + key * LDK + col) = kv;
      if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t w = vv[e >> 1];
          const float f = bf2f((e & 1) ? (w >> 16) : (w & 0xffffu));
          sm.vt[(col + e) * LDV + key] = (_Float16)f;
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) sm.vt[(col + e) * LDV + key] = __uint_as_float(vv[e]);
      }
    }
    __syncthreads();
    if (!wave_active) return;
    // scores S^T for two 32-key subtiles
    f32x16 s[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      s[kt] = (f32x16){};
#pragma unroll
      for (int ks = 0; ks < NQF; ++ks) {
        const T* kp = sm.ks + (kt * 32 + (lane & 31)) * LDK + ks * KSTEP + half * KPL;
        typename AT::qfrag kf;
        if constexpr (KPL == 8) kf = *(const u32x4*)kp; else kf = *kp;
        s[kt] = AT::mma_qk(kf, qf[ks], s[kt]);
      }
    }
    // mask, scale to log2 units, running max
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      // ancestor word of this 32-key subtile (t0 is a multiple of 64, so the word index is uniform)
      const int wi = (t0 >> 5) + kt;
      const uint32_t aw = wi == 0 ? my_anc[0] : wi == 1 ? my_anc[1] : wi == 2 ? my_anc[2] : my_anc[3];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int kidx = t0 + kt * 32 + tile_row(i, half);
        bool ok;
        if (!tree) ok = kidx < key1;
        else ok = kidx < T_ && ((aw >> (kidx & 31)) & 1u);
        const float v = ok ? s[kt][i] * scale_log2 : -INFINITY;
        s[kt][i] = v;
        mx = fmaxf(mx, v);
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);
    float psum = 0.f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = exp2f(s[kt][i] - m_use);
        s[kt][i] = p;
        psum += p;
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) o[dt] *= alpha;
    // O^T += V^T P^T; MFMA slot e of step st in half h carries key tile_row(st*KPL + e, h)
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int st = 0; st < 16 / KPL; ++st) {
        typename AT::pfrag pf;
        if constexpr (KPL == 8) {
#pragma unroll
          for (int e = 0; e < 8; ++e) pf[e] = (_Float16)s[kt][st * 8 + e];
        } else {
          pf = s[kt][st];
        }
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const typename AT::vt* vp = sm.vt + (dt * 32 + (lane & 31)) * LDV + kt * 32;
          typename AT::pfrag vf;
          if constexpr (KPL == 8) {
            const int k0 = tile_row(st * 8, half);        // 4 consecutive keys
            const int k1 = tile_row(st * 8 + 4, half);    // the next 4 consecutive keys
            const f16x4 lo = *(const f16x4*)(vp + k0);
            const f16x4 hi = *(const f16x4*)(vp + k1);
            vf = (f16x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          } else {
            vf = vp[tile_row(st, half)];
          }
          o[dt] = AT::mma_pv(vf, pf, o[dt]);
        }
      }
  };

  for (int t0 = key0; t0 < key1; t0 += ATT_KT) do_tile(t0, false);
  if (last)
    for (int t0 = 0; t0 < T_; t0 += ATT_KT) do_tile(t0, true);

  // ---- write the normalised result (single chunk) or a partial (m, l, O/l)
  if (rowbase >= R) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float qnan = __uint_as_float(0x7fc00000u);
  if (!row_ok) return;
  if (n_chunks == 1) {
    const int h = g * G + my_r % G;
    float* op = out + (((size_t)b * T_ + my_t) * Hq + h) * D;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 16; i += 4) {
        f32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = bad ? qnan : o[dt][i + e] * inv;
        *(f32x4*)(op + dt * 32 + tile_row(i, half)) = v;
      }
    if (lse != nullptr && half == 0)
      lse[((size_t)b * T_ + my_t) * Hq + h] = bad ? qnan : (m_run + log2f(l_tot)) * kLn2;
  } else {
    const size_t pr = (((size_t)b * Hkv + g) * n_chunks_max + c) * Rpad + my_r;
    float* op = part_o + pr * D;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 16; i += 4) {
        f32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = o[dt][i + e] * inv;
        *(f32x4*)(op + dt * 32 + tile_row(i, half)) = v;
      }
    if (half == 0) {
      part_ml[pr * 2 + 0] = bad ? qnan : m_run;
      part_ml[pr * 2 + 1] = bad ? qnan : l_tot;
    }
  }
}

// Merge the chunk partials of every (trajectory, KV head) that was split.
template <int D>
__global__ __launch_bounds__(256) void k_attn_combine(const int32_t* __restrict__ ctx_len,
                                                      const float* __restrict__ part_o,
                                                      const float* __restrict__ part_ml, float* __restrict__ out,
                                                      float* __restrict__ lse, int T_, int Hq, int Hkv,
                                                      int max_blocks, int R, int Rpad, int n_chunks_max) {
  constexpr int TPR = D / 4;                 // threads per row (4 floats each)
  constexpr int RPB = 256 / TPR;             // rows per block
  const int g = blockIdx.y, b = blockIdx.z;
  const int Lraw = ctx_len[b];
  const bool ctx_ok = Lraw >= 0 && Lraw <= max_blocks * ATT_BS;
  const int pages = ctx_ok ? (Lraw + ATT_BS - 1) / ATT_BS : 0;
  const int n_chunks = ctx_ok ? max(1, (pages + ATT_CHUNK_PAGES - 1) / ATT_CHUNK_PAGES) : 1;
  if (n_chunks <= 1) return;
  const int r = blockIdx.x * RPB + threadIdx.x / TPR;
  const int d4 = (threadIdx.x % TPR) * 4;
  if (r >= R) return;
  const size_t base = ((size_t)b * Hkv + g) * n_chunks_max * Rpad + r;
  float M = -INFINITY;
  bool nan = false;
  for (int c = 0; c < n_chunks; ++c) {
    const float m = part_ml[(base + (size_t)c * Rpad) * 2];
    const float l = part_ml[(base + (size_t)c * Rpad) * 2 + 1];
    nan |= isnan(m) || isnan(l);
    M = fmaxf(M, m);
  }
  const float Mu = (M == -INFINITY) ? 0.f : M;
  float W = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int c = 0; c < n_chunks; ++c) {
    const size_t pr = base + (size_t)c * Rpad;
    const float w = part_ml[pr * 2 + 1] * exp2f(part_ml[pr * 2] - Mu);
    W += w;
    acc += w * *(const f32x4*)(part_o + pr * D + d4);
  }
  const int G = Hq / Hkv;
  const int t = r / G, h = g * G + r % G;
  const float qnan = __uint_as_float(0x7fc00000u);
  const float inv = W > 0.f ? 1.f / W : 0.f;
  f32x4 v = acc * inv;
  if (nan) v = (f32x4){qnan, qnan, qnan, qnan};
  *(f32x4*)(out + (((size_t)b * T_ + t) * Hq + h) * D + d4) = v;
  if (lse != nullptr && d4 == 0) lse[((size_t)b * T_ + t) * Hq + h] = nan ? qnan : (M + log2f(W)) * kLn2;
}

AttnPlan attn_plan(const sr_attn_desc& d) {
  AttnPlan p;
  p.R = d.T * (d.Hq / d.Hkv);
  p.Rpad = (p.R + 31) / 32 * 32;
  p.row_groups = (p.R + ATT_ROWS - 1) / ATT_ROWS;
  p.chunk_pages = ATT_CHUNK_PAGES;
  p.n_chunks = std::max(1, (d.max_blocks + ATT_CHUNK_PAGES - 1) / ATT_CHUNK_PAGES);
  const size_t rows = (size_t)d.B * d.Hkv * p.n_chunks * p.Rpad;
  p.part_o_bytes = p.n_chunks > 1 ? rows * d.D * sizeof(float) : 0;
  p.part_ml_bytes = p.n_chunks > 1 ? rows * 2 * sizeof(float) : 0;
  return p;
}

template <typename T, int D>
static sr_status launch_attn_t(const sr_attn_desc& d, const AttnPlan& p, const void* q, const void* kc,
                               const void* vc, const int32_t* bt, const int32_t* cl, const void* kt,
                               const void* vt, const int32_t* par, float* out, float* lse, float* po, float* pml,
                               hipStream_t s) {
  const float scale_log2 = d.scale * kLog2e;
  dim3 grid(p.n_chunks * p.row_groups, d.Hkv, d.B);
  SR_LAUNCH("sr_tree_attn", (k_tree_attn<T, D>), grid, dim3(ATT_NW * 64), 0, s, (const T*)q, (const T*)kc,
            (const T*)vc, bt, cl, (const T*)kt, (const T*)vt, par, out, lse, po, pml, d.T, d.Hq, d.Hkv,
            d.max_blocks, d.num_blocks, scale_log2, p.R, p.Rpad, p.row_groups, p.n_chunks);
  if (p.n_chunks > 1) {
    constexpr int RPB = 256 / (D / 4);
    dim3 cgrid((p.R + RPB - 1) / RPB, d.Hkv, d.B);
    SR_LAUNCH("sr_attn_combine", (k_attn_combine<D>), cgrid, dim3(256), 0, s, cl, po, pml, out, lse, d.T, d.Hq,
              d.Hkv, d.max_blocks, p.R, p.Rpad, p.n_chunks);
  }
  return SR_OK;
}

sr_status launch_tree_attn(const sr_attn_desc& d, const AttnPlan& p, const void* q, const void* k_cache,
                           const void* v_cache, const int32_t* block_table, const int32_t* ctx_len,
                           const void* k_tree, const void* v_tree, const int32_t* parents, float* out,
                           float* lse, float* part_o, float* part_ml, hipStream_t s) {
#define SR_ATTN_CASE(TT, DD)                                                                                  \
  return launch_attn_t<TT, DD>(d, p, q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, parents, out, \
                               lse, part_o, part_ml, s)
  if (d.dtype == SR_BF16) {
    if (d.D == 128) SR_ATTN_CASE(bf16_t, 128);
    SR_ATTN_CASE(bf16_t, 64);
  }
  if (d.D == 128) SR_ATTN_CASE(float, 128);
  SR_ATTN_CASE(float, 64);
#undef SR_ATTN_CASE
}

}  // namespace sr
