// Tree-verify attention on gfx950.
//
// Paper: App. B.1 Eq. (nodep) -- the packed verification forward must give every tree node
// the result of an ordinary autoregressive forward at prefix ++ path(u). For one attention
// layer: node u's queries see the whole cached prefix and the tree tokens on u's root path.
//
// Work item = (trajectory b, KV head g, prefix chunk c, row group). The query rows of one
// work item are the T*G (node, head-in-group) pairs sharing KV head g, so every K/V tile
// staged in LDS is reused by all of them (GQA sharing). Scores are computed transposed,
// S^T = K Q^T on 32x32 MFMA tiles: a lane then holds 16 keys of one query row, so the row max
// needs one cross-half exchange; P stays in registers and feeds O^T = V^T P^T. The last chunk
// of a trajectory also processes the T tree keys under the ancestor mask. Several chunks of
// one (b, g) are merged by log-sum-exp in k_attn_combine.
//
// Three kernels share the item decomposition:
// * k_tree_attn_dma<D> (bf16): one persistent block of eight waves per CU takes items from a
//   counter. A row group holds at most 224 rows, so at least one wave has no query rows and
//   issues all K/V transfers straight from HBM into a four-slot LDS ring; every other wave owns
//   32 query rows and converts a share of each V tile from bf16 to fp16 in place. Scores use
//   v_mfma_f32_32x32x16_bf16, the probability-weighted V sum v_mfma_f32_32x32x16_f16 with P and
//   V in fp16 (bf16 P would cost ~3e-3 relative error at 4k-token contexts). fp16 holds a bf16
//   value exactly only for magnitudes in [2^-14, 65280] (or zero); the converting waves track the
//   range of every V value they convert, and an item that meets any other value is listed for
//   k_tree_attn_redo, which recomputes it.
// * k_tree_attn_redo<D> (bf16): the listed items, one block each, with V widened to fp32 and the
//   weighted sum on fp32 MFMA (exact for every finite bf16 V).
// * k_tree_attn<AT, D> (fp32 inputs; and the redo path's item body): one block per item, K/V
//   staged through registers into a two-slot LDS ring with V transposed, eight waves of 32 rows.
#include <math.h>

#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace sr {

constexpr int ATT_KT = 64;             // keys per LDS tile
constexpr int ATT_NW = 8;              // waves per block
constexpr int ATT_RB = 1;              // 32-row query blocks per wave
constexpr int ATT_ROWS = ATT_NW * ATT_RB * 32;  // query rows per block
constexpr int ATT_CHUNK_PAGES = 256;   // most prefix pages per work item (4096 tokens): with many
                                       // (trajectory, KV head) pairs; 128 or 32 with fewer (attn_plan)
constexpr int ATT_BS = 16;             // tokens per page

// Arithmetic of the register-staged kernel. QKPL / PKPL: elements a lane supplies per MFMA slot for the
// scores and for the weighted V sum.
// fp32 inputs: fp32 MFMA for both products.
struct AttnF32 {
  typedef float T;
  static constexpr int QKPL = 1, PKPL = 1;
  typedef float qfrag;
  typedef float vt;                    // V^T element in LDS
  typedef float pfrag;
  static __device__ __forceinline__ f32x16 mma_qk(qfrag a, qfrag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ f32x16 mma_pv(pfrag a, pfrag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};
// bf16 inputs for any V: bf16 MFMA for the scores (as the DMA kernel), V widened exactly to fp32 and the
// weighted sum on fp32 MFMA with P in fp32.
struct AttnBf16Wide {
  typedef bf16_t T;
  static constexpr int QKPL = 8, PKPL = 1;
  typedef u32x4 qfrag;                 // 8 x bf16
  typedef float vt;
  typedef float pfrag;
  static __device__ __forceinline__ f32x16 mma_qk(qfrag a, qfrag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  }
  static __device__ __forceinline__ f32x16 mma_pv(pfrag a, pfrag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

// key (within a 32-key subtile) held by register i of a lane in half h of a 32x32 output tile
__device__ __forceinline__ int tile_row(int i, int h) { return 8 * (i >> 2) + 4 * h + (i & 3); }

// LDS swizzle of V^T rows: 4-key groups of row d live at group position g ^ vswz(d), which keeps both
// the transposing writes (rows 4 apart) and the MFMA operand reads (32 consecutive rows) free of bank
// conflicts.
__device__ __forceinline__ int vswz(int d) { return (d ^ (d >> 2)) & 15; }

template <class AT, int D>
struct AttnGeom {
  static constexpr int E = sizeof(typename AT::T);       // element bytes in the cache
  static constexpr int ROWB = D * E;                     // bytes of one K row
  static constexpr int NCH = ROWB / 16;                  // 16-byte chunks per K row
  static constexpr int KTILE = ATT_KT * ROWB;            // bytes of a K tile
  static constexpr int VE = sizeof(typename AT::vt);
  static constexpr int VROWB = ATT_KT * VE;              // bytes of one V^T row (64 keys)
  static constexpr int VTILE = D * VROWB;
  static constexpr int NT = ATT_NW * 64;
  static constexpr int KVEC = KTILE / 16;                // 16-byte K vectors per tile
  static constexpr int KVPT = KVEC / NT;                 // per thread
  static constexpr int VITEMS = (ATT_KT / 4) * (D / 4);  // 4 keys x 4 dims per item
  static constexpr int VIPT = (VITEMS + NT - 1) / NT;    // per thread (the last round may be partial)
  static_assert(KVEC % NT == 0 && VITEMS % 64 == 0, "tile staging must split evenly over the block");
};

// Per-block metadata of one work item: the byte offset of every prefix page of the chunk (this KV
// head), the tree's parents and ancestor masks (last chunk only), an input-error flag and (DMA kernel)
// the flag of a V value outside fp16's exact range.
struct AttnMeta {
  long long pgoff[ATT_CHUNK_PAGES];
  uint32_t anc[SR_MAX_TREE][SR_MAX_TREE / 32];
  int parent[SR_MAX_TREE];
  int bad;
  int vwide;
};

// Fills AttnMeta for pages [page0, page1) of trajectory b and, for the last chunk, its tree; validates
// the block table entries and the parent array this block reads. Whole block; returns the error flag.
template <int D, int E>
__device__ bool attn_meta(AttnMeta& m, bool ctx_ok, bool last, int page0, int page1, const int32_t* bt_b,
                          const int32_t* par_b, int T_, int Hkv, int g, int num_blocks) {
  const int tid = threadIdx.x, nt = blockDim.x;
  if (tid == 0) { m.bad = ctx_ok ? 0 : 1; m.vwide = 0; }
  __syncthreads();
  for (int p = page0 + tid; p < page1; p += nt) {
    int blk = bt_b[p];
    if (blk < 0 || blk >= num_blocks) { atomicOr(&m.bad, 1); blk = 0; }
    m.pgoff[p - page0] = (((long long)blk * Hkv + g) * ATT_BS) * D * (long long)E;
  }
  if (last) {
    for (int i = tid; i < T_; i += nt) {
      int p = par_b[i];
      if ((i == 0 && p != -1) || (i > 0 && (p < 0 || p >= i))) atomicOr(&m.bad, 1);
      m.parent[i] = p;
    }
    __syncthreads();
    if (!m.bad)
      for (int i = tid; i < T_; i += nt) {
        uint32_t a[SR_MAX_TREE / 32] = {0, 0, 0, 0};
        for (int u = i; u >= 0; u = m.parent[u]) a[u >> 5] |= 1u << (u & 31);
#pragma unroll
        for (int w = 0; w < SR_MAX_TREE / 32; ++w) m.anc[i][w] = a[w];
      }
  }
  __syncthreads();
  return m.bad != 0;
}

template <class AT, int D>
struct AttnSmem {
  using G = AttnGeom<AT, D>;
  __attribute__((aligned(16))) unsigned char k[2][G::KTILE];
  __attribute__((aligned(16))) unsigned char v[2][G::VTILE];
  AttnMeta meta;
};

// registers holding one tile's K and V while the previous tile is being computed
template <class AT, int D>
struct TileRegs {
  using G = AttnGeom<AT, D>;
  u32x4 k[G::KVPT];
  uint32_t v[G::VIPT][4][G::E];  // per item: 4 keys x (4 dims x E bytes)
};

// Work item (trajectory b, KV head g, chunk c, row group rg) of the register-staged path, rows
// [rg group_rows, min(R, (rg + 1) group_rows)) with group_rows <= ATT_ROWS. Whole block.
template <class AT, int D>
__device__ __forceinline__ void attn_item_regs(
    AttnSmem<AT, D>& sm, int b, int g, int c, int rg, const typename AT::T* __restrict__ q,
    const typename AT::T* __restrict__ k_cache, const typename AT::T* __restrict__ v_cache,
    const int32_t* __restrict__ block_table, const int32_t* __restrict__ ctx_len,
    const typename AT::T* __restrict__ k_tree, const typename AT::T* __restrict__ v_tree,
    const int32_t* __restrict__ parents, float* __restrict__ out, float* __restrict__ lse,
    float* __restrict__ part_o, float* __restrict__ part_ml, int T_, int Hq, int Hkv, int max_blocks,
    int num_blocks, float scale_log2, int R, int Rpad, int group_rows, int n_chunks_max, int cp) {
  using T = typename AT::T;
  using G = AttnGeom<AT, D>;
  constexpr int QKPL = AT::QKPL, KSTEP = 2 * QKPL, PKPL = AT::PKPL;
  constexpr int NQF = D / KSTEP;      // Q fragments per lane and row block
  constexpr int NDT = D / 32;         // 32-wide output tiles along D
  constexpr int NT = G::NT;
  constexpr int RB = ATT_RB;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
  const int G_ = Hq / Hkv;
  const int Lraw = ctx_len[b];
  const bool ctx_ok = Lraw >= 0 && Lraw <= max_blocks * ATT_BS;
  const int L = ctx_ok ? Lraw : 0;
  const int pages = (L + ATT_BS - 1) / ATT_BS;
  const int n_chunks = ctx_ok ? max(1, (pages + cp - 1) / cp) : 1;
  if (c >= n_chunks) return;
  const bool last = c == n_chunks - 1;
  const int page0 = c * cp, page1 = min(pages, page0 + cp);
  const int key0 = page0 * ATT_BS, key1 = min(L, page1 * ATT_BS);

  // ---- stage page offsets and (last chunk) the ancestor masks; validate what this block reads
  const bool bad = attn_meta<D, sizeof(T)>(sm.meta, ctx_ok, last, page0, page1, block_table + (size_t)b * max_blocks,
                                           parents + (size_t)b * T_, T_, Hkv, g, num_blocks);

  // ---- this wave's query rows: row r <-> (node t = r / G, head g*G + r % G); RB blocks of 32
  const int rend = min(R, (rg + 1) * group_rows);
  const int wrow0 = rg * group_rows + wave * RB * 32;
  int my_r[RB], my_t[RB];
  bool row_ok[RB];
  typename AT::qfrag qf[RB][NQF];
  uint32_t my_anc[RB][SR_MAX_TREE / 32];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    my_r[rb] = wrow0 + rb * 32 + (lane & 31);
    row_ok[rb] = my_r[rb] < rend;
    my_t[rb] = row_ok[rb] ? my_r[rb] / G_ : 0;
    const T* qp = q + (((size_t)b * T_ + my_t[rb]) * Hq + g * G_ + (row_ok[rb] ? my_r[rb] % G_ : 0)) * D;
#pragma unroll
    for (int kq = 0; kq < NQF; ++kq) {
      const int dd = kq * KSTEP + half * QKPL;
      if constexpr (QKPL == 8) {
        u32x4 z = {0, 0, 0, 0};
        if (row_ok[rb]) z = *(const u32x4*)(qp + dd);
        qf[rb][kq] = z;
      } else {
        qf[rb][kq] = row_ok[rb] ? qp[dd] : 0.f;
      }
    }
#pragma unroll
    for (int w = 0; w < SR_MAX_TREE / 32; ++w) my_anc[rb][w] = (last && !bad && row_ok[rb]) ? sm.meta.anc[my_t[rb]][w] : 0u;
  }

  f32x16 o[RB][NDT];
  float m_run[RB], l_run[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int i = 0; i < NDT; ++i) o[rb][i] = (f32x16){};
    m_run[rb] = -INFINITY;
    l_run[rb] = 0.f;
  }
  const bool wave_active = wrow0 < rend && !bad;

  // ---- tile schedule: prefix tiles of this chunk, then (last chunk) the tree tiles
  const int n_pre = (key1 - key0 + ATT_KT - 1) / ATT_KT;
  const int n_tiles = bad ? 0 : n_pre + (last ? (T_ + ATT_KT - 1) / ATT_KT : 0);

  // global -> registers for tile i. A key past the range is loaded from the range's last key instead
  // (so nothing past ctx_len is read and every staged value is finite); its score is masked to -inf,
  // so its K row never matters and its V row is multiplied by an exact zero.
  const unsigned char* kc_b = (const unsigned char*)k_cache;
  const unsigned char* vc_b = (const unsigned char*)v_cache;
  const unsigned char* kt_b = (const unsigned char*)(k_tree + ((size_t)b * T_ * Hkv + g) * D);
  const unsigned char* vt_b = (const unsigned char*)(v_tree + ((size_t)b * T_ * Hkv + g) * D);
  const int tree_rowb = Hkv * G::ROWB;                                  // bytes between tree nodes
  auto load_tile = [&](const unsigned char* kb, const unsigned char* vb, int t0, int lim, auto off_of,
                       TileRegs<AT, D>& r) {
#pragma unroll
    for (int j = 0; j < G::KVPT; ++j) {
      const int vi = tid + j * NT;
      const int key = vi / G::NCH, ch = vi % G::NCH;
      r.k[j] = *(const u32x4*)(kb + off_of(min(t0 + key, lim - 1)) + ch * 16);
    }
#pragma unroll
    for (int it = 0; it < G::VIPT; ++it) {
      const int item = tid + it * NT;
      if (item >= G::VITEMS) break;                   // uniform per wave
      const int kg = item / (D / 4), dg = item % (D / 4);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const unsigned char* src = vb + off_of(min(t0 + kg * 4 + j, lim - 1)) + dg * 4 * G::E;
        if constexpr (G::E == 2) {
          const u32x2 z = *(const u32x2*)src;
          r.v[it][j][0] = z[0];
          r.v[it][j][1] = z[1];
        } else {
          const u32x4 z = *(const u32x4*)src;
#pragma unroll
          for (int w = 0; w < 4; ++w) r.v[it][j][w] = z[w];
        }
      }
    }
  };
  auto fetch = [&](int i, TileRegs<AT, D>& r) {
    if (i < n_pre) {
      load_tile(kc_b, vc_b, key0 + i * ATT_KT, key1,
                [&](int kidx) -> long long { return sm.meta.pgoff[(kidx >> 4) - page0] + (kidx & 15) * G::ROWB; }, r);
    } else {
      load_tile(kt_b, vt_b, (i - n_pre) * ATT_KT, T_, [&](int kidx) -> long long { return (long long)kidx * tree_rowb; },
                r);
    }
  };
  // registers -> LDS stage (K row-major with chunk swizzle, V transposed with group swizzle; bf16 V is
  // widened to the fp32 V^T element exactly)
  auto stash = [&](int st, const TileRegs<AT, D>& r) {
#pragma unroll
    for (int j = 0; j < G::KVPT; ++j) {
      const int vi = tid + j * NT;
      const int key = vi / G::NCH, ch = vi % G::NCH;
      *(u32x4*)(sm.k[st] + key * G::ROWB + ((ch ^ (key & (G::NCH - 1))) * 16)) = r.k[j];
    }
#pragma unroll
    for (int it = 0; it < G::VIPT; ++it) {
      const int item = tid + it * NT;
      if (item >= G::VITEMS) break;
      const int kg = item / (D / 4), dg = item % (D / 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = dg * 4 + i;
        unsigned char* dst = sm.v[st] + d * G::VROWB + ((kg ^ vswz(d)) * 4 * G::VE);
        f32x4 h;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if constexpr (G::E == 2) {
            const uint32_t w = r.v[it][j][i >> 1];
            h[j] = bf2f((i & 1) ? (w >> 16) : (w & 0xffffu));
          } else {
            h[j] = __uint_as_float(r.v[it][j][i]);
          }
        }
        *(f32x4*)dst = h;
      }
    }
  };
  static_assert(G::VE == 4, "V^T is staged as fp32");

  auto compute = [&](int i, int st) {
    const bool tree = i >= n_pre;
    const int t0 = tree ? (i - n_pre) * ATT_KT : key0 + i * ATT_KT;
    const unsigned char* ks_ = sm.k[st];
    const unsigned char* vs_ = sm.v[st];
    // scores S^T: each K fragment feeds every row block
    f32x16 s[RB][2];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) s[rb][0] = s[rb][1] = (f32x16){};
#pragma unroll
    for (int kq = 0; kq < NQF; ++kq) {
      const int e = kq * KSTEP + half * QKPL;           // first element this lane supplies
      const int ch = (e * G::E) / 16;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const int key = kt * 32 + (lane & 31);
        const unsigned char* p = ks_ + key * G::ROWB + ((ch ^ (key & (G::NCH - 1))) * 16) + (e * G::E) % 16;
        typename AT::qfrag kf;
        if constexpr (QKPL == 8) kf = *(const u32x4*)p; else kf = *(const float*)p;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) s[rb][kt] = AT::mma_qk(kf, qf[rb][kq], s[rb][kt]);
      }
    }
    // online softmax per row block; vis holds one bit per key of each 32-key subtile, pre-shifted by
    // this lane half's row offset
    typename AT::pfrag pf[RB][2][16 / PKPL];
    const bool full = !tree && t0 + ATT_KT <= key1;      // every key of the tile is visible to every row
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      uint32_t vis[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const int kb = t0 + kt * 32;
        uint32_t v;
        if (tree) {
          const int wi = kb >> 5;
          v = wi == 0 ? my_anc[rb][0] : wi == 1 ? my_anc[rb][1] : wi == 2 ? my_anc[rb][2] : my_anc[rb][3];
        } else {
          const int nv = key1 - kb;
          v = nv >= 32 ? 0xffffffffu : (nv <= 0 ? 0u : ((1u << nv) - 1u));
        }
        vis[kt] = v >> (4 * half);
      }
      if (!full) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const bool ok = (vis[kt] >> (8 * (r >> 2) + (r & 3))) & 1u;
            s[rb][kt][r] = ok ? s[rb][kt][r] : -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[rb][kt][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      // the reference max moves only when the tile max exceeds it by more than 2^8 (P in [0, 256]), so
      // the accumulator is rarely rescaled
      const float tmax = mx * scale_log2;
      const float m_new = (tmax > m_run[rb] + 8.f) ? tmax : m_run[rb];
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run[rb] - m_use);
      float psum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[rb][kt][r], scale_log2, -m_use));
          psum += p;
          pf[rb][kt][r] = p;
        }
      l_run[rb] = l_run[rb] * alpha + psum;
      m_run[rb] = m_new;
      if (__ballot(alpha != 1.f) != 0) {      // rescale only when some row's running max moved
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) o[rb][dt] *= alpha;
      }
    }
    // O^T += V^T P^T; each V fragment feeds every row block
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int kq = 0; kq < 16 / PKPL; ++kq) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const int d = dt * 32 + (lane & 31);
          const unsigned char* vrow = vs_ + d * G::VROWB;
          const int sw = vswz(d);
          const int key = kt * 32 + tile_row(kq, half);
          const float vf = *(const float*)(vrow + (((key >> 2) ^ sw) * 16) + (key & 3) * 4);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) o[rb][dt] = AT::mma_pv(vf, pf[rb][kt][kq], o[rb][dt]);
        }
      }
  };

  // ---- software pipeline: tile i+1 is in flight (registers) while tile i is computed from LDS
  if (n_tiles > 0) {
    TileRegs<AT, D> regs;
    fetch(0, regs);
    stash(0, regs);
    __syncthreads();
    for (int i = 0; i < n_tiles; ++i) {
      const int st = i & 1;
      const bool more = i + 1 < n_tiles;
      if (more) fetch(i + 1, regs);
      if (wave_active) compute(i, st);
      if (more) stash(st ^ 1, regs);
      __syncthreads();
    }
  }

  // ---- write the normalised result (single chunk) or a partial (m, l, O/l)
  const float qnan = __uint_as_float(0x7fc00000u);
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const float l_tot = l_run[rb] + __shfl_xor(l_run[rb], 32, 64);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    if (!row_ok[rb]) continue;
    if (n_chunks == 1) {
      const int h = g * G_ + my_r[rb] % G_;
      float* op = out + (((size_t)b * T_ + my_t[rb]) * Hq + h) * D;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int i = 0; i < 16; i += 4) {
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = bad ? qnan : o[rb][dt][i + e] * inv;
          *(f32x4*)(op + dt * 32 + tile_row(i, half)) = v;
        }
      if (lse != nullptr && half == 0)
        lse[((size_t)b * T_ + my_t[rb]) * Hq + h] = bad ? qnan : (m_run[rb] + log2f(l_tot)) * kLn2;
    } else {
      const size_t pr = (((size_t)b * Hkv + g) * n_chunks_max + c) * Rpad + my_r[rb];
      float* op = part_o + pr * D;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int i = 0; i < 16; i += 4) {
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = o[rb][dt][i + e] * inv;
          *(f32x4*)(op + dt * 32 + tile_row(i, half)) = v;
        }
      if (half == 0) {
        part_ml[pr * 2 + 0] = bad ? qnan : m_run[rb];
        part_ml[pr * 2 + 1] = bad ? qnan : l_tot;
      }
    }
  }
}

// fp32 inputs: one block per item, grid (B Hkv row_groups, chunks).
template <int D>
__global__ __launch_bounds__(ATT_NW * 64) void k_tree_attn(
    const float* __restrict__ q, const float* __restrict__ k_cache, const float* __restrict__ v_cache,
    const int32_t* __restrict__ block_table, const int32_t* __restrict__ ctx_len, const float* __restrict__ k_tree,
    const float* __restrict__ v_tree, const int32_t* __restrict__ parents, float* __restrict__ out,
    float* __restrict__ lse, float* __restrict__ part_o, float* __restrict__ part_ml, int T_, int Hq, int Hkv,
    int max_blocks, int num_blocks, float scale_log2, int R, int Rpad, int row_groups, int group_rows,
    int n_chunks_max, int cp) {
  __shared__ AttnSmem<AttnF32, D> sm;
  const int rg = blockIdx.x % row_groups, bg = blockIdx.x / row_groups;
  attn_item_regs<AttnF32, D>(sm, bg / Hkv, bg % Hkv, blockIdx.y, rg, q, k_cache, v_cache, block_table, ctx_len,
                             k_tree, v_tree, parents, out, lse, part_o, part_ml, T_, Hq, Hkv, max_blocks, num_blocks,
                             scale_log2, R, Rpad, group_rows, n_chunks_max, cp);
}

// bf16 items that k_tree_attn_dma listed (a V value outside fp16's exact range), recomputed with V in
// fp32. redo[0] = count, redo[1..] = item indices ((c B + b) Hkv + g) row_groups + rg. The loop bound
// is read once per block and is uniform, so every wave runs the same iterations.
template <int D>
__global__ __launch_bounds__(ATT_NW * 64) void k_tree_attn_redo(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k_cache, const bf16_t* __restrict__ v_cache,
    const int32_t* __restrict__ block_table, const int32_t* __restrict__ ctx_len, const bf16_t* __restrict__ k_tree,
    const bf16_t* __restrict__ v_tree, const int32_t* __restrict__ parents, float* __restrict__ out,
    float* __restrict__ lse, float* __restrict__ part_o, float* __restrict__ part_ml, int B_, int T_, int Hq,
    int Hkv, int max_blocks, int num_blocks, float scale_log2, int R, int Rpad, int row_groups, int group_rows,
    int n_chunks_max, int cp, int n_items, const unsigned* __restrict__ redo) {
  __shared__ AttnSmem<AttnBf16Wide, D> sm;
  const int n = min((int)__builtin_amdgcn_readfirstlane(redo[0]), n_items);
  for (int k = blockIdx.x; k < n; k += gridDim.x) {
    const int item = (int)__builtin_amdgcn_readfirstlane(redo[1 + k]);
    if (item < 0 || item >= n_items) continue;   // uniform
    const int rg = item % row_groups, bg = item / row_groups;
    const int g = bg % Hkv, b = (bg / Hkv) % B_, c = bg / (Hkv * B_);
    __syncthreads();                              // the previous item's LDS reads are done
    attn_item_regs<AttnBf16Wide, D>(sm, b, g, c, rg, q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree,
                                    parents, out, lse, part_o, part_ml, T_, Hq, Hkv, max_blocks, num_blocks,
                                    scale_log2, R, Rpad, group_rows, n_chunks_max, cp);
  }
}

// ============================================================================ bf16, direct-to-LDS
// The bf16 path streams K and V tiles from HBM straight into LDS (global_load_lds_dwordx4) through a
// four-slot ring: while tile i is finished and tile i+1 prepared, tiles i+2 and i+3 are in flight. In LDS,
// 16-byte chunk c of key row k sits at chunk position c ^ (k mod NCH) for K and c ^ (4 (k mod 4) mod NCH)
// for V, chosen by the source address each lane loads, which keeps the operand reads free of bank
// conflicts. Once per tile the block converts the tile's V from bf16 to fp16 in place, and the P V
// MFMAs read their V^T fragments straight from the row-major tile with the transposing LDS read
// (ds_read_b64_tr_b16: within 16 lanes, lane i receives element i mod 4 of the 8-byte rows addressed by
// lanes i/4, 4 + i/4, 8 + i/4 and 12 + i/4, so lanes addressing four keys of four consecutive dims each
// receive four keys of one dim). Each wave computes the scores of tile i+1 in the same instruction
// stream as the exponentials of tile i, so its matrix and vector work overlap. One barrier per tile.
template <int D>
struct DmaGeom {
  static constexpr int ROWB = D * 2;                   // bytes of one K or V row
  static constexpr int NCH = ROWB / 16;                // 16-byte chunks per row
  static constexpr int KPB = 1024 / ROWB;              // keys per 1 KB DMA block
  static constexpr int TILE = ATT_KT * ROWB;           // bytes of a K (or raw V) tile
  static constexpr int BLK = TILE / 1024;              // DMA blocks per tile, each of K and V
  static constexpr int CITEMS = TILE / 16;             // 16-byte chunks of a V tile (conversion items)
  static constexpr int CPL = CITEMS / 64;                // V chunks of a tile per lane of one wave
  static constexpr int CD = CPL - (ATT_NW - 1);          // converted per lane by the DMA wave; one by each other wave
  static_assert(CITEMS % 64 == 0 && CD >= 1, "tile split");
  static_assert(2 * BLK <= 63, "one tile of DMA per wave must fit the vmcnt counter");
  static_assert(KPB % 4 == 0, "a DMA block holds whole 4-key groups");
};

// max of x over lanes l and l ^ 32 (v_permlane32_swap exchanges the two 32-lane halves without LDS)
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// chunk-position swizzle of V row k: the eight rows of one transposing read (k mod 4 = 0..3, twice)
// take four different 64-byte column groups
template <int NCH> __device__ __forceinline__ int vswz(int k) { return (4 * (k & 3)) & (NCH - 1); }

// Complete this wave's LDS writes and its DMA for the next tile, then meet the block. The DMA wave (2 BLK
// transfers per tile) may leave the transfers of the tile after that in flight when `ahead`.
template <int D>
__device__ __forceinline__ void attn_sync(bool dma_wave, bool ahead) {
  constexpr int BLK = DmaGeom<D>::BLK;
  if (!dma_wave || !ahead) {
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  } else {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(2 * BLK) : "memory");
  }
}

// One work item (chunk c of trajectory b, KV head g, row group rg); item = ((c B + b) Hkv + g) row_groups
// + rg. Whole block; returns with the block's DMA drained. ring: four slots of a K tile then a V tile
// (bf16 as loaded, fp16 once converted).
template <int D>
__device__ __forceinline__ void attn_item_dma(
    int item, unsigned char (&ring)[4][2 * DmaGeom<D>::TILE], AttnMeta& meta,
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k_cache, const bf16_t* __restrict__ v_cache,
    const int32_t* __restrict__ block_table, const int32_t* __restrict__ ctx_len, const bf16_t* __restrict__ k_tree,
    const bf16_t* __restrict__ v_tree, const int32_t* __restrict__ parents, float* __restrict__ out,
    float* __restrict__ lse, float* __restrict__ part_o, float* __restrict__ part_ml, int B_, int T_, int Hq,
    int Hkv, int max_blocks, int num_blocks, float scale_log2, int R, int Rpad, int row_groups, int group_rows,
    int n_chunks_max, int cp, unsigned* __restrict__ redo) {
  using G = DmaGeom<D>;
  constexpr int NQF = D / 16;         // Q fragments per lane
  constexpr int NDT = D / 32;         // 32-wide output tiles along D

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;
  const int rg = item % row_groups, bg = item / row_groups;
  const int g = bg % Hkv, b = (bg / Hkv) % B_, c = bg / (Hkv * B_);
  const int G_ = Hq / Hkv;
  const int Lraw = ctx_len[b];
  const bool ctx_ok = Lraw >= 0 && Lraw <= max_blocks * ATT_BS;
  const int L = ctx_ok ? Lraw : 0;
  const int pages = (L + ATT_BS - 1) / ATT_BS;
  const int n_chunks = ctx_ok ? max(1, (pages + cp - 1) / cp) : 1;
  if (c >= n_chunks) return;
  const bool last = c == n_chunks - 1;
  const int page0 = c * cp, page1 = min(pages, page0 + cp);
  const int key0 = page0 * ATT_BS, key1 = min(L, page1 * ATT_BS);

  // ---- this wave's 32 query rows: row r <-> (node t = r / G, head g*G + r % G); their loads are issued
  // before the item's metadata, so both are in flight together
  const int rend = min(R, (rg + 1) * group_rows);   // this row group's rows: [rg group_rows, rend)
  const int my_r = rg * group_rows + wave * 32 + (lane & 31);
  const bool row_ok = my_r < rend;
  const int my_t = row_ok ? my_r / G_ : 0;
  u32x4 qf[NQF];
  {
    const bf16_t* qp = q + (((size_t)b * T_ + my_t) * Hq + g * G_ + (row_ok ? my_r % G_ : 0)) * D;
#pragma unroll
    for (int kq = 0; kq < NQF; ++kq) {
      u32x4 z = {0, 0, 0, 0};
      if (row_ok) z = *(const u32x4*)(qp + kq * 16 + half * 8);
      qf[kq] = z;
    }
  }

  const bool bad = attn_meta<D, 2>(meta, ctx_ok, last, page0, page1, block_table + (size_t)b * max_blocks,
                                   parents + (size_t)b * T_, T_, Hkv, g, num_blocks);
  // the K/V DMA below is invisible to the compiler's wait counting, so every compiler-tracked load must
  // have landed before the first transfer is issued
#pragma unroll
  for (int kq = 0; kq < NQF; ++kq) asm volatile("" ::"v"(qf[kq]));

  f32x16 o[NDT];
#pragma unroll
  for (int i = 0; i < NDT; ++i) o[i] = (f32x16){};
  float m_run = -INFINITY, l_run = 0.f;
  // Roles. A row group holds at most ATT_ROWS - 32 rows (attn_plan), so wave n_act has no query rows: it
  // issues all of the DMA, pacing itself on the memory system, and converts most of every V tile to fp16;
  // each other wave converts one 16-byte chunk per lane of it. The DMA wave runs its own loop (the same
  // barriers), so its conversion registers never share the compute waves' code. Measured per 64-key tile
  // at the 7B shape (about 4.4k cycles): issuing a tile's 32 transfers took the DMA wave about 1.9k cycles
  // and converting all of its V about 2.0k; the second compute wave of each SIMD about 3.3-3.5k.
  const int n_act = min(ATT_NW - 1, (rend - rg * group_rows + 31) / 32);
  const bool wave_active = wave < n_act && !bad;
  const bool dma_wave = wave == n_act;

  const int n_pre = (key1 - key0 + ATT_KT - 1) / ATT_KT;
  const int n_tiles = bad ? 0 : n_pre + (last ? (T_ + ATT_KT - 1) / ATT_KT : 0);

  const unsigned char* kc_b = (const unsigned char*)k_cache;
  const unsigned char* vc_b = (const unsigned char*)v_cache;
  const unsigned char* kt_b = (const unsigned char*)(k_tree + ((size_t)b * T_ * Hkv + g) * D);
  const unsigned char* vt_b = (const unsigned char*)(v_tree + ((size_t)b * T_ * Hkv + g) * D);
  const long long tree_rowb = (long long)Hkv * G::ROWB;

  // global -> LDS for tile i. A key past the range is loaded from the range's last key instead (nothing
  // past ctx_len is read and every staged value is finite); its score is masked to -inf, so its K row
  // never matters and its V row is multiplied by an exact zero.
  // Source of DMA block blk (KPB keys x 1 KB) of tile i for this lane: the K and V byte offsets.
  auto block_src = [&](int i, int blk, long long& ko, long long& vo) __attribute__((always_inline)) {
    const bool tree = i >= n_pre;
    const int t0 = tree ? (i - n_pre) * ATT_KT : key0 + i * ATT_KT;
    int ln = lane;
    asm volatile("" : "+v"(ln));                  // not hoisted out of the tile loop
    const int kk = blk * G::KPB + ln / G::NCH, pos = ln % G::NCH;
    long long off;
    if (tree) {
      off = (long long)min(t0 + kk, T_ - 1) * tree_rowb;
    } else {
      const int key = min(t0 + kk, key1 - 1);
      off = meta.pgoff[(key >> 4) - page0] + (key & 15) * G::ROWB;
    }
    const long long base = tree ? (long long)(kt_b - kc_b) : 0;   // tree rows are addressed from kc_b
    ko = base + off + ((pos ^ (kk & (G::NCH - 1))) * 16);
    vo = (tree ? (long long)(vt_b - vc_b) : 0) + off + ((pos ^ vswz<G::NCH>(kk)) * 16);
  };
  // one producer wave issues the whole tile. A full prefix tile is four whole pages: each page's K and V
  // bases are uniform (scalar registers) and a block's per-lane offset inside its page depends only on
  // the block's position in the page, so every transfer is a scalar base plus one of BPP lane offsets.
  // Other tiles take the per-lane clamped path.
  auto issue_prod = [&](int i, unsigned char* slot) __attribute__((always_inline)) {
    const bool tree = i >= n_pre;
    const int t0 = tree ? 0 : key0 + i * ATT_KT;
    if (!tree && t0 + ATT_KT <= key1) {
      constexpr int BPP = ATT_BS / G::KPB;          // DMA blocks per page
      const int pg = (t0 >> 4) - page0;
      int ln = lane;
      asm volatile("" : "+v"(ln));                  // lane offsets are rebuilt per tile, not kept live
      uint32_t ko[BPP], vo[BPP];
#pragma unroll
      for (int j = 0; j < BPP; ++j) {
        const int kr = j * G::KPB + ln / G::NCH, pos = ln % G::NCH;   // key row in the page, chunk
        ko[j] = kr * G::ROWB + ((pos ^ (kr & (G::NCH - 1))) * 16);
        vo[j] = kr * G::ROWB + ((pos ^ vswz<G::NCH>(kr)) * 16);
      }
      const uint32_t lds0 = __builtin_amdgcn_readfirstlane(
          (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)slot);
#pragma unroll
      for (int p = 0; p < ATT_KT / ATT_BS; ++p) {
        const long long po0 = meta.pgoff[pg + p];   // same for every lane: made scalar
        const long long po = (long long)(((unsigned long long)__builtin_amdgcn_readfirstlane((uint32_t)(po0 >> 32)) << 32) |
                                         __builtin_amdgcn_readfirstlane((uint32_t)po0));
        const unsigned char* kb = kc_b + po;
        const unsigned char* vb = vc_b + po;
#pragma unroll
        for (int j = 0; j < BPP; ++j) {
          const int blk = p * BPP + j;
          lds_dma16_sv(ko[j], kb, lds0 + blk * 1024);
          lds_dma16_sv(vo[j], vb, lds0 + G::TILE + blk * 1024);
        }
      }
    } else {
      for (int blk = 0; blk < G::BLK; ++blk) {
        long long ko, vo;
        block_src(i, blk, ko, vo);
        lds_dma16_manual(kc_b + ko, slot + blk * 1024);
        lds_dma16_manual(vc_b + vo, slot + G::TILE + blk * 1024);
      }
    }
  };
  auto issue = [&](int i, unsigned char* slot) __attribute__((always_inline)) { issue_prod(i, slot); };
  // V of a tile, bf16 -> fp16 in place: every converting lane takes whole 16-byte chunks (their positions
  // do not matter). The reads (conv_load) are issued early and the converted chunks written later
  // (conv_store), so the LDS latency overlaps other work. The conversion is exact for magnitudes in
  // [2^-14, 65280] and truncates smaller ones to fp16's subnormal step, an absolute error below 2^-24;
  // larger ones would overflow. Each converting lane keeps the largest magnitude pattern of everything it
  // converts (two 16-bit lanes per register): an item is recomputed with fp32 V when that exceeds 65280
  // (pattern 0x477f; inf and NaN included) or when the item's largest |v| is below 2^-6 (pattern 0x3c80),
  // where 2^-24 would no longer be negligible against the scale of V.
  // The DMA wave converts chunks lane + 64 k (k < CD) of a tile; every other wave converts one chunk,
  // (CD + its index among the other waves) * 64 + lane, beside its own work: the DMA wave's issue is paced
  // by the memory system and takes a large part of a tile's time.
  u16x2 vmag_hi = {0, 0};
  auto conv_chunk = [&](const u32x4& x, unsigned char* dst) __attribute__((always_inline)) {
    // two values per instruction, rounding toward zero: exact for every value in fp16's normal range,
    // within one subnormal step (2^-24) below it; out-of-range items are recomputed anyway
    u32x4 h;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      h[w] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(__uint_as_float(x[w] << 16),
                                                                     __uint_as_float(x[w] & 0xffff0000u)));
      vmag_hi = __builtin_elementwise_max(vmag_hi, __builtin_bit_cast(u16x2, x[w] & 0x7fff7fffu));
    }
    *(u32x4*)dst = h;
  };
  u32x4 cw[G::CD];
  auto conv_load = [&](const unsigned char* v) __attribute__((always_inline)) {
    int ln = lane;
    asm volatile("" : "+v"(ln));                  // addresses are not hoisted out of the tile loop
#pragma unroll
    for (int k = 0; k < G::CD; ++k) cw[k] = *(const u32x4*)(v + (ln + k * 64) * 16);
  };
  auto conv_store = [&](unsigned char* v) __attribute__((always_inline)) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
#pragma unroll
    for (int k = 0; k < G::CD; ++k) conv_chunk(cw[k], v + (ln + k * 64) * 16);
  };
  const int help_off = ((G::CD + (wave < n_act ? wave : wave - 1)) * 64 + lane) * 16;   // other waves' chunk
  // scores S^T = K Q^T of the tile in ks
  auto qk = [&](const unsigned char* ks, f32x16 (&s)[2]) {
    s[0] = s[1] = (f32x16){};
#pragma unroll
    for (int kq = 0; kq < NQF; ++kq) {
      const int ch = 2 * kq + half;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const int key = kt * 32 + (lane & 31);
        const u32x4 kf = *(const u32x4*)(ks + key * G::ROWB + ((ch ^ (key & (G::NCH - 1))) * 16));
        s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kf),
                                                        __builtin_bit_cast(bf16x8, qf[kq]), s[kt], 0, 0, 0);
      }
    }
  };
  // mask, online softmax and O^T += V^T P^T for tile i (scores s); the next tile's scores (K in nks) are
  // computed into sn in the same basic block as this tile's exponentials
  float f_muse = 0.f, f_alpha = 1.f;
  // mask of tile i's scores (a whole prefix tile needs none)
  auto tile_full = [&](int i) -> bool { return i < n_pre && key0 + i * ATT_KT + ATT_KT <= key1; };
  auto mask_tile = [&](int i, f32x16 (&s)[2]) {
    const bool tree = i >= n_pre;
    const int t0 = tree ? (i - n_pre) * ATT_KT : key0 + i * ATT_KT;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int kb = t0 + kt * 32;
      uint32_t v;
      if (tree) {
        v = (row_ok && last) ? meta.anc[my_t][kb >> 5] : 0u;
      } else {
        const int nv = key1 - kb;
        v = nv >= 32 ? 0xffffffffu : (nv <= 0 ? 0u : ((1u << nv) - 1u));
      }
      v >>= 4 * half;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool ok = (v >> (8 * (r >> 2) + (r & 3))) & 1u;
        s[kt][r] = ok ? s[kt][r] : -INFINITY;
      }
    }
  };
  // from a lane's max of a tile's (masked) scores: the row max, the new reference max and the accumulator
  // rescale. The reference max moves only when the tile max exceeds it by more than 2^8, so the accumulator
  // is rarely rescaled. Run for the first tile and for a tile whose weights outgrow the reference
  // (finish_rest).
  auto commit_max = [&](float mx) {
    mx = max_halves(mx);
    const float tmax = mx * scale_log2;
    const float m_new = (tmax > m_run + 8.f) ? tmax : m_run;
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    if (__ballot(alpha != 1.f) != 0) {      // rescale only when some row's running max moved
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) o[dt] *= alpha;
    }
    m_run = m_new;
    f_muse = m_use;
    f_alpha = alpha;
  };
  auto finish_max = [&](int i, f32x16 (&s)[2]) {
    if (!tile_full(i)) mask_tile(i, s);
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kt][r]);
    commit_max(mx);
  };
  // exponentials of tile i (scores s) against the current reference max, computed in one basic block with
  // the scores of the next tile (K in nks, into sn), then O^T += V^T P^T with V of tile i (vs); with `next`,
  // the mask of the next tile's scores (partial or tree tiles)
  auto finish_rest = [&](int i, f32x16 (&s)[2], const unsigned char* vs, const unsigned char* nks, f32x16 (&sn)[2],
                         bool next) {
    float m_use = f_muse;
    // From here on one basic block, laid out by hand with scheduling fences: each step issues the
    // K fragment reads one step ahead, two score MFMAs of the next tile and 32/NQF of this tile's
    // exponentials (the matrix core works while the vector ALU exponentiates); then the P V MFMAs
    // with their V fragment reads two ahead.
    constexpr int EPQ = 32 / NQF;                 // exponentials per score step
    f16x8 pf[2][2];
    float psum = 0.f;
    // weights of scores e, e+1 of this tile into pf; the row sum takes the fp16 weights the P V product
    // uses, in fp32 (v_dot2_f32_f16)
    auto exp_pair = [&](int e) __attribute__((always_inline)) {
      const int kt = e >> 4, r = e & 15;
      const _Float16 h0 = (_Float16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[kt][r], scale_log2, -m_use));
      const _Float16 h1 = (_Float16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[kt][r + 1], scale_log2, -m_use));
      pf[kt][r >> 3][r & 7] = h0;
      pf[kt][r >> 3][(r & 7) + 1] = h1;
      psum = __builtin_amdgcn_fdot2((f16x2){h0, h1}, (f16x2){(_Float16)1.f, (_Float16)1.f}, psum, false);
    };
    u32x4 kf[2][2];
    auto kread = [&](int kq, u32x4 (&dst)[2]) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const int key = kt * 32 + (lane & 31), ch = 2 * kq + half;
        dst[kt] = *(const u32x4*)(nks + key * G::ROWB + ((ch ^ (key & (G::NCH - 1))) * 16));
      }
    };
    sn[0] = sn[1] = (f32x16){};
    kread(0, kf[0]);
#pragma unroll
    for (int kq = 0; kq < NQF; ++kq) {
      if (kq + 1 < NQF) kread(kq + 1, kf[(kq + 1) & 1]);
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
        sn[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kf[kq & 1][kt]),
                                                         __builtin_bit_cast(bf16x8, qf[kq]), sn[kt], 0, 0, 0);
#pragma unroll
      for (int e = kq * EPQ; e < (kq + 1) * EPQ; e += 2) exp_pair(e);
      __builtin_amdgcn_sched_barrier(0);
    }
    // The reference max is lazy: no tile max is taken while every lane's weights stay small. A tile whose
    // half-row weights add up past 2^14 (or overflow) moves the reference to its own max (the row max and
    // the accumulator rescale as for the first tile) and is weighted again; weights below 2^14 are exact in
    // fp16 up to its rounding, like those below 2^8.
    if (__ballot(!(psum <= 16384.f)) != 0) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kt][r]);
      const float a0 = f_alpha;
      commit_max(mx);
      f_alpha *= a0;
      m_use = f_muse;
      psum = 0.f;
#pragma unroll
      for (int e = 0; e < 32; e += 2) exp_pair(e);
    }
    l_run = l_run * f_alpha + psum;
    f_alpha = 1.f;
    constexpr int NPV = 4 * NDT;                  // P V MFMAs per tile
    f16x8 vf[3];
    // V^T fragment (dims dt*32 + lane%32; keys of k-slot 8*half + j: 16 kq + 8 (j/4) + 4 half + j%4) as two
    // transposing reads of four keys each: lane s of a 16-lane group addresses key row kb + s/4, dims
    // d0 + 4 (s mod 4) .. + 3
    auto vread = [&](int j) __attribute__((always_inline)) -> f16x8 {
      const int kt = j / (2 * NDT), kq = (j / NDT) & 1, dt = j % NDT;
      const int s16 = lane & 15, d0 = dt * 32 + 16 * ((lane >> 4) & 1);
      const int col = d0 + 4 * (s16 & 3);             // first of the four dims this lane addresses
      f16x4 part[2];
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int row = kt * 32 + kq * 16 + 8 * r + 4 * half + (s16 >> 2);
        const unsigned char* a = vs + row * G::ROWB + (((col >> 3) ^ vswz<G::NCH>(row)) * 16) + (col & 7) * 2;
        part[r] = __builtin_bit_cast(f16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                                (__attribute__((address_space(3))) v4i16*)(a)));
      }
      return (f16x8){part[0][0], part[0][1], part[0][2], part[0][3], part[1][0], part[1][1], part[1][2], part[1][3]};
    };
    if (next && !tile_full(i + 1)) mask_tile(i + 1, sn);
    vf[0] = vread(0);
    vf[1] = vread(1);
#pragma unroll
    for (int j = 0; j < NPV; ++j) {
      if (j + 2 < NPV) vf[(j + 2) % 3] = vread(j + 2);
      const int kt = j / (2 * NDT), kq = (j / NDT) & 1, dt = j % NDT;
      o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf[j % 3], pf[kt][kq], o[dt], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // ---- pipeline. Compute waves, step(i): wait for tile i+1, then finish tile i while computing the scores of
  // tile i+1 (slot of tile i: si). DMA wave, the same barriers: wait for tile i+1 (tiles i+2, i+3 may stay in
  // flight), read tile i+1's V, refill the slot of tile i-1 with tile i+3 (whose issue stalls overlap the
  // reads), convert tile i+1's V; it is consumed after the next barrier.
  f32x16 sa[2], sb[2];
  auto step = [&](int i, int si, f32x16 (&s)[2], f32x16 (&sn)[2]) {
    const int sn_ = (si + 1) & 3;
    attn_sync<D>(false, false);
    const bool cvn = i + 1 < n_tiles;
    unsigned char* hc = ring[sn_] + G::TILE + help_off;   // this wave's chunk of tile i+1's V
    u32x4 hw;
    if (cvn) hw = *(const u32x4*)hc;
    // after the last tile the next scores come from a slot no DMA is writing and are discarded
    if (wave_active) finish_rest(i, s, ring[si] + G::TILE, ring[sn_], sn, cvn);
    if (cvn) conv_chunk(hw, hc);
  };
  if (n_tiles > 0) {
    if (dma_wave) {
      issue(0, ring[0]);
      if (n_tiles > 1) issue(1, ring[1]);
      attn_sync<D>(true, n_tiles > 1);          // tile 0 landed (tile 1 may be in flight)
      if (n_tiles > 2) issue(2, ring[2]);
      conv_load(ring[0] + G::TILE);
      conv_store(ring[0] + G::TILE);
      int si = 0;
      for (int i = 0; i < n_tiles; ++i) {
        const int sn_ = (si + 1) & 3, sf = (si + 3) & 3;
        attn_sync<D>(true, i + 2 < n_tiles);
        const bool cv = i + 1 < n_tiles;
        if (cv) conv_load(ring[sn_] + G::TILE);
        if (i + 3 < n_tiles) issue(i + 3, ring[sf]);
        if (cv) conv_store(ring[sn_] + G::TILE);
        si = (si + 1) & 3;
      }
    } else {
      attn_sync<D>(false, false);               // tile 0 landed
      {
        unsigned char* hc = ring[0] + G::TILE + help_off;
        const u32x4 hw = *(const u32x4*)hc;
        if (wave_active) {
          qk(ring[0], sa);
          finish_max(0, sa);
        }
        conv_chunk(hw, hc);
      }
      int si = 0;
      for (int i = 0; i < n_tiles; i += 2) {
        step(i, si, sa, sb);
        si = (si + 1) & 3;
        if (i + 1 < n_tiles) {
          step(i + 1, si, sb, sa);
          si = (si + 1) & 3;
        }
      }
    }
  }

  // ---- V too large for fp16 or too small for its subnormal step: list the item for the fp32-V
  // recomputation (its outputs written below are then overwritten before anything reads them). Items
  // without tiles (invalid input) are not listed.
  {
    uint32_t hi = max((uint32_t)vmag_hi[0], (uint32_t)vmag_hi[1]);
    hi = (uint32_t)warp_max_i((int)hi);
    if (lane == 0) atomicMax(&meta.vwide, (int)hi);
    __syncthreads();
    if (threadIdx.x == 0 && n_tiles > 0 && (meta.vwide > 0x477f || meta.vwide < 0x3c80)) {
      const unsigned k = atomicAdd(redo, 1u);
      redo[1 + k] = (unsigned)item;
    }
  }

  // ---- write the normalised result (single chunk) or a partial (m, l, O/l)
  const float qnan = __uint_as_float(0x7fc00000u);
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (!row_ok) return;
  if (n_chunks == 1) {
    const int h = g * G_ + my_r % G_;
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

// Persistent blocks (one per CU) take work items from a counter, in the order k_attn_order lists them
// (most tiles first, so the last items to start are the shortest and the blocks end close together). Every
// wave runs the same iterations (the item is broadcast through LDS), and the loop ends for all once the
// counter passes the list. Between items the block meets with LDS-only barriers: the previous item's
// global stores need not have landed before the next item starts.
template <int D>
__global__ __launch_bounds__(ATT_NW * 64) void k_tree_attn_dma(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k_cache, const bf16_t* __restrict__ v_cache,
    const int32_t* __restrict__ block_table, const int32_t* __restrict__ ctx_len, const bf16_t* __restrict__ k_tree,
    const bf16_t* __restrict__ v_tree, const int32_t* __restrict__ parents, float* __restrict__ out,
    float* __restrict__ lse, float* __restrict__ part_o, float* __restrict__ part_ml, int B_, int T_, int Hq,
    int Hkv, int max_blocks, int num_blocks, float scale_log2, int R, int Rpad, int row_groups, int group_rows,
    int n_chunks_max, int cp, int n_items, unsigned* __restrict__ work) {
  // work: item counter, then the redo list (count, items), the number of listed items and the list
  __shared__ __attribute__((aligned(1024))) unsigned char ring[4][2 * DmaGeom<D>::TILE];
  __shared__ AttnMeta meta;
  __shared__ int s_item;
  const unsigned n_live = work[2 + n_items];
  const unsigned* order = work + 3 + n_items;
  for (;;) {
    lds_barrier();                       // every wave is done with the previous item (ring, meta, s_item)
    if (threadIdx.x == 0) {
      const unsigned k = atomicAdd(work, 1u);
      s_item = k < n_live ? (int)order[k] : -1;
    }
    lds_barrier();
    const int item = __builtin_amdgcn_readfirstlane(s_item);   // uniform: its derived values stay scalar
    if (item < 0) break;
    attn_item_dma<D>(item, ring, meta, q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, parents, out,
                     lse, part_o, part_ml, B_, T_, Hq, Hkv, max_blocks, num_blocks, scale_log2, R, Rpad,
                     row_groups, group_rows, n_chunks_max, cp, work + 1);
  }
}

// The work list of the persistent kernel: one block computes every item's tile count from ctx_len and
// counting-sorts the items by it, most tiles first (greedy list scheduling then ends the blocks close
// together). Items past a trajectory's chunk count are left out; a trajectory with an invalid ctx_len keeps
// its first item, which writes its NaN rows. Items of equal count keep no particular order (no result
// depends on it). Also zeroes the item counter and the redo count. work: [0] item counter, [1] redo count,
// [2, 2 + n_items) redo items, [2 + n_items] listed items, [3 + n_items, ...) the list.
constexpr int ATT_ORDER_BUCKETS = 64;
__global__ __launch_bounds__(1024) void k_attn_order(const int32_t* __restrict__ ctx_len, unsigned* __restrict__ work,
                                                     int B_, int T_, int Hkv, int row_groups, int max_blocks, int cp,
                                                     int n_items) {
  __shared__ unsigned cnt[ATT_ORDER_BUCKETS];
  const int tid = threadIdx.x;
  if (tid < ATT_ORDER_BUCKETS) cnt[tid] = 0u;
  if (tid < 2) work[tid] = 0u;
  __syncthreads();
  // bucket of an item: ATT_ORDER_BUCKETS - 1 - min(tiles, ATT_ORDER_BUCKETS - 1), or -1 when it has no work
  auto bucket = [&](int item) -> int {
    const int bg = item / row_groups;
    const int b = (bg / Hkv) % B_, c = bg / (Hkv * B_);
    const int Lraw = ctx_len[b];
    if (Lraw < 0 || Lraw > max_blocks * ATT_BS) return c == 0 ? ATT_ORDER_BUCKETS - 1 : -1;
    const int pages = (Lraw + ATT_BS - 1) / ATT_BS;
    const int n_chunks = max(1, (pages + cp - 1) / cp);
    if (c >= n_chunks) return -1;
    const int page0 = c * cp, page1 = min(pages, page0 + cp);
    const int keys = min(Lraw, page1 * ATT_BS) - page0 * ATT_BS;
    const int tiles = (keys + ATT_KT - 1) / ATT_KT + (c == n_chunks - 1 ? (T_ + ATT_KT - 1) / ATT_KT : 0);
    return ATT_ORDER_BUCKETS - 1 - min(tiles, ATT_ORDER_BUCKETS - 1);
  };
  for (int k = tid; k < n_items; k += blockDim.x) {
    const int bk = bucket(k);
    if (bk >= 0) atomicAdd(&cnt[bk], 1u);
  }
  __syncthreads();
  if (tid == 0) {
    unsigned run = 0;
    for (int i = 0; i < ATT_ORDER_BUCKETS; ++i) {
      const unsigned c = cnt[i];
      cnt[i] = run;
      run += c;
    }
    work[2 + n_items] = run;
  }
  __syncthreads();
  unsigned* order = work + 3 + n_items;
  for (int k = tid; k < n_items; k += blockDim.x) {
    const int bk = bucket(k);
    if (bk >= 0) order[atomicAdd(&cnt[bk], 1u)] = (unsigned)k;
  }
}

// Merge the chunk partials of every (trajectory, KV head) that was split.
template <int D>
__global__ __launch_bounds__(256) void k_attn_combine(const int32_t* __restrict__ ctx_len,
                                                      const float* __restrict__ part_o,
                                                      const float* __restrict__ part_ml, float* __restrict__ out,
                                                      float* __restrict__ lse, int T_, int Hq, int Hkv,
                                                      int max_blocks, int R, int Rpad, int n_chunks_max, int cp) {
  constexpr int TPR = D / 4;                 // threads per row (4 floats each)
  constexpr int RPB = 256 / TPR;             // rows per block
  const int g = blockIdx.y, b = blockIdx.z;
  const int Lraw = ctx_len[b];
  const bool ctx_ok = Lraw >= 0 && Lraw <= max_blocks * ATT_BS;
  const int pages = ctx_ok ? (Lraw + ATT_BS - 1) / ATT_BS : 0;
  const int n_chunks = ctx_ok ? max(1, (pages + cp - 1) / cp) : 1;
  if (n_chunks <= 1) return;
  const int r = blockIdx.x * RPB + threadIdx.x / TPR;
  const int d4 = (threadIdx.x % TPR) * 4;
  if (r >= R) return;
  const size_t base = ((size_t)b * Hkv + g) * n_chunks_max * Rpad + r;
  // chunks in groups of four: every load of a group is in flight at once, then the group is merged into
  // the running (M, W, acc) (one group, i.e. up to four chunks, is the plain max-then-sum)
  constexpr int CGRP = 4;
  float M = -INFINITY, W = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  bool nan = false;
  for (int c0 = 0; c0 < n_chunks; c0 += CGRP) {
    float2 ml[CGRP];
    f32x4 po[CGRP];
#pragma unroll
    for (int k = 0; k < CGRP; ++k) {
      const size_t pr = base + (size_t)(c0 + k) * Rpad;
      if (c0 + k < n_chunks) {
        ml[k] = *(const float2*)(part_ml + pr * 2);
        po[k] = *(const f32x4*)(part_o + pr * D + d4);
      } else {
        ml[k] = make_float2(-INFINITY, 0.f);
        po[k] = (f32x4){0.f, 0.f, 0.f, 0.f};
      }
    }
    float Mn = M;
#pragma unroll
    for (int k = 0; k < CGRP; ++k) {
      nan |= isnan(ml[k].x) || isnan(ml[k].y);
      Mn = fmaxf(Mn, ml[k].x);
    }
    const float Mu = (Mn == -INFINITY) ? 0.f : Mn;
    const float sc = exp2f(M - Mu);           // 0 while nothing is merged yet (M = -inf)
    W *= sc;
    acc *= sc;
#pragma unroll
    for (int k = 0; k < CGRP; ++k) {
      const float w = ml[k].y * exp2f(ml[k].x - Mu);
      W += w;
      acc += w * po[k];
    }
    M = Mn;
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
  // bf16: more than 224 rows split evenly into groups of at most 224, so every work item keeps a wave
  // free of query rows to issue its DMA (fp32: groups of 256)
  p.group_rows = ATT_ROWS;
  if (d.dtype == SR_BF16 && p.R > ATT_ROWS - 32) {
    const int ng = (p.R + (ATT_ROWS - 32) - 1) / (ATT_ROWS - 32);
    p.group_rows = ((p.R + ng - 1) / ng + 31) / 32 * 32;
  }
  p.row_groups = (p.R + p.group_rows - 1) / p.group_rows;
  // Few (trajectory, KV head, row group) triples leave most CUs idle unless each prefix is split finer;
  // with many, finer chunks only add partial results and per-chunk set-up. Chunks stay whole 64-key tiles.
  const long long triples = (long long)d.B * d.Hkv * p.row_groups;
  const int cp = triples < 64 ? 32 : triples < 512 ? 128 : ATT_CHUNK_PAGES;
  p.chunk_pages = cp;
  p.n_chunks = std::max(1, (d.max_blocks + cp - 1) / cp);
  const size_t rows = (size_t)d.B * d.Hkv * p.n_chunks * p.Rpad;
  p.part_o_bytes = p.n_chunks > 1 ? rows * d.D * sizeof(float) : 0;
  p.part_ml_bytes = p.n_chunks > 1 ? rows * 2 * sizeof(float) : 0;
  // bf16: the persistent kernel's item counter, the count and items of the fp32-V redo list, the number of
  // listed items and the list (k_attn_order)
  p.n_items = (long long)d.B * d.Hkv * p.row_groups * p.n_chunks;
  p.work_bytes = d.dtype == SR_BF16 ? (size_t)(3 + 2 * p.n_items) * sizeof(unsigned) : 0;
  return p;
}

// compute units of the current device (cached per device)
static int cu_count() {
  static int cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

template <typename T, int D>
static sr_status launch_attn_t(const sr_attn_desc& d, const AttnPlan& p, const void* q, const void* kc,
                               const void* vc, const int32_t* bt, const int32_t* cl, const void* kt,
                               const void* vt, const int32_t* par, float* out, float* lse, float* po, float* pml,
                               unsigned* work, hipStream_t s) {
  const float scale_log2 = d.scale * kLog2e;
  // chunk index slowest: consecutive blocks (which the dispatcher deals round-robin to the XCDs) are
  // different (trajectory, KV head) pairs of one chunk index, so every XCD receives an equal share of the
  // first chunks (always present) and of the later ones (present only for long contexts); the long
  // first chunks also start first
  dim3 grid(d.B * d.Hkv * p.row_groups, p.n_chunks);
  if constexpr (sizeof(T) == 2) {
    const long long n_items = (long long)grid.x * grid.y;
    if (n_items > INT32_MAX / 2) return SR_ERR_INVALID;
    SR_LAUNCH("sr_attn_order", k_attn_order, dim3(1), dim3(1024), 0, s, cl, work, d.B, d.T, d.Hkv, p.row_groups,
              d.max_blocks, p.chunk_pages, (int)n_items);
    const int nb = (int)std::min<long long>(n_items, cu_count());
    SR_LAUNCH("sr_tree_attn", (k_tree_attn_dma<D>), dim3(nb), dim3(ATT_NW * 64), 0, s, (const T*)q, (const T*)kc,
              (const T*)vc, bt, cl, (const T*)kt, (const T*)vt, par, out, lse, po, pml, d.B, d.T, d.Hq, d.Hkv,
              d.max_blocks, d.num_blocks, scale_log2, p.R, p.Rpad, p.row_groups, p.group_rows, p.n_chunks,
              p.chunk_pages, (int)n_items, work);
    // items holding a V value outside fp16's exact range, recomputed with fp32 V (blocks exit at once when
    // the list is empty)
    SR_LAUNCH("sr_attn_redo", (k_tree_attn_redo<D>), dim3(nb), dim3(ATT_NW * 64), 0, s, (const T*)q, (const T*)kc,
              (const T*)vc, bt, cl, (const T*)kt, (const T*)vt, par, out, lse, po, pml, d.B, d.T, d.Hq, d.Hkv,
              d.max_blocks, d.num_blocks, scale_log2, p.R, p.Rpad, p.row_groups, p.group_rows, p.n_chunks,
              p.chunk_pages, (int)n_items, (const unsigned*)(work + 1));
  } else {
    SR_LAUNCH("sr_tree_attn", (k_tree_attn<D>), grid, dim3(ATT_NW * 64), 0, s, (const T*)q, (const T*)kc,
              (const T*)vc, bt, cl, (const T*)kt, (const T*)vt, par, out, lse, po, pml, d.T, d.Hq, d.Hkv,
              d.max_blocks, d.num_blocks, scale_log2, p.R, p.Rpad, p.row_groups, p.group_rows, p.n_chunks,
              p.chunk_pages);
  }
  if (p.n_chunks > 1) {
    constexpr int RPB = 256 / (D / 4);
    dim3 cgrid((p.R + RPB - 1) / RPB, d.Hkv, d.B);
    SR_LAUNCH("sr_attn_combine", (k_attn_combine<D>), cgrid, dim3(256), 0, s, cl, po, pml, out, lse, d.T, d.Hq,
              d.Hkv, d.max_blocks, p.R, p.Rpad, p.n_chunks, p.chunk_pages);
  }
  return SR_OK;
}

sr_status launch_tree_attn(const sr_attn_desc& d, const AttnPlan& p, const void* q, const void* k_cache,
                           const void* v_cache, const int32_t* block_table, const int32_t* ctx_len,
                           const void* k_tree, const void* v_tree, const int32_t* parents, float* out,
                           float* lse, float* part_o, float* part_ml, unsigned* work, hipStream_t s) {
#define SR_ATTN_CASE(TT, DD)                                                                                  \
  return launch_attn_t<TT, DD>(d, p, q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, parents, out, \
                               lse, part_o, part_ml, work, s)
  if (d.dtype == SR_BF16) {
    if (d.D == 128) SR_ATTN_CASE(bf16_t, 128);
    SR_ATTN_CASE(bf16_t, 64);
  }
  if (d.D == 128) SR_ATTN_CASE(float, 128);
  SR_ATTN_CASE(float, 64);
#undef SR_ATTN_CASE
}

}  // namespace sr
