// C ABI of the speculative verification step: argument checks, workspace layout,
// error reporting and the kernel timing hook. Compute lives in k_*.hip.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <cmath>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"
#include "kernels.hpp"

namespace sr {

static thread_local std::string g_err;

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
}

sr_status hip_fail(hipError_t e, const char* what) {
  set_error("%s: %s", what, hipGetErrorString(e));
  return SR_ERR_HIP;
}

// ---------------------------------------------------------------- timing hook
struct Prof {
  bool on = false;
  std::string pat;
  std::vector<hipEvent_t> start, stop;
  int used = 0;
  static constexpr int kMax = 4096;
};
static Prof g_prof;

// A timed launch gets a start and a stop event that the kernel's dispatch records itself
// (hipExtLaunchKernelGGL): the timing adds no commands to the stream between kernels.
LaunchGuard::LaunchGuard(const char* n, hipStream_t s)
    : name(n), stream(s), slot(-1), ev_start(nullptr), ev_stop(nullptr) {
  if (g_prof.on && strstr(n, g_prof.pat.c_str()) != nullptr && g_prof.used < Prof::kMax) {
    if ((int)g_prof.start.size() <= g_prof.used) {
      hipEvent_t a, b;
      if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) return;
      g_prof.start.push_back(a);
      g_prof.stop.push_back(b);
    }
    slot = g_prof.used;
    ev_start = g_prof.start[slot];
    ev_stop = g_prof.stop[slot];
  }
}

sr_status LaunchGuard::done() {
  hipError_t e = hipGetLastError();
  if (slot >= 0) ++g_prof.used;
  if (e != hipSuccess) {
    set_error("launch of %s failed: %s", name, hipGetErrorString(e));
    return SR_ERR_HIP;
  }
  return SR_OK;
}

// ---------------------------------------------------------------- helpers
static size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }
static size_t esize(sr_dtype t) { return t == SR_BF16 ? 2 : 4; }
static bool dtype_ok(sr_dtype t) { return t == SR_F32 || t == SR_BF16; }

#define SR_CHECK(cond, ...)        \
  do {                             \
    if (!(cond)) {                 \
      ::sr::set_error(__VA_ARGS__); \
      return SR_ERR_INVALID;       \
    }                              \
  } while (0)

struct HeadsLayout {
  size_t x, n, z, logits, top_id, top_val, gmax, total;
};
static HeadsLayout heads_layout(const sr_heads_desc& d, bool need_z, bool need_logits) {
  HeadsLayout L;
  size_t off = 0;
  const size_t B = d.B, H = d.H, dd = d.d, V = d.V, M = d.max_children;
  L.x = off; off = align_up(off + B * dd * 4);
  L.n = off; off = align_up(off + B * dd * esize(d.dtype));
  L.z = off; if (need_z) off = align_up(off + B * H * dd * esize(d.dtype));
  L.logits = off; if (need_logits) off = align_up(off + B * H * V * 4);
  L.top_id = off; off = align_up(off + B * H * M * 4);
  L.top_val = off; off = align_up(off + B * H * M * 4);
  L.gmax = off; off = align_up(off + group_max_count(d) * 4);
  L.total = off;
  return L;
}

static sr_status check_heads_desc(const sr_heads_desc* d, bool tree_only) {
  SR_CHECK(d != nullptr, "null descriptor");
  SR_CHECK(d->B >= 1, "B must be >= 1 (got %d)", d->B);
  SR_CHECK(d->H >= 1, "H must be >= 1 (got %d)", d->H);
  // logits rows are written four columns per store: whole quads per row (the acceptance walk and the
  // feedback take multiples of 8 of the same vocabulary)
  SR_CHECK(d->V >= 8 && d->V % 8 == 0, "V must be a positive multiple of 8 (got %d)", d->V);
  SR_CHECK(d->T >= 1 && d->T <= SR_MAX_TREE, "T must be in [1, %d] (got %d)", SR_MAX_TREE, d->T);
  SR_CHECK(d->max_children >= 0 && d->max_children <= d->T - 1, "max_children must be in [0, T-1] (got %d)",
           d->max_children);
  SR_CHECK(d->T == 1 || d->max_children >= 1, "a tree with T > 1 needs max_children >= 1");
  SR_CHECK(d->max_children <= d->V, "max_children (%d) exceeds V (%d)", d->max_children, d->V);
  if (!tree_only) {
    SR_CHECK(d->d >= 64 && d->d % 64 == 0, "d must be a positive multiple of 64 (got %d)", d->d);
    SR_CHECK(dtype_ok(d->dtype), "unknown dtype %d", (int)d->dtype);
    SR_CHECK(std::isfinite(d->clip_norm) && d->clip_norm > 0.f, "clip_norm must be finite and > 0");
    SR_CHECK(std::isfinite(d->ln_eps) && d->ln_eps >= 0.f, "ln_eps must be finite and >= 0");
    SR_CHECK((size_t)d->H * d->d <= (size_t)INT32_MAX, "H*d too large");
  }
  SR_CHECK((size_t)d->B * d->H <= (size_t)INT32_MAX, "B*H too large");
  return SR_OK;
}

static sr_status check_ws(const void* ws, size_t have, size_t need) {
  if (need == 0) return SR_OK;
  if (ws == nullptr || have < need) {
    set_error("workspace of %zu bytes required, %zu given%s", need, have, ws ? "" : " (null)");
    return SR_ERR_WORKSPACE;
  }
  if (((uintptr_t)ws & 255u) != 0) {
    set_error("workspace must be 256-byte aligned");
    return SR_ERR_INVALID;
  }
  return SR_OK;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// ---------------------------------------------------------------- scratch of the allocation-free attention call
// One array per GPU, created with the library's code object on that GPU and held until the process ends. In
// host code `scratch` names a host-side stand-in, never the device memory: its device address is taken once
// per device with hipGetSymbolAddress and only that address is handed to kernels.
static __device__ __align__(256) unsigned char scratch[SR_ATTN_NOALLOC_MAX_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices];

// device address of the current device's scratch array (looked up at the first call on that device)
static sr_status scratch_base(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) {
    set_error("device %d: at most %d devices are supported", dev, kMaxDevices);
    return SR_ERR_UNSUPPORTED;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (p == nullptr || ((uintptr_t)p & 255u) != 0) {
      set_error("scratch array of device %d has no usable device address", dev);
      return SR_ERR_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SR_OK;
}

}  // namespace sr

using namespace sr;

extern "C" {

const char* sr_last_error(void) { return g_err.c_str(); }

const char* sr_version(void) { return "specroll-mi355x 0.1 (gfx950)"; }

const char* sr_kernel_names(void) {
  return "sr_clip_ln;sr_head_gemm;sr_vocab_gemm;sr_group_max;sr_topm;sr_topm_full;sr_tree_build;sr_attn_order;"
         "sr_tree_attn;sr_attn_redo;sr_attn_combine;sr_tree_accept;sr_commit_path;sr_reflex_feedback;"
         "sr_reflex_correct";
}

// ------------------------------------------------------------------ proposal
size_t sr_heads_propose_workspace(const sr_heads_desc* d) {
  if (check_heads_desc(d, false) != SR_OK) return 0;
  return heads_layout(*d, true, true).total;
}

sr_status sr_heads_propose(const sr_heads_desc* d, const void* hidden, const float* corr, const uint8_t* corr_active,
                           const void* A, const void* bias, const void* W, const int32_t* parents,
                           const int32_t* root_token, const float* u_tree, float* logits, void* z, int32_t* tokens,
                           float* child_logit, void* workspace, size_t workspace_bytes, void* stream) {
  sr_status st = check_heads_desc(d, false);
  if (st != SR_OK) return st;
  SR_CHECK(hidden && A && bias && W && parents && root_token && u_tree && tokens && child_logit,
           "a required pointer is null");
  SR_CHECK(aligned16(hidden) && aligned16(A) && aligned16(W) && aligned16(bias), "hidden/A/bias/W must be 16-byte aligned");
  SR_CHECK(z == nullptr || aligned16(z), "z must be 16-byte aligned");
  SR_CHECK(logits == nullptr || aligned16(logits), "logits must be 16-byte aligned");
  const HeadsLayout L = heads_layout(*d, z == nullptr, logits == nullptr);
  st = check_ws(workspace, workspace_bytes, L.total);
  if (st != SR_OK) return st;
  char* ws = (char*)workspace;
  float* x = (float*)(ws + L.x);
  void* n = ws + L.n;
  void* zz = z ? z : (void*)(ws + L.z);
  float* lg = logits ? logits : (float*)(ws + L.logits);
  hipStream_t s = (hipStream_t)stream;
  float* gmax = (float*)(ws + L.gmax);
  st = launch_heads(*d, hidden, corr, corr_active, A, bias, W, x, n, zz, lg, gmax, s);
  if (st != SR_OK) return st;
  return launch_tree_build(*d, lg, gmax, parents, root_token, u_tree, tokens, child_logit,
                           (int32_t*)(ws + L.top_id), (float*)(ws + L.top_val), s);
}

sr_status sr_heads_propose_reflex(const sr_heads_desc* d, const sr_reflex_gate_desc* g, const void* hidden,
                                  const float* corr, const uint8_t* corr_active, const void* A, const void* bias,
                                  const void* W, const int32_t* parents, const int32_t* root_token,
                                  const float* u_tree, const float* memory, const float* align, const float* P,
                                  float* logits, void* z, int32_t* tokens, float* child_logit, float* sketch_out,
                                  float* alpha_out, void* workspace, size_t workspace_bytes, void* stream) {
  sr_status st = check_heads_desc(d, false);
  if (st != SR_OK) return st;
  SR_CHECK(g != nullptr, "null gate descriptor");
  SR_CHECK(d->H <= 8, "H must be <= 8 with the gated correction (got %d)", d->H);
  SR_CHECK(d->d <= 8192, "d must be <= 8192 with the gated correction (got %d)", d->d);
  SR_CHECK(g->rank >= 0 && g->rank <= 64, "rank must be in [0, 64] (got %d)", g->rank);
  SR_CHECK(std::isfinite(g->z_delta) && g->z_delta >= 0.f, "z_delta must be finite and >= 0");
  SR_CHECK(std::isfinite(g->eps) && g->eps > 0.f, "eps must be finite and > 0");
  SR_CHECK(std::isfinite(g->m_floor) && g->m_floor >= 0.f, "m_floor must be finite and >= 0");
  for (int h = 0; h < d->H; ++h) {
    SR_CHECK(std::isfinite(g->alpha_min[h]) && std::isfinite(g->alpha_max[h]) && g->alpha_min[h] >= 0.f &&
                 g->alpha_min[h] <= g->alpha_max[h],
             "need 0 <= alpha_min <= alpha_max (head %d)", h);
    SR_CHECK(g->n_fb_min[h] >= 0 && g->n_align_min[h] >= 0, "minimum counts must be >= 0 (head %d)", h);
  }
  SR_CHECK(hidden && A && bias && W && parents && root_token && u_tree && tokens && child_logit && memory && align,
           "a required pointer is null");
  SR_CHECK(g->rank == 0 || P != nullptr, "P is null with rank > 0");
  SR_CHECK(P == nullptr || aligned16(P), "P must be 16-byte aligned");
  SR_CHECK(aligned16(hidden) && aligned16(A) && aligned16(W) && aligned16(bias), "hidden/A/bias/W must be 16-byte aligned");
  SR_CHECK(z == nullptr || aligned16(z), "z must be 16-byte aligned");
  SR_CHECK(logits == nullptr || aligned16(logits), "logits must be 16-byte aligned");
  const HeadsLayout L = heads_layout(*d, z == nullptr, logits == nullptr);
  st = check_ws(workspace, workspace_bytes, L.total);
  if (st != SR_OK) return st;
  char* ws = (char*)workspace;
  void* zz = z ? z : (void*)(ws + L.z);
  float* lg = logits ? logits : (float*)(ws + L.logits);
  float* gmax = (float*)(ws + L.gmax);
  hipStream_t s = (hipStream_t)stream;
  st = launch_heads_z(*d, hidden, corr, corr_active, A, bias, (float*)(ws + L.x), ws + L.n, zz, s);
  if (st != SR_OK) return st;
  st = launch_reflex_correct(*d, *g, zz, memory, align, P, sketch_out, alpha_out, s);
  if (st != SR_OK) return st;
  st = launch_vocab(*d, zz, W, lg, gmax, s);
  if (st != SR_OK) return st;
  return launch_tree_build(*d, lg, gmax, parents, root_token, u_tree, tokens, child_logit,
                           (int32_t*)(ws + L.top_id), (float*)(ws + L.top_val), s);
}

static size_t tree_ws_parts(const sr_heads_desc& d, size_t* top, size_t* gm) {
  *top = align_up((size_t)d.B * d.H * d.max_children * 4);
  *gm = align_up(group_max_count(d) * 4);
  return 2 * *top + *gm;
}

size_t sr_tree_build_workspace(const sr_heads_desc* d) {
  if (check_heads_desc(d, true) != SR_OK) return 0;
  size_t a, b;
  return tree_ws_parts(*d, &a, &b);
}

sr_status sr_tree_build(const sr_heads_desc* d, const float* logits, const int32_t* parents,
                        const int32_t* root_token, const float* u_tree, int32_t* tokens, float* child_logit,
                        void* workspace, size_t workspace_bytes, void* stream) {
  sr_status st = check_heads_desc(d, true);
  if (st != SR_OK) return st;
  SR_CHECK(logits && parents && root_token && u_tree && tokens && child_logit, "a required pointer is null");
  size_t top, gm;
  st = check_ws(workspace, workspace_bytes, tree_ws_parts(*d, &top, &gm));
  if (st != SR_OK) return st;
  char* ws = (char*)workspace;
  float* gmax = (float*)(ws + 2 * top);
  hipStream_t s = (hipStream_t)stream;
  st = launch_group_max(*d, logits, gmax, s);
  if (st != SR_OK) return st;
  return launch_tree_build(*d, logits, gmax, parents, root_token, u_tree, tokens, child_logit, (int32_t*)ws,
                           (float*)(ws + top), s);
}

// ------------------------------------------------------------------ attention
static sr_status check_attn_desc(const sr_attn_desc* d) {
  SR_CHECK(d != nullptr, "null descriptor");
  SR_CHECK(d->B >= 1 && d->B <= 65535, "B must be in [1, 65535] (got %d)", d->B);
  SR_CHECK(d->T >= 1 && d->T <= SR_MAX_TREE, "T must be in [1, %d] (got %d)", SR_MAX_TREE, d->T);
  SR_CHECK(d->Hkv <= 65535, "Hkv too large");
  SR_CHECK(d->Hq >= 1 && d->Hkv >= 1 && d->Hq % d->Hkv == 0, "need Hq >= 1, Hkv >= 1 and Hq %% Hkv == 0");
  SR_CHECK(d->D == 64 || d->D == 128, "D must be 64 or 128 (got %d)", d->D);
  SR_CHECK(d->block_size == 16, "block_size must be 16 (got %d)", d->block_size);
  SR_CHECK(d->max_blocks >= 1 && d->num_blocks >= 1, "max_blocks and num_blocks must be >= 1");
  SR_CHECK((size_t)d->max_blocks * 16 <= (size_t)INT32_MAX / 2, "max_blocks too large");
  SR_CHECK(dtype_ok(d->dtype), "unknown dtype %d", (int)d->dtype);
  SR_CHECK(std::isfinite(d->scale) && d->scale > 0.f, "scale must be finite and > 0");
  return SR_OK;
}

size_t sr_tree_verify_attn_workspace(const sr_attn_desc* d) {
  if (check_attn_desc(d) != SR_OK) return 0;
  const AttnPlan p = attn_plan(*d);
  return align_up(p.part_o_bytes) + align_up(p.part_ml_bytes) + align_up(p.work_bytes);
}

static sr_status check_attn_args(const sr_attn_desc* d, const void* q, const void* k_cache, const void* v_cache,
                                 const int32_t* block_table, const int32_t* ctx_len, const void* k_tree,
                                 const void* v_tree, const int32_t* parents, const float* out) {
  sr_status st = check_attn_desc(d);
  if (st != SR_OK) return st;
  SR_CHECK(q && k_cache && v_cache && block_table && ctx_len && k_tree && v_tree && parents && out,
           "a required pointer is null");
  SR_CHECK(aligned16(q) && aligned16(k_cache) && aligned16(v_cache) && aligned16(k_tree) && aligned16(v_tree) &&
               aligned16(out),
           "q, caches, tree K/V and out must be 16-byte aligned");
  return SR_OK;
}

static sr_status run_attn(const sr_attn_desc* d, const AttnPlan& p, const void* q, const void* k_cache,
                          const void* v_cache, const int32_t* block_table, const int32_t* ctx_len, const void* k_tree,
                          const void* v_tree, const int32_t* parents, float* out, float* lse, char* ws,
                          void* stream) {
  float* po = p.part_o_bytes ? (float*)ws : nullptr;
  float* pml = p.part_ml_bytes ? (float*)(ws + align_up(p.part_o_bytes)) : nullptr;
  unsigned* work = p.work_bytes ? (unsigned*)(ws + align_up(p.part_o_bytes) + align_up(p.part_ml_bytes)) : nullptr;
  return launch_tree_attn(*d, p, q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, parents, out, lse, po,
                          pml, work, (hipStream_t)stream);
}

sr_status sr_tree_verify_attn(const sr_attn_desc* d, const void* q, const void* k_cache, const void* v_cache,
                              const int32_t* block_table, const int32_t* ctx_len, const void* k_tree,
                              const void* v_tree, const int32_t* parents, float* out, float* lse, void* workspace,
                              size_t workspace_bytes, void* stream) {
  sr_status st = check_attn_args(d, q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, parents, out);
  if (st != SR_OK) return st;
  const AttnPlan p = attn_plan(*d);
  const size_t need = align_up(p.part_o_bytes) + align_up(p.part_ml_bytes) + align_up(p.work_bytes);
  st = check_ws(workspace, workspace_bytes, need);
  if (st != SR_OK) return st;
  return run_attn(d, p, q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, parents, out, lse,
                  (char*)workspace, stream);
}

sr_status sr_tree_verify_attn_noalloc(const sr_attn_desc* d, const void* q, const void* k_cache, const void* v_cache,
                                      const int32_t* block_table, const int32_t* ctx_len, const void* k_tree,
                                      const void* v_tree, const int32_t* parents, float* out, float* lse,
                                      void* stream) {
  sr_status st = check_attn_args(d, q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, parents, out);
  if (st != SR_OK) return st;
  const AttnPlan p = attn_plan(*d);
  const size_t need = align_up(p.part_o_bytes) + align_up(p.part_ml_bytes) + align_up(p.work_bytes);
  if (need > (size_t)SR_ATTN_NOALLOC_MAX_BYTES) {
    set_error("request needs %zu bytes of scratch; the allocation-free call holds %zu "
              "(use sr_tree_verify_attn with a workspace)", need, (size_t)SR_ATTN_NOALLOC_MAX_BYTES);
    return SR_ERR_UNSUPPORTED;
  }
  void* base = nullptr;
  st = scratch_base(&base);
  if (st != SR_OK) return st;
  return run_attn(d, p, q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, parents, out, lse, (char*)base,
                  stream);
}

// ------------------------------------------------------------------ acceptance
static sr_status check_accept_desc(const sr_accept_desc* d) {
  SR_CHECK(d != nullptr, "null descriptor");
  SR_CHECK(d->B >= 1, "B must be >= 1 (got %d)", d->B);
  SR_CHECK(d->T >= 1 && d->T <= SR_MAX_TREE, "T must be in [1, %d] (got %d)", SR_MAX_TREE, d->T);
  SR_CHECK(d->V >= 8 && d->V <= 262144 && d->V % 8 == 0, "V must be a multiple of 8 in [8, 262144] (got %d)", d->V);
  SR_CHECK(d->max_depth >= 0 && d->max_depth <= SR_MAX_TREE, "max_depth must be in [0, %d]", SR_MAX_TREE);
  SR_CHECK(dtype_ok(d->logit_dtype), "unknown logit dtype %d", (int)d->logit_dtype);
  SR_CHECK(std::isfinite(d->temperature) && d->temperature > 0.f, "temperature must be finite and > 0");
  SR_CHECK(d->top_p > 0.f && d->top_p <= 1.f, "top_p must be in (0, 1] (got %g)", (double)d->top_p);
  return SR_OK;
}

size_t sr_tree_accept_workspace(const sr_accept_desc* d) {
  (void)d;
  return 0;
}

sr_status sr_tree_accept(const sr_accept_desc* d, const void* target_logits, const float* child_logit,
                         const int32_t* tokens, const int32_t* parents, const float* u_acc, const float* u_fin,
                         int32_t* acc_nodes, int32_t* out_tokens, int32_t* out_len, uint8_t* final_kind,
                         float* min_margin, void* workspace, size_t workspace_bytes, void* stream) {
  (void)workspace;
  (void)workspace_bytes;
  sr_status st = check_accept_desc(d);
  if (st != SR_OK) return st;
  SR_CHECK(target_logits && child_logit && tokens && parents && u_acc && u_fin && out_tokens && out_len && final_kind,
           "a required pointer is null");
  SR_CHECK(d->max_depth == 0 || acc_nodes != nullptr, "acc_nodes is null");
  SR_CHECK(aligned16(target_logits), "target_logits must be 16-byte aligned");
  return launch_tree_accept(*d, target_logits, child_logit, tokens, parents, u_acc, u_fin, acc_nodes, out_tokens,
                            out_len, final_kind, min_margin, (hipStream_t)stream);
}

// ------------------------------------------------------------------ engine glue
sr_status sr_tree_budget(const sr_budget_desc* d, int32_t live, int32_t* n_t, int32_t* horizon_count,
                         int32_t* parents, int32_t parents_cap, int32_t* n_nodes) {
  SR_CHECK(d != nullptr, "null descriptor");
  SR_CHECK(n_t && parents && n_nodes, "a required pointer is null");
  SR_CHECK(d->c_peak >= 1, "c_peak must be >= 1 (got %d)", d->c_peak);
  SR_CHECK(d->n_min >= 1 && d->n_min <= d->n_max && d->n_max <= SR_MAX_TREE,
           "need 1 <= n_min <= n_max <= %d (got %d, %d)", SR_MAX_TREE, d->n_min, d->n_max);
  SR_CHECK(d->n_alloc >= 0 && d->n_alloc <= SR_MAX_TREE, "n_alloc must be in [0, %d]", SR_MAX_TREE);
  SR_CHECK(d->n_alloc == 0 || d->alloc != nullptr, "alloc is null");
  SR_CHECK(live >= 1, "live must be >= 1 (got %d)", live);
  for (int h = 0; h < d->n_alloc; ++h) SR_CHECK(d->alloc[h] >= 0, "alloc[%d] is negative", h);
  // Eq. (verification-budget): the per-response share of the capacity, clipped
  const int32_t share = d->c_peak / live;
  const int32_t budget = share < d->n_min ? d->n_min : (share > d->n_max ? d->n_max : share);
  // Eq. (tree-budget): the anchor plus the horizons, filled shallowest first
  int32_t cnt[SR_MAX_TREE];
  int32_t used = 1, levels = 0;
  for (int h = 0; h < d->n_alloc; ++h) {
    const int32_t give = d->alloc[h] < budget - used ? d->alloc[h] : budget - used;
    if (give <= 0) break;
    cnt[levels++] = give;
    used += give;
  }
  SR_CHECK(used <= parents_cap, "parents_cap %d cannot hold the %d-node tree", parents_cap, used);
  parents[0] = -1;
  int32_t prev_first = 0, prev_n = 1, next = 1;
  for (int h = 0; h < levels; ++h) {
    for (int32_t k = 0; k < cnt[h]; ++k) parents[next + k] = prev_first + (k * prev_n) / cnt[h];
    prev_first = next;
    prev_n = cnt[h];
    next += cnt[h];
  }
  if (horizon_count)
    for (int h = 0; h < d->n_alloc; ++h) horizon_count[h] = h < levels ? cnt[h] : 0;
  *n_t = budget;
  *n_nodes = used;
  return SR_OK;
}

sr_status sr_commit_path(const sr_commit_desc* d, const int32_t* acc_nodes, const int32_t* out_len,
                         const int32_t* parents, const void* k_tree, const void* v_tree, const int32_t* block_table,
                         const int32_t* ctx_len, void* k_cache, void* v_cache, int32_t* new_ctx_len, void* stream) {
  SR_CHECK(d != nullptr, "null descriptor");
  SR_CHECK(d->n_layers >= 1 && d->n_layers <= 65535, "n_layers must be in [1, 65535] (got %d)", d->n_layers);
  SR_CHECK(d->B >= 1, "B must be >= 1 (got %d)", d->B);
  SR_CHECK(d->T >= 1 && d->T <= SR_MAX_TREE, "T must be in [1, %d] (got %d)", SR_MAX_TREE, d->T);
  SR_CHECK(d->Hkv >= 1 && d->D >= 1, "Hkv and D must be >= 1");
  SR_CHECK(dtype_ok(d->dtype), "unknown dtype %d", (int)d->dtype);
  SR_CHECK(((size_t)d->D * esize(d->dtype)) % 16 == 0, "D * element size must be a multiple of 16 bytes (D = %d)",
           d->D);
  SR_CHECK(d->block_size >= 1 && d->max_blocks >= 1 && d->num_blocks >= 1,
           "block_size, max_blocks and num_blocks must be >= 1");
  SR_CHECK((size_t)d->max_blocks * d->block_size <= (size_t)INT32_MAX / 2, "max_blocks * block_size too large");
  SR_CHECK(d->max_depth >= 0 && d->max_depth <= SR_MAX_TREE, "max_depth must be in [0, %d]", SR_MAX_TREE);
  SR_CHECK((size_t)2 * (d->max_depth + 1) * d->Hkv * d->D <= (size_t)INT32_MAX / 4, "Hkv * D too large");
  SR_CHECK(out_len && k_tree && v_tree && block_table && ctx_len && k_cache && v_cache && new_ctx_len,
           "a required pointer is null");
  SR_CHECK(d->max_depth == 0 || acc_nodes != nullptr, "acc_nodes is null");
  SR_CHECK(aligned16(k_tree) && aligned16(v_tree) && aligned16(k_cache) && aligned16(v_cache),
           "tree K/V and caches must be 16-byte aligned");
  SR_CHECK(new_ctx_len != ctx_len, "new_ctx_len must not overlap ctx_len");
  return launch_commit_path(*d, acc_nodes, out_len, parents, k_tree, v_tree, block_table, ctx_len, k_cache, v_cache,
                            new_ctx_len, (hipStream_t)stream);
}

// ------------------------------------------------------------------ Reflex feedback
sr_status sr_reflex_feedback(const sr_reflex_desc* d, const void* target_logits, const int32_t* p_row,
                             const float* head_logits, const int32_t* q_row, const int32_t* cand,
                             const int32_t* y_star, const int32_t* traj, const int32_t* horizon, const void* W,
                             float* memory, float* stats, float* e_out, const float* P, const float* rec_sketch,
                             float* align, void* stream) {
  SR_CHECK(d != nullptr, "null descriptor");
  SR_CHECK(d->R >= 1, "R must be >= 1 (got %d)", d->R);
  SR_CHECK(d->V >= 8 && d->V <= 262144 && d->V % 8 == 0, "V must be a multiple of 8 in [8, 262144] (got %d)", d->V);
  SR_CHECK(d->d >= 8 && d->d <= 8192 && d->d % 8 == 0, "d must be a multiple of 8 in [8, 8192] (got %d)", d->d);
  SR_CHECK(d->B >= 1 && d->H >= 1 && d->H <= 8, "need B >= 1 and 1 <= H <= 8");
  SR_CHECK(d->n_p_rows >= 1 && d->n_q_rows >= 1, "n_p_rows and n_q_rows must be >= 1");
  SR_CHECK(d->support >= 1 && d->support <= 64 && d->support <= d->V, "support must be in [1, min(64, V)] (got %d)",
           d->support);
  SR_CHECK(d->max_cand >= 1 && d->max_cand <= d->support, "max_cand must be in [1, support] (got %d)", d->max_cand);
  SR_CHECK(d->n_boundary >= 1, "n_boundary must be >= 1");
  SR_CHECK(dtype_ok(d->p_dtype) && dtype_ok(d->w_dtype), "unknown dtype");
  SR_CHECK(std::isfinite(d->temperature) && d->temperature > 0.f, "temperature must be finite and > 0");
  SR_CHECK(std::isfinite(d->eps) && d->eps > 0.f, "eps must be finite and > 0");
  SR_CHECK(std::isfinite(d->w_dist) && std::isfinite(d->w_cov) && d->w_dist >= 0.f && d->w_cov >= 0.f,
           "w_dist and w_cov must be finite and >= 0");
  SR_CHECK(std::isfinite(d->sev_tv) && std::isfinite(d->sev_out) && std::isfinite(d->w_min),
           "severity coefficients must be finite");
  for (int h = 0; h < d->H; ++h)
    SR_CHECK(d->rho[h] >= 0.f && d->rho[h] < 1.f, "rho[%d] must be in [0, 1)", h);
  SR_CHECK(d->rank >= 0 && d->rank <= 64, "rank must be in [0, 64] (got %d)", d->rank);
  SR_CHECK(d->rank == 0 || align == nullptr || (P != nullptr && rec_sketch != nullptr),
           "P and rec_sketch are required for alignment observations with rank > 0");
  SR_CHECK(P == nullptr || aligned16(P), "P must be 16-byte aligned");
  SR_CHECK(target_logits && p_row && head_logits && q_row && cand && y_star && traj && horizon && W && memory && stats,
           "a required pointer is null");
  SR_CHECK(aligned16(target_logits) && aligned16(head_logits) && aligned16(W),
           "target_logits, head_logits and W must be 16-byte aligned");
  return launch_reflex_feedback(*d, target_logits, p_row, head_logits, q_row, cand, y_star, traj, horizon, W, memory,
                                stats, e_out, P, rec_sketch, align, (hipStream_t)stream);
}

// ------------------------------------------------------------------ timing hook
sr_status sr_prof_begin(const char* kernel_substr) {
  SR_CHECK(kernel_substr != nullptr, "null kernel name");
  g_prof.on = true;
  g_prof.pat = kernel_substr;
  g_prof.used = 0;
  return SR_OK;
}

sr_status sr_prof_end(double* total_ms, int32_t* launches) {
  SR_CHECK(total_ms && launches, "null output");
  double tot = 0.0;
  for (int i = 0; i < g_prof.used; ++i) {
    hipError_t e = hipEventSynchronize(g_prof.stop[i]);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, g_prof.start[i], g_prof.stop[i]);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    tot += ms;
  }
  *total_ms = tot;
  *launches = g_prof.used;
  g_prof.on = false;
  g_prof.used = 0;
  return SR_OK;
}

}  // extern "C"
