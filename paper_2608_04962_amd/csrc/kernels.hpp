// Launchers implemented in the kernel translation units, called by the C ABI layer.
#pragma once

#include "common.hpp"

namespace sr {

// ---- proposal (k_heads.hip)
sr_status launch_heads(const sr_heads_desc& d, const void* hidden, const float* corr, const uint8_t* active,
                       const void* A, const void* bias, const void* W, float* x, void* n, void* z,
                       float* logits, float* gmax, hipStream_t s);
// the two halves of launch_heads: clip + LayerNorm + head GEMM (z), then the vocabulary GEMM (+ group maxima)
sr_status launch_heads_z(const sr_heads_desc& d, const void* hidden, const float* corr, const uint8_t* active,
                         const void* A, const void* bias, float* x, void* n, void* z, hipStream_t s);
sr_status launch_vocab(const sr_heads_desc& d, const void* z, const void* W, float* logits, float* gmax,
                       hipStream_t s);
// per-row maxima of the 64-column groups of fp32 logits [B*H, V]
size_t group_max_count(const sr_heads_desc& d);
sr_status launch_group_max(const sr_heads_desc& d, const float* logits, float* gmax, hipStream_t s);
// top-M supports + ordered child lists; gmax may be null (then a full selection per row runs)
sr_status launch_tree_build(const sr_heads_desc& d, const float* logits, const float* gmax,
                            const int32_t* parents, const int32_t* root_token, const float* u_tree,
                            int32_t* tokens, float* child_logit, int32_t* top_id, float* top_val, hipStream_t s);

// ---- attention (k_attn.hip)
struct AttnPlan {
  int R;            // query rows per (trajectory, KV head) = T * Hq / Hkv
  int Rpad;         // R rounded up to 32
  int row_groups;   // blocks along the rows
  int group_rows;   // query rows per row group (a multiple of 32, at most 256)
  int chunk_pages;  // prefix pages per work item
  int n_chunks;     // work items per (trajectory, KV head), worst case
  size_t part_o_bytes, part_ml_bytes;
  long long n_items;  // work items (trajectory, KV head, row group, chunk)
  size_t work_bytes;  // bf16: item counter, then the redo count and list (2 + n_items words)
};
AttnPlan attn_plan(const sr_attn_desc& d);
sr_status launch_tree_attn(const sr_attn_desc& d, const AttnPlan& p, const void* q, const void* k_cache,
                           const void* v_cache, const int32_t* block_table, const int32_t* ctx_len,
                           const void* k_tree, const void* v_tree, const int32_t* parents, float* out,
                           float* lse, float* part_o, float* part_ml, unsigned* work, hipStream_t s);

// ---- acceptance (k_accept.hip)
sr_status launch_tree_accept(const sr_accept_desc& d, const void* target_logits, const float* child_logit,
                             const int32_t* tokens, const int32_t* parents, const float* u_acc,
                             const float* u_fin, int32_t* acc_nodes, int32_t* out_tokens, int32_t* out_len,
                             uint8_t* final_kind, float* min_margin, hipStream_t s);

// ---- engine glue (k_engine.hip)
sr_status launch_commit_path(const sr_commit_desc& d, const int32_t* acc_nodes, const int32_t* out_len,
                             const int32_t* parents, const void* k_tree, const void* v_tree,
                             const int32_t* block_table, const int32_t* ctx_len, void* k_cache, void* v_cache,
                             int32_t* new_ctx_len, hipStream_t s);

// ---- Reflex feedback (k_reflex.hip)
sr_status launch_reflex_feedback(const sr_reflex_desc& d, const void* target_logits, const int32_t* p_row,
                                 const float* head_logits, const int32_t* q_row, const int32_t* cand,
                                 const int32_t* y_star, const int32_t* traj, const int32_t* horizon, const void* W,
                                 float* memory, float* stats, float* e_out, const float* P, const float* rec_sketch,
                                 float* align, hipStream_t s);
sr_status launch_reflex_correct(const sr_heads_desc& d, const sr_reflex_gate_desc& g, void* z, const float* memory,
                                const float* align, const float* P, float* sketch_out, float* alpha_out,
                                hipStream_t s);

}  // namespace sr
