// Accepted-path cache extraction: the root and the accepted nodes' K/V rows of every layer are
// appended to each trajectory's paged cache after the acceptance walk.
//
// HBM-bound copy with almost no arithmetic: a launch moves 2 * (1 + n_acc) * Hkv * D elements per
// (layer, trajectory) in and out. A step commits only a few rows per trajectory, so the copy is short
// and latency-bound; what pays is many small independent workgroups: one per (trajectory, layer)
// validates the trajectory's inputs into LDS, then its lanes stream 16-byte vectors (grouping several
// layers per workgroup, with their loads in flight together, measured twice as slow at the 7B shape).
// Consecutive lanes take consecutive vectors of one (row, head), so each 16-lane group moves one
// contiguous 256-byte head row at D = 128 bf16, source and destination alike.
#include "common.hpp"
#include "kernels.hpp"

namespace sr {

constexpr int CM_NT = 256;

__global__ __launch_bounds__(CM_NT) void k_commit_path(
    const int32_t* __restrict__ acc_nodes, const int32_t* __restrict__ out_len, const int32_t* __restrict__ parents,
    const uint4* __restrict__ k_tree, const uint4* __restrict__ v_tree, const int32_t* __restrict__ block_table,
    const int32_t* __restrict__ ctx_len, uint4* __restrict__ k_cache, uint4* __restrict__ v_cache,
    int32_t* __restrict__ new_ctx_len, int T, int Hkv, int row_vec, int bs, int max_blocks, int num_blocks,
    int max_depth) {
  __shared__ int s_node[SR_MAX_TREE + 1];
  __shared__ int s_page[SR_MAX_TREE + 1];
  __shared__ int s_bad;
  const int b = blockIdx.x, layer = blockIdx.y, B = gridDim.x;
  const int tid = threadIdx.x;
  if (tid == 0) s_bad = 0;
  const int n1 = out_len[b];
  const int L = ctx_len[b];
  // uniform over the block: every lane reads the same two values
  const bool shape_bad = n1 < 1 || n1 > max_depth + 1 || L < 0 || (long long)L + n1 > (long long)max_blocks * bs;
  __syncthreads();
  if (!shape_bad) {
    for (int i = tid; i < n1; i += CM_NT) {
      const int u = i == 0 ? 0 : acc_nodes[(size_t)b * max_depth + (i - 1)];
      bool ok = i == 0 || (u >= 1 && u < T);
      if (ok && i > 0 && parents != nullptr) {
        const int want = i == 1 ? 0 : acc_nodes[(size_t)b * max_depth + (i - 2)];
        ok = parents[(size_t)b * T + u] == want;
      }
      const int pos = L + i;
      const int page = block_table[(size_t)b * max_blocks + pos / bs];
      ok = ok && page >= 0 && page < num_blocks;
      s_node[i] = u;
      s_page[i] = page;
      if (!ok) atomicOr(&s_bad, 1);
    }
  }
  __syncthreads();
  if (shape_bad || s_bad) {
    if (layer == 0 && tid == 0) new_ctx_len[b] = -1;
    return;
  }
  if (layer == 0 && tid == 0) new_ctx_len[b] = L + n1;

  const size_t head_vec = (size_t)row_vec;              // 16-byte vectors per (row, head)
  const size_t node_vec = (size_t)Hkv * head_vec;       // per tree node
  const size_t slot_vec = head_vec;                     // per cache slot of one head
  const size_t page_head_vec = (size_t)bs * head_vec;   // one head's part of a page
  const size_t page_vec = (size_t)Hkv * page_head_vec;
  const size_t tree_base = ((size_t)layer * B + b) * (size_t)T * node_vec;
  const size_t cache_base = (size_t)layer * (size_t)num_blocks * page_vec;
  const int per_kv = n1 * Hkv * row_vec;
  for (int it = tid; it < 2 * per_kv; it += CM_NT) {
    const int kv = it >= per_kv;
    const int r = it - kv * per_kv;
    const int c = r % row_vec;
    const int gh = r / row_vec;
    const int g = gh % Hkv;
    const int i = gh / Hkv;
    const int pos = L + i;
    const size_t src = tree_base + (size_t)s_node[i] * node_vec + (size_t)g * head_vec + c;
    const size_t dst = cache_base + (size_t)s_page[i] * page_vec + (size_t)g * page_head_vec +
                       (size_t)(pos % bs) * slot_vec + c;
    if (kv)
      v_cache[dst] = v_tree[src];
    else
      k_cache[dst] = k_tree[src];
  }
}

sr_status launch_commit_path(const sr_commit_desc& d, const int32_t* acc_nodes, const int32_t* out_len,
                             const int32_t* parents, const void* k_tree, const void* v_tree,
                             const int32_t* block_table, const int32_t* ctx_len, void* k_cache, void* v_cache,
                             int32_t* new_ctx_len, hipStream_t s) {
  const int esz = d.dtype == SR_BF16 ? 2 : 4;
  const int row_vec = d.D * esz / 16;
  SR_LAUNCH("sr_commit_path", k_commit_path, dim3(d.B, d.n_layers), dim3(CM_NT), 0, s, acc_nodes, out_len, parents,
            (const uint4*)k_tree, (const uint4*)v_tree, block_table, ctx_len, (uint4*)k_cache, (uint4*)v_cache,
            new_ctx_len, d.T, d.Hkv, row_vec, d.block_size, d.max_blocks, d.num_blocks, d.max_depth);
  return SR_OK;
}

}  // namespace sr
