/*
 * specroll.h -- C ABI of the MI355X (gfx950) speculative verification step.
 *
 * One speculative round for a batch of live trajectories, after SpecRoll
 * (arXiv 2608.04962):
 *   1. sr_heads_propose     future-token heads on the last hidden state plus a
 *                           norm-clipped Reflex correction propose a draft tree
 *                           (Sec. 3.2 Eq. (heads); App. C "Future-token
 *                           proposer"; App. B.1 Eq. (slotq), Eq. (childlist)).
 *      sr_tree_build        the tree-build part of step 1 on given head logits.
 *   2. sr_tree_verify_attn  target attention of every tree node over its
 *                           trajectory's paged KV prefix and its own root path
 *                           (App. B.1 Eq. (nodep)).
 *   3. sr_tree_accept       exact node-wise speculative acceptance walk
 *                           (App. B.2 Eq. (nodeaccept), Eq. (noderesidual),
 *                           Alg. "Exact node-wise tree verification").
 *   4. sr_commit_path       the accepted path's K/V rows appended to the paged
 *                           cache, every layer in one launch.
 *      sr_tree_budget       host rule for the per-response node budget and the
 *                           tree it allows (Sec. 3.2 Eq. (verification-budget),
 *                           Eq. (tree-budget)).
 *   5. sr_reflex_feedback   verifier feedback of matured proposals folded into the
 *                           trajectory-local Reflex memory and its delayed-alignment
 *                           statistics (Sec. 3.3; Sec. 3.4 Eq. (support) to Eq. (ema),
 *                           Eq. (reliability-score)).
 *      sr_heads_propose_reflex  step 1 with the paper-form gated correction of the
 *                           head states from that memory (Sec. 3.4
 *                           Eq. (reflex-correction)).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers named in an argument list are DEVICE pointers unless stated
 *   otherwise; descriptors are HOST pointers. All arrays are dense, row-major,
 *   in the layout given. The caller owns every buffer; the library allocates no
 *   device memory and keeps no per-call state.
 * - `stream` is a hipStream_t (NULL = the null stream). Work is enqueued and the
 *   call returns without synchronising; faults inside kernels surface at the
 *   caller's next synchronisation.
 * - `workspace` is device scratch of at least the size the matching
 *   *_workspace query returns (which may be 0, and then `workspace` may be NULL);
 *   it must be 256-byte aligned. Bulk operand and output arrays (hidden, A, bias,
 *   W, logits, z, q, caches, target_logits) must be 16-byte aligned.
 * - Arguments are checked on the host before anything is enqueued. A failed
 *   check returns a non-zero sr_status, leaves every output untouched and sets a
 *   thread-local message readable through sr_last_error().
 * - Values that live on the device (parents, ctx_len, block ids, tokens) are
 *   checked by the kernels themselves; a trajectory whose device-side inputs are
 *   malformed gets the "invalid" outputs each call documents, never an
 *   out-of-bounds access.
 * - Tree topology: parents[b][0] == -1 and 0 <= parents[b][c] < c for c >= 1.
 *   The children of a node, in increasing node index, are its slots 1..m.
 *   T <= SR_MAX_TREE.
 * - Element types: SR_F32 or SR_BF16 (bfloat16 stored as 16-bit patterns).
 *   Matrix products take bf16 operands with fp32 accumulation, or fp32
 *   operands with fp32 accumulation.
 */
#ifndef SPECROLL_H
#define SPECROLL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SR_MAX_TREE 128

typedef enum {
  SR_OK = 0,
  SR_ERR_INVALID = 1,      /* bad descriptor, null pointer or shape          */
  SR_ERR_UNSUPPORTED = 2,  /* valid request outside the built kernel set     */
  SR_ERR_WORKSPACE = 3,    /* workspace missing or smaller than required     */
  SR_ERR_HIP = 4           /* a HIP runtime call or kernel launch failed     */
} sr_status;

typedef enum { SR_F32 = 0, SR_BF16 = 1 } sr_dtype;

/* Message for the last non-OK status returned on this thread ("" if none). */
const char* sr_last_error(void);
/* Library version string. */
const char* sr_version(void);

/* ========================================================================== *
 * 1. Proposal: heads + tree build
 * ========================================================================== *
 * For every trajectory b (Sec. 3.2 Eq. (heads); App. C):
 *   D'_b  = active_b ? corr_b * min(1, clip_norm / ||corr_b||_2) : 0
 *           (a zero correction stays zero)
 *   x_b   = hidden_b + D'_b                                       (fp32)
 *   n_b   = LayerNorm(x_b), biased variance, eps = ln_eps, no affine;
 *           rounded to `dtype`
 *   z_b,h = x_b + SiLU(A_h n_b + bias_h),  h = 1..H;  rounded to `dtype`
 *   logits_b,h = W z_b,h                                           (fp32)
 * then the draft tree (App. B.1): node u at depth d is proposed from by head
 * k = min(d + 1, H). With m_u children, C_u = the m_u largest entries of
 * logits_b,k ordered by (logit descending, token id ascending). The children
 * of u fill slots 1..m_u in index order; slot j draws without replacement from
 * the not-yet-drawn part R of C_u with weights exp(l_v - max_R l), by inverse
 * CDF over R in C_u's order: the first v with U * S < cumulative weight
 * through v, S the total, U = u_tree[b][child]. Weights and sums are float64.
 */
typedef struct {
  int32_t B;             /* trajectories, >= 1                                */
  int32_t d;             /* hidden size, multiple of 64                       */
  int32_t H;             /* future-token heads, >= 1                          */
  int32_t V;             /* vocabulary, a multiple of 8, >= max_children      */
  int32_t T;             /* tree nodes incl. the root, 1..SR_MAX_TREE         */
  int32_t max_children;  /* upper bound on any node's child count, 0..T-1     */
  sr_dtype dtype;        /* element type of hidden, A, bias, W and z          */
  float clip_norm;       /* L2 bound c of the Reflex correction, > 0          */
  float ln_eps;          /* LayerNorm epsilon, >= 0                           */
} sr_heads_desc;

size_t sr_heads_propose_workspace(const sr_heads_desc* desc);

/*
 * hidden      [B,d]    dtype   last hidden state h_t of each trajectory
 * corr        [B,d]    fp32    Reflex correction vector (NULL = none)
 * corr_active [B]      uint8   nonzero = apply corr (NULL = all active)
 * A           [H,d,d]  dtype   head matrices, A[h][out][in]
 * bias        [H,d]    dtype
 * W           [V,d]    dtype   shared vocabulary projection (row = token)
 * parents     [B,T]    int32   tree topology (see conventions)
 * root_token  [B]      int32   the anchor token, already sampled
 * u_tree      [B,T]    fp32    uniforms in (0,1); entry c orders the slot node c fills
 * logits      [B,H,V]  fp32    OUT (optional, NULL = keep in workspace); 16-byte aligned
 * z           [B,H,d]  dtype   OUT (optional, NULL = keep in workspace); 16-byte aligned
 * tokens      [B,T]    int32   OUT; tokens[b][0] = root_token[b]
 * child_logit [B,T]    fp32    OUT; head logit of tokens[b][c] under the proposing
 *                              head; 0 at the root
 * Invalid trajectory (bad topology, more than max_children children at a node):
 * its tokens are -1 and child_logit NaN for every non-root node.
 */
sr_status sr_heads_propose(const sr_heads_desc* desc,
                           const void* hidden, const float* corr, const uint8_t* corr_active,
                           const void* A, const void* bias, const void* W,
                           const int32_t* parents, const int32_t* root_token, const float* u_tree,
                           float* logits, void* z, int32_t* tokens, float* child_logit,
                           void* workspace, size_t workspace_bytes, void* stream);

/* Tree build alone (the second half of sr_heads_propose) on caller-supplied fp32
 * head logits [B,H,V]; desc->d, dtype, clip_norm and ln_eps are ignored. */
size_t sr_tree_build_workspace(const sr_heads_desc* desc);
sr_status sr_tree_build(const sr_heads_desc* desc, const float* logits,
                        const int32_t* parents, const int32_t* root_token, const float* u_tree,
                        int32_t* tokens, float* child_logit,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ========================================================================== *
 * 2. Tree-verify attention (App. B.1 Eq. (nodep))
 * ========================================================================== *
 * For trajectory b, node u and query head h (KV head g = h / (Hq/Hkv)):
 *   keys   = prefix tokens 0..ctx_len[b]-1 from the paged cache, then the tree
 *            tokens on u's root path (ancestors and u itself)
 *   out[b][u][h] = softmax(scale * q . K^T) V,   lse[b][u][h] = logsumexp(scale * q . K^T)
 * which equals ordinary causal attention at u's position of the sequence
 * prefix ++ path(u). Scores and softmax are fp32. For bf16 inputs the
 * probability-weighted sum over V runs on fp16 matrix cores with V converted
 * bf16 -> fp16: exact for |v| in [2^-14, 65280], within 2^-24 absolute below.
 * A work item (trajectory, KV head, prefix chunk) whose largest |v| exceeds
 * 65280 (or is not finite) or lies below 2^-6 is recomputed with V in fp32,
 * so no finite bf16 V overflows and the conversion error stays below 2^-18 of
 * the item's V scale.
 */
typedef struct {
  int32_t B, T;          /* trajectories; tree nodes (1..SR_MAX_TREE)           */
  int32_t Hq, Hkv;       /* query / KV heads; Hq % Hkv == 0                     */
  int32_t D;             /* head dim: 64 or 128                                 */
  int32_t block_size;    /* tokens per KV page: 16                              */
  int32_t max_blocks;    /* columns of block_table                              */
  int32_t num_blocks;    /* pages in k_cache / v_cache                          */
  sr_dtype dtype;        /* element type of q, caches and tree K/V              */
  float scale;           /* score scale, usually 1/sqrt(D)                      */
} sr_attn_desc;

size_t sr_tree_verify_attn_workspace(const sr_attn_desc* desc);

/*
 * q           [B,T,Hq,D]                         dtype  queries of the tree nodes (positions applied)
 * k_cache     [num_blocks,Hkv,block_size,D]      dtype  paged prefix keys
 * v_cache     [num_blocks,Hkv,block_size,D]      dtype  paged prefix values
 * block_table [B,max_blocks]                     int32  physical page of logical page i
 * ctx_len     [B]                                int32  prefix tokens in the cache, 0..max_blocks*block_size
 * k_tree      [B,T,Hkv,D]                        dtype  keys of the tree tokens (node order)
 * v_tree      [B,T,Hkv,D]                        dtype  values of the tree tokens
 * parents     [B,T]                              int32  tree topology
 * out         [B,T,Hq,D]                         fp32   OUT
 * lse         [B,T,Hq]                           fp32   OUT (optional, NULL = not written)
 * Cache slots past ctx_len in a trajectory's last page are never read, nor are
 * block_table entries past its last page. Invalid trajectory (ctx_len out of
 * range, a page id outside [0,num_blocks), bad topology): out and lse are NaN.
 * Workspace: the partial results of trajectories split into prefix chunks and,
 * for bf16, the work-item counter of the persistent kernel, the list of work
 * items to recompute with fp32 V and the work items ordered by length (longest
 * first), all of which the call rebuilds itself with a kernel on the stream
 * (no initialisation by the caller, no memset). Two calls
 * that share a workspace must not run concurrently (on one stream they don't).
 */
sr_status sr_tree_verify_attn(const sr_attn_desc* desc,
                              const void* q, const void* k_cache, const void* v_cache,
                              const int32_t* block_table, const int32_t* ctx_len,
                              const void* k_tree, const void* v_tree, const int32_t* parents,
                              float* out, float* lse,
                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * sr_tree_verify_attn without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc). Arguments and results as sr_tree_verify_attn. The
 * scratch the call needs (the chunk partials, the work-item counter and list,
 * the fp32-V recomputation list: sr_tree_verify_attn_workspace bytes) lives in a
 * static device array of SR_ATTN_NOALLOC_MAX_BYTES per GPU, which the library
 * holds on every GPU it runs on until the process ends; the call itself
 * allocates nothing. A request that needs more returns SR_ERR_UNSUPPORTED with
 * nothing enqueued (use sr_tree_verify_attn with a workspace instead). The
 * current device must be the stream's device. Every call on one GPU shares
 * that GPU's array and leaves its contents there; the counters are zeroed by a
 * kernel on the stream at each call (no memset), so calls ordered on one stream
 * are safe, while calls that overlap on one GPU (other streams or threads
 * without ordering) race and give wrong results.
 */
#define SR_ATTN_NOALLOC_MAX_BYTES (256u << 20)
sr_status sr_tree_verify_attn_noalloc(const sr_attn_desc* desc,
                                      const void* q, const void* k_cache, const void* v_cache,
                                      const int32_t* block_table, const int32_t* ctx_len,
                                      const void* k_tree, const void* v_tree, const int32_t* parents,
                                      float* out, float* lse, void* stream);

/* ========================================================================== *
 * 3. Exact acceptance walk (App. B.2)
 * ========================================================================== *
 * Per trajectory, starting at the root u: p_u = softmax(target_logits[b][u] /
 * temperature), r = p_u. For the children c of u in slot order: y = tokens[c],
 * q = softmax of child_logit over the children not yet tried, accept iff
 * u_acc[b][c] <= min(1, r(y)/q(y)); on rejection r <- [r - q]_+ / Z over the
 * whole vocabulary. An accepted child with children is visited next; an
 * accepted leaf adds a bonus token drawn from its own p; if every child of a
 * node is rejected, a fallback token is drawn from the final residual. Draws use
 * the inverse CDF in token-id order with U = u_fin[b]: the first v with
 * U * S < sum_{w<=v} r(w). Walk scalars are float64; exponentials are fp32 of
 * (logit - running max) * (1/temperature), summed in float64.
 * The children of one node must carry distinct tokens.
 * With top_p < 1 every p above (visited nodes and the bonus leaf) is first cut to
 * its nucleus, as the paper's rollouts sample (App. C "Training protocol":
 * nucleus threshold 0.95): tokens ranked by (logit desc, id asc) stay while the
 * mass ranked before them is below top_p, and p is renormalised on them. Masses
 * of the cut are fp32 exponentials summed in 40-bit fixed point; the cut's
 * margin (distance of top_p to the cumulative mass around the last kept token)
 * enters min_margin.
 */
typedef struct {
  int32_t B, T, V;       /* trajectories; tree nodes (1..SR_MAX_TREE); vocabulary */
  int32_t max_depth;     /* columns of acc_nodes, >= the deepest node's depth    */
  sr_dtype logit_dtype;  /* element type of target_logits                        */
  float temperature;     /* > 0                                                  */
  float top_p;           /* nucleus threshold in (0, 1]; 1 = no truncation       */
} sr_accept_desc;

size_t sr_tree_accept_workspace(const sr_accept_desc* desc);

/*
 * target_logits [B,T,V]           dtype  row u = target logits after prefix ++ path(u)
 * child_logit   [B,T]             fp32   draft logit of each node's token (entry 0 unused)
 * tokens        [B,T]             int32  token of each node (entry 0 = the anchor, unused)
 * parents       [B,T]             int32  tree topology
 * u_acc         [B,T]             fp32   uniform of the slot test of node c (entry 0 unused)
 * u_fin         [B]               fp32   uniform of the terminal draw
 * acc_nodes     [B,max_depth]     int32  OUT accepted node ids in walk order, -1 padded
 * out_tokens    [B,max_depth+1]   int32  OUT accepted tokens then the terminal token, -1 padded
 * out_len       [B]               int32  OUT accepted count + 1
 * final_kind    [B]               uint8  OUT 0 = fallback, 1 = bonus, 255 = invalid input
 * min_margin    [B]               fp32   OUT (optional) smallest decision margin of the walk:
 *                                        |min(1,r/q) - U| for slot tests, distance of U*S to the
 *                                        drawn token's cumulative boundaries / S for draws
 * Invalid trajectory (bad topology, a token outside [0,V), duplicate sibling
 * tokens, depth > max_depth): acc_nodes/out_tokens -1, out_len 0, final_kind 255.
 */
sr_status sr_tree_accept(const sr_accept_desc* desc,
                         const void* target_logits, const float* child_logit,
                         const int32_t* tokens, const int32_t* parents,
                         const float* u_acc, const float* u_fin,
                         int32_t* acc_nodes, int32_t* out_tokens, int32_t* out_len,
                         uint8_t* final_kind, float* min_margin,
                         void* workspace, size_t workspace_bytes, void* stream);

/* ========================================================================== *
 * 4. Engine glue around the step
 * ========================================================================== *
 * Concurrency-aware node budget (Sec. 3.2 Eq. (verification-budget) and
 * Eq. (tree-budget); App. C "Implementation and Reproducibility Details",
 * paragraph "Concurrency-aware sparse tree verification"). With `live`
 * unfinished responses, each response gets
 *   N_t = clip(floor(c_peak / live), n_min, n_max)
 * tree nodes, the anchor counted once. Horizon h = 1, 2, ... receives
 * min(alloc[h-1], nodes still left of N_t - 1), shallowest first; the first
 * horizon that receives none ends the tree. Node k (0-based) of horizon h hangs
 * under node floor(k * n_{h-1} / n_h) of horizon h-1, and nodes are numbered
 * breadth-first, so `parents` is a valid topology for the calls above. The
 * paper's settings are c_peak 512, n_min 1, n_max 10 and alloc {5, 4, 0}.
 * Host-only: every pointer of this call is a HOST pointer and nothing touches
 * a GPU.
 */
typedef struct {
  int32_t c_peak;        /* profiled verification capacity, nodes per step, >= 1    */
  int32_t n_min, n_max;  /* 1 <= n_min <= n_max <= SR_MAX_TREE                       */
  int32_t n_alloc;       /* horizons listed in alloc, 0..SR_MAX_TREE                  */
  const int32_t* alloc;  /* HOST [n_alloc] nominal non-root nodes per horizon, >= 0   */
} sr_budget_desc;

/*
 * live          unfinished responses B_t, >= 1
 * n_t           OUT    the budget N_t
 * horizon_count OUT    HOST [n_alloc] (NULL = not written) nodes given to each
 *                      horizon, 0 from the first empty horizon on
 * parents       OUT    HOST [parents_cap] the tree's topology; entries past
 *                      n_nodes are not written
 * n_nodes       OUT    tree size 1 + sum(horizon_count), <= n_t
 * parents_cap >= n_max always suffices; a smaller capacity that cannot hold the
 * tree is an SR_ERR_INVALID with nothing written.
 */
sr_status sr_tree_budget(const sr_budget_desc* desc, int32_t live, int32_t* n_t, int32_t* horizon_count,
                         int32_t* parents, int32_t parents_cap, int32_t* n_nodes);

/*
 * Accepted-path cache extraction (the commit that follows acceptance in the
 * step's timing, App. C paragraph "Metrics and timing"). For every layer l and trajectory b with
 * n = out_len[b] - 1 accepted nodes, the K/V rows of the root (the anchor,
 * node 0) and then of acc_nodes[b][0..n-1] are copied, bit for bit, to sequence
 * positions ctx_len[b], ctx_len[b] + 1, ... of b's paged cache (position p is
 * slot p % block_size of page block_table[b][p / block_size]), and
 * new_ctx_len[b] = ctx_len[b] + out_len[b]. The terminal (fallback or bonus)
 * token becomes the next round's anchor and has no K/V yet. Layers are stacked
 * along the leading dimension, so one launch commits the whole model.
 */
typedef struct {
  int32_t n_layers;      /* stacked layers, 1..65535                                   */
  int32_t B, T;          /* trajectories; tree nodes (1..SR_MAX_TREE)                 */
  int32_t Hkv, D;        /* KV heads; head dim with D * element size a multiple of 16 */
  int32_t block_size;    /* tokens per KV page, >= 1                                  */
  int32_t max_blocks;    /* columns of block_table, >= 1                              */
  int32_t num_blocks;    /* pages per layer in k_cache / v_cache, >= 1                */
  int32_t max_depth;     /* columns of acc_nodes, 0..SR_MAX_TREE                      */
  sr_dtype dtype;        /* element type of the caches and tree K/V                   */
} sr_commit_desc;

/*
 * acc_nodes   [B,max_depth]                          int32  accepted node ids in walk order (as
 *                                                           sr_tree_accept writes them); may be NULL
 *                                                           when max_depth == 0
 * out_len     [B]                                    int32  1 + accepted count (as sr_tree_accept
 *                                                           writes it; its invalid 0 is rejected here)
 * parents     [B,T]                                  int32  (optional, NULL = not checked) topology;
 *                                                           when given the nodes must form a root path
 * k_tree      [n_layers,B,T,Hkv,D]                   dtype  keys of the tree tokens, every layer
 * v_tree      [n_layers,B,T,Hkv,D]                   dtype  values of the tree tokens
 * block_table [B,max_blocks]                         int32  physical page of logical page i
 * ctx_len     [B]                                    int32  tokens already in the cache
 * k_cache     [n_layers,num_blocks,Hkv,block_size,D] dtype  IN/OUT paged keys
 * v_cache     [n_layers,num_blocks,Hkv,block_size,D] dtype  IN/OUT paged values
 * new_ctx_len [B]                                    int32  OUT; -1 for a rejected trajectory
 * Rejected trajectory (out_len outside [1, max_depth + 1]; a node id outside
 * [1, T); a broken root path when parents is given; ctx_len < 0 or
 * ctx_len + out_len > max_blocks * block_size; a page to write outside
 * [0, num_blocks)): none of its cache rows is written. new_ctx_len must not
 * overlap ctx_len; tree K/V must not overlap the caches; no two trajectories
 * may write the same page slot (their writes would race). k_tree, v_tree and
 * the caches must be 16-byte aligned.
 */
sr_status sr_commit_path(const sr_commit_desc* desc, const int32_t* acc_nodes, const int32_t* out_len,
                         const int32_t* parents, const void* k_tree, const void* v_tree,
                         const int32_t* block_table, const int32_t* ctx_len, void* k_cache, void* v_cache,
                         int32_t* new_ctx_len, void* stream);

/* ========================================================================== *
 * 5. Reflex verifier feedback and memory update
 * ========================================================================== *
 * For every matured proposal record r (trajectory i, horizon h, candidate set C
 * of K tokens, realised target token y*), with p = softmax(target logits /
 * temperature) and q = softmax(head logits / temperature) over the whole
 * vocabulary (Sec. 3.3 Eq. (conditional-distributions) to
 * Eq. (acceptance-gap-decomposition); Sec. 3.4):
 *   d_dist = p(C) TV(p_C, q_C),   d_cov = p(Top_K(p)) - p(C)
 *   S      = C, then Top_K(p), then y*, then alternately the next token of
 *            Top_k(p) and of Top_k(q), duplicates skipped, at most k = support
 *            entries; top lists ordered by (logit desc, id asc)      Eq. (support)
 *   r_dist = sum_{v in S} (p_S(v) - q_S(v)) W_v                       Eq. (distdir)
 *   r_cov  = sum_{y in O} p_S(y) (W_y - mean_{b in B} W_b), O = Top_K(p) \ C,
 *            B = the n_boundary candidates of lowest head logit (ties to the lower
 *            id)                                                      Eq. (covdir)
 *   g      = w_dist d_dist r_dist / (RMS(r_dist) + eps)
 *          + w_cov d_cov r_cov / (RMS(r_cov) + eps)
 *   e      = (d_dist + d_cov) g / (RMS(g) + eps)               Eq. (unified-feedback)
 *   w      = clip(sev_tv TV(p_S, q_S) + sev_out (1 - p(C)), 0, 1)
 * and if w >= w_min: memory[i][h-1] <- rho[h-1] memory[i][h-1] + (1 - rho[h-1]) e
 * (Eq. (ema)). The paper's settings (App. C, "Verifier-derived feedback";
 * Tab. "reflex-hparams") are support 48, w_dist 0.15, w_cov 1.25, sev_tv 0.3,
 * sev_out 0.7, w_min 0.03, n_boundary 4, rho (.85, .90, .95). Exponentials are
 * fp32, sums and the per-record scalars float64, the d-vectors fp32.
 */
typedef struct {
  int32_t R;             /* records, >= 1                                          */
  int32_t V, d;          /* vocabulary (multiple of 8, <= 262144); hidden size of W
                            (multiple of 8, <= 8192)                               */
  int32_t B, H;          /* memory slots [B,H,d]; H <= 8                           */
  int32_t n_p_rows;      /* rows of target_logits                                  */
  int32_t n_q_rows;      /* rows of head_logits                                    */
  int32_t max_cand;      /* columns of cand, 1..support                            */
  int32_t support;       /* support budget k, 1..64, <= V                          */
  int32_t n_boundary;    /* boundary tokens, >= 1                                  */
  sr_dtype p_dtype;      /* element type of target_logits                          */
  sr_dtype w_dtype;      /* element type of W                                      */
  float temperature;     /* > 0                                                    */
  float w_dist, w_cov;   /* direction weights, >= 0                                */
  float sev_tv, sev_out; /* severity coefficients                                  */
  float w_min;           /* severity gate                                          */
  float eps;             /* RMS stabiliser, > 0                                    */
  float rho[8];          /* per-horizon decay in [0, 1), entries 0..H-1 used       */
  int32_t rank;          /* rows of the sketch projection P, 0..64 (0 = no alignment
                            observations)                                          */
} sr_reflex_desc;

/*
 * target_logits [n_p_rows,V]  p_dtype  target logit rows (any rows; p_row picks one per record)
 * p_row         [R]           int32    row of target_logits holding record r's target logits
 * head_logits   [n_q_rows,V]  fp32     proposal (head) logit rows
 * q_row         [R]           int32    row of head_logits holding record r's head logits
 * cand          [R,max_cand]  int32    candidate ids, distinct, in slot order, then -1 padding
 * y_star        [R]           int32    realised target token
 * traj          [R]           int32    trajectory i in [0, B)
 * horizon       [R]           int32    h in [1, H]
 * W             [V,d]         w_dtype  the shared output projection (row = token)
 * memory        [B,H,d]       fp32     IN/OUT Reflex memory m
 * stats         [R,8]         fp32     OUT d_dist, d_cov, TV(p_S,q_S), w, |S|, applied, p(C),
 *                                      p(Top_K(p)); applied = 1 (memory updated), 0 (w < w_min),
 *                                      -1 (an earlier record of the call has the same (i, h): skipped,
 *                                      so one call applies at most one record per slot, the first),
 *                                      -2 (invalid record); the other entries are NaN for -1 and -2
 * e_out         [R,d]         fp32     OUT (optional, NULL = not written) the feedback vector e
 *                                      (NaN rows for skipped and invalid records)
 * P             [rank,d]      fp32     sketch projection (NULL when rank == 0), 16-byte aligned
 * rec_sketch    [R,rank]      fp32     unit memory sketch stored when record r was proposed (as
 *                                      sr_heads_propose_reflex writes it); all zero = none
 * align         [B,H,4]       fp32     IN/OUT (optional, NULL = not kept) per (i, h): count, mean and M2
 *                                      of the alignments, and the count of applied feedback records.
 *                                      An applied record adds 1 to the last; with rank > 0 and a stored
 *                                      sketch s it adds the observation a = <s, P e / |P e|> to the
 *                                      moments by the one-pass update (no observation when P e = 0)
 * Invalid record: a row index, trajectory, horizon, y* or candidate id out of
 * range, duplicate candidates, a candidate after a -1, or no candidate.
 * Records are independent blocks; memory rows of distinct (i, h) are written by
 * distinct records only. target_logits, head_logits and W must be 16-byte
 * aligned.
 */
sr_status sr_reflex_feedback(const sr_reflex_desc* desc, const void* target_logits, const int32_t* p_row,
                             const float* head_logits, const int32_t* q_row, const int32_t* cand,
                             const int32_t* y_star, const int32_t* traj, const int32_t* horizon, const void* W,
                             float* memory, float* stats, float* e_out, const float* P, const float* rec_sketch,
                             float* align, void* stream);

/*
 * Gated head-state correction (Sec. 3.4 "Reliability from delayed alignment",
 * Eq. (reliability-score); "Gated hidden-state correction", Eq. (reflex-correction);
 * App. C "Reflex configuration", Tab. "reflex-hparams"). For trajectory b and head
 * h (horizon h+1, 0-based h here) with memory m = memory[b][h], alignment moments
 * (n, mean, M2) and feedback count n_fb = align[b][h]:
 *   Rel   = mean - z_delta * sqrt(M2 / (n - 1)) / sqrt(n)               (n >= 2)
 *   gate  = n_fb >= n_fb_min[h] and n >= max(n_align_min[h], 2) and Rel > 0
 *           and RMS(m) > m_floor
 *   alpha = gate ? alpha_min[h] + (alpha_max[h] - alpha_min[h]) * min(Rel, 1) : 0
 *   z~    = z + alpha * RMS(z) * m / (RMS(m) + eps), rounded to the head dtype
 * and the memory sketch P m / |P m| (zero when P m = 0) is written for the caller
 * to store with the records proposed now. The paper's settings: z_delta 0.6,
 * n_fb_min (1, 2, 4), n_align_min (6, 16, 48), intervals (1.0-2.5 %, 0.4-1.0 %,
 * 0.25-0.6 %), the last entry reused for further heads.
 */
typedef struct {
  int32_t rank;          /* rows of P, 0..64 (0 = no sketches)                     */
  float z_delta;         /* >= 0                                                   */
  float eps;             /* > 0                                                    */
  float m_floor;         /* >= 0: memory with RMS <= m_floor is negligible          */
  float alpha_min[8];    /* per head, 0 <= alpha_min <= alpha_max                  */
  float alpha_max[8];
  int32_t n_fb_min[8];   /* per head, >= 0                                         */
  int32_t n_align_min[8];
} sr_reflex_gate_desc;

/*
 * Step 1 (sr_heads_propose) with the gated correction applied to the head states
 * between the head GEMM and the vocabulary projection. Arguments as
 * sr_heads_propose (H <= 8; the workspace size is sr_heads_propose_workspace's),
 * plus:
 * memory      [B,H,d]     fp32  Reflex memory
 * align       [B,H,4]     fp32  alignment moments and feedback counts (sr_reflex_feedback's)
 * P           [rank,d]    fp32  sketch projection (NULL when rank == 0), 16-byte aligned
 * sketch_out  [B,H,rank]  fp32  OUT (optional) unit memory sketch of every (b, h)
 * alpha_out   [B,H]       fp32  OUT (optional) the applied ratio alpha (0 = no correction)
 * z then holds z~ when requested.
 */
sr_status sr_heads_propose_reflex(const sr_heads_desc* desc, const sr_reflex_gate_desc* gate,
                                  const void* hidden, const float* corr, const uint8_t* corr_active,
                                  const void* A, const void* bias, const void* W,
                                  const int32_t* parents, const int32_t* root_token, const float* u_tree,
                                  const float* memory, const float* align, const float* P,
                                  float* logits, void* z, int32_t* tokens, float* child_logit,
                                  float* sketch_out, float* alpha_out,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* ========================================================================== *
 * Kernel timing hook
 * ========================================================================== *
 * Between sr_prof_begin and sr_prof_end, every launch of the kernel whose name
 * contains `kernel_substr` is bracketed by a pair of HIP events on its own
 * stream (at most 4096 launches). sr_prof_end synchronises those events and
 * returns the summed duration in milliseconds and the launch count. Kernel names
 * are listed by sr_kernel_names (a ';'-separated host string). Not thread-safe.
 */
sr_status sr_prof_begin(const char* kernel_substr);
sr_status sr_prof_end(double* total_ms, int32_t* launches);
const char* sr_kernel_names(void);

#ifdef __cplusplus
}
#endif

#endif /* SPECROLL_H */
