"""Engine steps around the verification step (oracle; test infrastructure only).

Paper: Sec. 3.2, Eq. (verification-budget) and Eq. (tree-budget); App. C "Implementation and
Reproducibility Details", paragraph "Concurrency-aware sparse tree verification" (C_peak = 512,
N_min = 1, N_max = 10, root counted, nominal non-root allocation (5, 4, 0) over the horizons,
truncated to the budget); App. C, paragraph "Metrics and timing" (accepted-path cache extraction is
part of each step).

Readings taken here (the paper leaves them open):
* Truncation keeps the shallowest horizons first: horizon h receives min(n_h^nominal, what is left of
  N_t - 1 after horizons 1..h-1). A horizon that receives no node ends the tree (deeper horizons would
  have no parents).
* Nodes of horizon h hang under the nodes of horizon h-1 in slot order: node k of horizon h (0-based)
  has parent number floor(k * n_{h-1} / n_h) of horizon h-1; nodes are numbered breadth-first.
* Cache extraction appends the root (anchor, node 0) and then the accepted nodes in walk order at
  positions L_b, L_b + 1, ... of the trajectory's paged cache; the final (fallback or bonus) token is
  the next round's anchor and has no K/V yet. ctx_len grows by out_len = 1 + n_acc.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


def tree_budget(live: int, c_peak: int = 512, n_min: int = 1, n_max: int = 10,
                alloc: Sequence[int] = (5, 4, 0)) -> Tuple[int, List[int], np.ndarray]:
    """Per-response node budget N_t = clip(floor(c_peak / live), n_min, n_max) and the tree it allows.

    Returns (N_t, per-horizon node counts, parents array of the tree, breadth-first, parents[0] = -1).
    """
    if live < 1:
        raise ValueError("live must be >= 1")
    if not (1 <= n_min <= n_max):
        raise ValueError("need 1 <= n_min <= n_max")
    n_t = min(max(c_peak // live, n_min), n_max)
    left = n_t - 1                      # the root is counted in N_t
    counts: List[int] = []
    for a in alloc:
        if a < 0:
            raise ValueError("allocations must be >= 0")
        take = min(a, left)
        if take == 0:
            break
        counts.append(take)
        left -= take
    parents = [-1]
    prev_start, prev_n, start = 0, 1, 1
    for n in counts:
        for k in range(n):
            parents.append(prev_start + (k * prev_n) // n)
        prev_start, prev_n = start, n
        start += n
    return n_t, counts, np.asarray(parents, dtype=np.int32)


def commit_path(k_cache: np.ndarray, v_cache: np.ndarray, block_table: np.ndarray, ctx_len: np.ndarray,
                k_tree: np.ndarray, v_tree: np.ndarray, acc_nodes: np.ndarray, out_len: np.ndarray,
                block_size: int = 16):
    """Write the root and the accepted nodes' K/V rows into each trajectory's pages.

    k_cache/v_cache [num_blocks, Hkv, block_size, D], block_table [B, max_blocks], ctx_len [B],
    k_tree/v_tree [B, T, Hkv, D], acc_nodes [B, max_depth] (-1 padded), out_len [B] = 1 + n_acc.
    Returns new (k_cache, v_cache, ctx_len) arrays; the inputs are not modified.
    """
    kc = np.array(k_cache, copy=True)
    vc = np.array(v_cache, copy=True)
    ctx = np.array(ctx_len, dtype=np.int32, copy=True)
    for b in range(ctx.shape[0]):
        n = int(out_len[b]) - 1
        nodes = [0] + [int(x) for x in acc_nodes[b, :n]]
        for i, u in enumerate(nodes):
            pos = int(ctx_len[b]) + i
            page = int(block_table[b, pos // block_size])
            slot = pos % block_size
            kc[page, :, slot, :] = k_tree[b, u]
            vc[page, :, slot, :] = v_tree[b, u]
        ctx[b] = int(ctx_len[b]) + len(nodes)
    return kc, vc, ctx
