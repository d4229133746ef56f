"""Draft-tree construction from head logits (oracle; test infrastructure only).

Paper: App. B.1 ("Tree proposal law"). A node u at speculative depth d is
proposed from by head k = d + 1; nodes at one depth share that head's logits.
The builder picks a finite support C_u and draws an ordered list of m_u
distinct children without replacement: slot j draws from q_{u,j}, the head
distribution restricted to the not-yet-drawn part R_{u,j} of C_u and
renormalised (Eq. (slotq)); the list has probability prod_j q_{u,j}(y_{u,j})
(Eq. (childlist)).

Readings taken here:
* C_u is the m_u highest-logit tokens of the head row, ordered by (logit
  descending, token id ascending); so |C_u| = m_u.
* When a node is deeper than the number of heads, the last head proposes
  (the paper allows a proposal that ignores part of its context).
* Slot j is drawn by inverse CDF over R_{u,j} in C_u's order with the
  uniform indexed by the child node that fills the slot: the first v with
  U * S < (cumulative weight through v), weights exp(l_v - max_R l), S the
  total weight.
* Children of a node, in increasing node index, are its slots 1..m_u.
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np


def tree_structure(parents: np.ndarray) -> Tuple[np.ndarray, List[List[int]]]:
    """Depth of every node and each node's children in increasing index (= slot order).

    Requires parents[0] == -1 and 0 <= parents[c] < c for c >= 1.
    """
    parents = np.asarray(parents)
    T = parents.shape[0]
    if T < 1 or parents[0] != -1:
        raise ValueError("node 0 must be the root (parent -1)")
    depth = np.zeros(T, dtype=np.int64)
    kids: List[List[int]] = [[] for _ in range(T)]
    for c in range(1, T):
        p = int(parents[c])
        if not 0 <= p < c:
            raise ValueError(f"parents[{c}]={p} is not an earlier node")
        depth[c] = depth[p] + 1
        kids[p].append(c)
    return depth, kids


def top_m(row: np.ndarray, m: int) -> np.ndarray:
    """Ids of the m largest entries, ordered by (value descending, id ascending)."""
    ids = np.arange(row.shape[0])
    order = np.lexsort((ids, -np.asarray(row, dtype=np.float64)))
    return order[:m]


def sample_ordered_children(cand_ids: np.ndarray, cand_logits: np.ndarray, us) -> Tuple[list, list, float]:
    """Sequential draws without replacement (Eq. (slotq)); one uniform per slot.

    Returns the drawn ids, their logits and the smallest relative distance of
    U*S to a cumulative-weight boundary seen over the draws (the decision margin).
    """
    remaining = list(range(len(cand_ids)))
    drawn_ids, drawn_logits = [], []
    margin = np.inf
    for U in us:
        lg = np.asarray([cand_logits[i] for i in remaining], dtype=np.float64)
        w = np.exp(lg - lg.max())
        cum = np.cumsum(w)
        S = cum[-1]
        target = float(U) * S
        pick = int(np.searchsorted(cum, target, side="right"))  # first index with target < cum
        pick = min(pick, len(remaining) - 1)
        lo = cum[pick - 1] if pick > 0 else 0.0
        margin = min(margin, (target - lo) / S, (cum[pick] - target) / S)
        i = remaining.pop(pick)
        drawn_ids.append(int(cand_ids[i]))
        drawn_logits.append(float(cand_logits[i]))
    return drawn_ids, drawn_logits, margin


def tree_build(logits: np.ndarray, parents: np.ndarray, root_token: np.ndarray, u_tree: np.ndarray):
    """Tokens and draft logits of every tree node.

    logits [B,H,V] (head logits, float), parents [B,T], root_token [B], u_tree [B,T].
    Returns tokens [B,T] int32, child_logit [B,T] float64 (0 at the root) and
    margin [B] (smallest sampling margin of each trajectory, inf if none).
    """
    B, H, V = logits.shape
    T = parents.shape[1]
    tokens = np.zeros((B, T), dtype=np.int32)
    child_logit = np.zeros((B, T), dtype=np.float64)
    margin = np.full(B, np.inf)
    for b in range(B):
        depth, kids = tree_structure(parents[b])
        tokens[b, 0] = root_token[b]
        for u in range(T):
            ch = kids[u]
            if not ch:
                continue
            k = min(int(depth[u]) + 1, H)                      # proposing head (1-based)
            row = np.asarray(logits[b, k - 1], dtype=np.float64)
            cand = top_m(row, len(ch))                          # C_u
            ids, lgs, mg = sample_ordered_children(cand, row[cand], [u_tree[b, c] for c in ch])
            for j, c in enumerate(ch):
                tokens[b, c] = ids[j]
                child_logit[b, c] = lgs[j]
            margin[b] = min(margin[b], mg)
    return tokens, child_logit, margin
