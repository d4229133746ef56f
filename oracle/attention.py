"""Tree-masked target attention over a paged prefix (oracle; test infrastructure only).

Paper: App. B.1, Eq. (nodep). One packed target forward must give, at every
tree node u, exactly what an ordinary autoregressive forward gives at the
prefix x_{<=t} followed by path(u). For one attention layer that means: the
query of node u attends to the trajectory's whole cached prefix and to the
tree tokens on its own root path (ancestors and itself), nothing else.

Readings taken here: scores are scaled by ``scale`` (1/sqrt(D) by default);
query head h reads KV head h // (Hq/Hkv); queries and keys arrive with
positions already applied.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

from .numerics import logsumexp
from .tree import tree_structure


def gather_prefix(cache: np.ndarray, block_table: np.ndarray, L: int, block_size: int) -> np.ndarray:
    """Tokens 0..L-1 of one trajectory from a paged cache [num_blocks, Hkv, block_size, D] -> [L, Hkv, D]."""
    if L == 0:
        return np.zeros((0, cache.shape[1], cache.shape[3]), dtype=np.float64)
    pos = np.arange(L)
    blocks = block_table[pos // block_size]
    slots = pos % block_size
    return np.asarray(cache[blocks, :, slots, :], dtype=np.float64)


def _path(parents: np.ndarray, u: int) -> list:
    path = [u]
    while path[-1] != 0:
        path.append(int(parents[path[-1]]))
    return path[::-1]


def tree_attention_node(q_u: np.ndarray, keys: np.ndarray, values: np.ndarray, scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """Plain softmax attention of the Hq query vectors of one node over given keys/values [Lk, Hkv, D]."""
    Hq, D = q_u.shape
    Hkv = keys.shape[1]
    G = Hq // Hkv
    out = np.empty((Hq, D))
    lse = np.empty(Hq)
    for h in range(Hq):
        g = h // G
        s = (keys[:, g, :] @ q_u[h]) * scale
        lse[h] = logsumexp(s)
        out[h] = np.exp(s - lse[h]) @ values[:, g, :]
    return out, lse


def tree_attention(q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, parents, scale,
                   block_size: int = 16, nodes=None):
    """Attention output [B,T,Hq,D] and log-sum-exp [B,T,Hq] (float64).

    ``nodes`` optionally restricts the work to a list of (b, u) pairs; other
    entries are left NaN.
    """
    B, T, Hq, D = q.shape
    out = np.full((B, T, Hq, D), np.nan)
    lse = np.full((B, T, Hq), np.nan)
    want = None if nodes is None else {}
    if nodes is not None:
        for b, u in nodes:
            want.setdefault(int(b), []).append(int(u))
    for b in range(B):
        if want is not None and b not in want:
            continue
        tree_structure(parents[b])                     # validates the topology
        kp = gather_prefix(k_cache, block_table[b], int(ctx_len[b]), block_size)
        vp = gather_prefix(v_cache, block_table[b], int(ctx_len[b]), block_size)
        for u in (range(T) if want is None else want[b]):
            path = _path(parents[b], u)
            keys = np.concatenate([kp, np.asarray(k_tree[b, path], dtype=np.float64)], axis=0)
            vals = np.concatenate([vp, np.asarray(v_tree[b, path], dtype=np.float64)], axis=0)
            out[b, u], lse[b, u] = tree_attention_node(np.asarray(q[b, u], dtype=np.float64), keys, vals, scale)
    return out, lse
