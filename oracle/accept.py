"""Exact node-wise tree verification (oracle; test infrastructure only).

Paper: App. B.2. At a visited node u the residual starts as the target
distribution p_u. Children are tried in slot order; candidate y at slot j is
accepted with probability min(1, r(y) / q_{u,j}(y)) (Eq. (nodeaccept)), where
q_{u,j} is the draft distribution renormalised over the children not yet tried
(Eq. (slotq)). After a rejection the full-vocabulary residual becomes
[r - q_{u,j}]_+ / Z (Eq. (noderesidual)). An accepted child with children of
its own is visited next; an accepted leaf is followed by one bonus token drawn
from its own target distribution; if every child of a node is rejected, one
fallback token is drawn from the final residual (Alg. "Exact node-wise tree
verification"). App. B.3 proves the committed tokens follow the target law.

Readings taken here:
* Target distribution p_u = softmax(target_logits[u] / temperature), then, when top_p < 1, nucleus
  truncation as the rollouts use it (App. C "Training protocol": temperature 1.0, nucleus threshold 0.95):
  tokens are ranked by (logit desc, id asc) and the smallest prefix of that ranking whose mass reaches
  top_p is kept (a token is kept iff the mass ranked before it is below top_p); p_u is renormalised on
  it. The same law is used at every visited node and for the bonus token. The margin of the truncation
  is the distance of top_p to the cumulative mass before and through the last kept token.
* The draft distribution over the children of u is the softmax of their
  ``child_logit`` values (the head logits of the drafted tokens), restricted
  to the children not yet tried.
* A candidate is accepted iff U <= min(1, r(y)/q(y)), U = u_acc[child].
* The terminal token (fallback or bonus) is drawn by inverse CDF in token-id
  order with U = u_fin: the first v with U * S < sum_{w <= v} r(w), S = sum r.
* The decision margin of a slot test is |min(1, r/q) - U|; that of an
  inverse-CDF draw is the distance of U*S to the nearer boundary of the drawn
  token's cumulative interval, divided by S.
"""
from __future__ import annotations

import numpy as np

from .tree import tree_structure

FALLBACK = 0
BONUS = 1


def inverse_cdf(r: np.ndarray, U: float):
    """First token v with U * S < cumsum(r)[v]; returns (v, relative margin)."""
    cum = np.cumsum(r)
    S = cum[-1]
    target = float(U) * S
    v = int(np.searchsorted(cum, target, side="right"))
    v = min(v, r.shape[0] - 1)
    lo = cum[v - 1] if v > 0 else 0.0
    return v, min(target - lo, cum[v] - target) / S


def _target_dist(logits_row: np.ndarray, temperature: float, top_p: float = 1.0):
    """(p_u, truncation margin); the margin is inf without truncation."""
    row = np.asarray(logits_row, dtype=np.float64)
    s = row / temperature
    e = np.exp(s - s.max())
    p = e / e.sum()
    if top_p >= 1.0:
        return p, np.inf
    order = np.lexsort((np.arange(row.shape[0]), -row))      # logit desc, id asc
    cum = np.cumsum(p[order])
    before = cum - p[order]
    n_keep = int(np.count_nonzero(before < top_p))
    kept = order[:n_keep]
    out = np.zeros_like(p)
    out[kept] = p[kept] / p[kept].sum()
    margin = min(top_p - before[n_keep - 1], cum[n_keep - 1] - top_p)
    return out, abs(margin)


def tree_accept_one(target_logits: np.ndarray, child_logit: np.ndarray, tokens: np.ndarray,
                    parents: np.ndarray, u_acc: np.ndarray, u_fin: float, temperature: float = 1.0,
                    top_p: float = 1.0):
    """One trajectory. target_logits [T,V]; the other arrays are [T].

    Returns dict(acc_nodes, out_tokens, kind, margin, slot_margins).
    """
    depth, kids = tree_structure(parents)
    V = target_logits.shape[1]
    acc_nodes, out_tokens, margins = [], [], []
    u = 0
    while True:
        p, tm = _target_dist(target_logits[u], temperature, top_p)
        if top_p < 1.0:
            margins.append(tm)
        r = p.copy()                                           # r_u^(0) = p_u
        ch = kids[u]
        accepted = None
        for j, c in enumerate(ch):
            rest = ch[j:]                                      # R_{u,j}: children not yet tried
            cl = np.asarray([child_logit[x] for x in rest], dtype=np.float64)
            w = np.exp(cl - cl.max())
            q = np.zeros(V)
            q[[int(tokens[x]) for x in rest]] = w / w.sum()    # q_{u,j} on the full vocabulary
            y = int(tokens[c])
            A = min(1.0, r[y] / q[y])
            U = float(u_acc[c])
            margins.append(abs(A - U))
            if U <= A:
                accepted = c
                break
            pos = np.maximum(r - q, 0.0)
            r = pos / pos.sum()                                # Eq. (noderesidual)
        if accepted is None:
            tok, mg = inverse_cdf(r, u_fin)                    # fallback from the final residual
            margins.append(mg)
            out_tokens.append(tok)
            kind = FALLBACK
            break
        acc_nodes.append(accepted)
        out_tokens.append(int(tokens[accepted]))
        if kids[accepted]:
            u = accepted
            continue
        pl, tm = _target_dist(target_logits[accepted], temperature, top_p)
        if top_p < 1.0:
            margins.append(tm)
        tok, mg = inverse_cdf(pl, u_fin)                       # bonus at the leaf
        margins.append(mg)
        out_tokens.append(tok)
        kind = BONUS
        break
    return dict(acc_nodes=acc_nodes, out_tokens=out_tokens, kind=kind,
                margin=min(margins) if margins else np.inf, slot_margins=margins)


def tree_accept(target_logits, child_logit, tokens, parents, u_acc, u_fin, temperature: float = 1.0,
                max_depth: int = None, rows=None, top_p: float = 1.0):
    """Batched wrapper with the library's output layout.

    target_logits [B,T,V] (float64 values), child_logit/tokens/parents/u_acc [B,T], u_fin [B].
    Returns acc_nodes [B,max_depth] (-1 padded), out_tokens [B,max_depth+1] (-1 padded),
    out_len [B], final_kind [B], min_margin [B].
    ``rows`` restricts the work to those trajectories (others stay -1 / NaN).
    """
    B, T = tokens.shape
    if max_depth is None:
        max_depth = max(int(tree_structure(parents[b])[0].max()) for b in range(B))
    acc = np.full((B, max_depth), -1, dtype=np.int32)
    outt = np.full((B, max_depth + 1), -1, dtype=np.int32)
    out_len = np.zeros(B, dtype=np.int32)
    kind = np.full(B, 255, dtype=np.uint8)
    margin = np.full(B, np.nan)
    for b in (range(B) if rows is None else rows):
        res = tree_accept_one(target_logits[b], child_logit[b], tokens[b], parents[b], u_acc[b],
                              float(u_fin[b]), temperature, top_p)
        n = len(res["acc_nodes"])
        acc[b, :n] = res["acc_nodes"]
        outt[b, :n + 1] = res["out_tokens"]
        out_len[b] = n + 1
        kind[b] = res["kind"]
        margin[b] = res["margin"]
    return dict(acc_nodes=acc, out_tokens=outt, out_len=out_len, final_kind=kind, min_margin=margin)
