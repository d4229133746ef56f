"""Reflex verifier feedback and trajectory-local memory update (oracle; test infrastructure only).

Paper: Sec. 3.3, Eq. (optimal-candidates), Eq. (conditional-distributions), Eq. (conditional-overlap),
Eq. (acceptance-gap-decomposition): the distribution error d_dist = p(C) TV(p_C, q_C) and the coverage
error d_cov = p(Top_K(p)) - p(C) of a matured proposal with candidate set C, |C| = K.
Sec. 3.4, Eq. (support), Eq. (distdir), Eq. (covdir), Eq. (unified-feedback), Eq. (ema): the sparse
support S, the distribution direction W_S^T (p_S - q_S), the coverage direction
sum_{y in O} p_S(y) (W_y - W_B) with O = Top_K(p) minus C, RMS normalisation, the combined feedback e and
the EMA m <- rho m + (1 - rho) e. App. A.1 (Prop. "Pointwise surrogate representation") gives the
coverage direction with a weighted boundary set B. App. C, paragraph "Verifier-derived feedback":
support budget 48, weights 0.15 and 1.25, severity clip(0.3 TV(p_S, q_S) + 0.7 p_out, 0, 1), records with
severity below 0.03 discarded, four boundary tokens; Tab. "reflex-hparams": rho = (.85, .90, .95).

Readings taken here (the paper is silent or inconsistent):
* p = softmax(target logits / temperature), q = softmax(head logits / temperature), both over the whole
  vocabulary (no nucleus truncation in the feedback).
* Support order: the candidates C in their given order, then Top_K(p) (K = |C|, so O is inside S), then
  the realised token y*, then alternately the next token of Top_k(p) and of Top_k(q) (k = the support
  budget); duplicates skipped; at most ``support`` entries. Top lists are ordered by (value desc, id asc).
* The boundary set B is the n_boundary candidates with the smallest q (ties to the lower id), with
  equal weights; O tokens that the support cap dropped contribute nothing.
* The weights 0.15 / 1.25 multiply the severities: g = 0.15 d_dist rbar_dist + 1.25 d_cov rbar_cov;
  e = (d_dist + d_cov) g / (RMS(g) + eps).
* p_out = 1 - p(C), the target mass outside the candidates.
* A record updates the memory iff its severity is >= w_min; RMS(x) = sqrt(mean(x^2)).
"""
from __future__ import annotations

from typing import Sequence

import numpy as np


def _dist(logits: np.ndarray, temperature: float) -> np.ndarray:
    s = np.asarray(logits, dtype=np.float64) / temperature
    e = np.exp(s - s.max())
    return e / e.sum()


def top_list(values: np.ndarray, k: int) -> np.ndarray:
    """Ids of the k largest entries ordered by (value desc, id asc)."""
    ids = np.arange(values.shape[0])
    order = np.lexsort((ids, -np.asarray(values, dtype=np.float64)))
    return order[:k]


def rms(x: np.ndarray) -> float:
    return float(np.sqrt(np.mean(np.square(x))))


def build_support(cand: Sequence[int], top_p: Sequence[int], top_q: Sequence[int], y_star: int,
                  K: int, cap: int) -> list:
    seq = list(cand) + list(top_p[:K]) + [int(y_star)]
    rest_p, rest_q = list(top_p[K:]), list(top_q)
    for i in range(max(len(rest_p), len(rest_q))):
        if i < len(rest_p):
            seq.append(rest_p[i])
        if i < len(rest_q):
            seq.append(rest_q[i])
    S = []
    for v in seq:
        v = int(v)
        if v not in S:
            S.append(v)
        if len(S) == cap:
            break
    return S


def feedback(p_logits: np.ndarray, q_logits: np.ndarray, cand: Sequence[int], y_star: int, W: np.ndarray,
             temperature: float = 1.0, support: int = 48, w_dist: float = 0.15, w_cov: float = 1.25,
             sev_tv: float = 0.3, sev_out: float = 0.7, eps: float = 1e-6, n_boundary: int = 4) -> dict:
    """Feedback of one matured record. Returns the statistics, the support and the vector e [d]."""
    p = _dist(p_logits, temperature)
    q = _dist(q_logits, temperature)
    C = [int(c) for c in cand]
    K = len(C)
    top_p = top_list(p_logits, max(support, K))
    top_q = top_list(q_logits, support)
    # Sec. 3.3: conditional distributions on C, their overlap, the budget-matched ceiling
    pC, qC = p[C].sum(), q[C].sum()
    tv_c = 0.5 * np.abs(p[C] / pC - q[C] / qC).sum()
    p_star = p[top_p[:K]].sum()
    d_dist = pC * tv_c
    d_cov = p_star - pC
    # Sec. 3.4: support, renormalised distributions, directions
    S = build_support(C, top_p, top_q, y_star, K, support)
    pS = p[S] / p[S].sum()
    qS = q[S] / q[S].sum()
    tv_s = 0.5 * np.abs(pS - qS).sum()
    W_S = np.asarray(W[S], dtype=np.float64)                  # rows of W are read as needed
    r_dist = W_S.T @ (pS - qS)
    by_q = sorted(C, key=lambda c: (q[c], c))
    Bset = by_q[:n_boundary]
    W_B = np.asarray(W[Bset], dtype=np.float64).mean(axis=0)
    O = [int(y) for y in top_p[:K] if int(y) not in C and int(y) in S]
    r_cov = np.zeros(W_S.shape[1])
    for y in O:
        r_cov += pS[S.index(y)] * (W_S[S.index(y)] - W_B)
    rbar_dist = r_dist / (rms(r_dist) + eps)
    rbar_cov = r_cov / (rms(r_cov) + eps)
    g = w_dist * d_dist * rbar_dist + w_cov * d_cov * rbar_cov
    e = (d_dist + d_cov) * g / (rms(g) + eps)
    sev = min(max(sev_tv * tv_s + sev_out * (1.0 - pC), 0.0), 1.0)
    return dict(d_dist=d_dist, d_cov=d_cov, tv_c=tv_c, tv_s=tv_s, severity=sev, p_C=pC, p_star=p_star,
                support=S, O=O, boundary=Bset, r_dist=r_dist, r_cov=r_cov, g=g, e=e)


def ema_update(m: np.ndarray, e: np.ndarray, rho: float) -> np.ndarray:
    """Eq. (ema)."""
    return rho * np.asarray(m, dtype=np.float64) + (1.0 - rho) * np.asarray(e, dtype=np.float64)


def reflex_feedback(p_rows: np.ndarray, p_row: np.ndarray, q_rows: np.ndarray, q_row: np.ndarray,
                    cand: np.ndarray, y_star: np.ndarray, traj: np.ndarray, horizon: np.ndarray, W: np.ndarray,
                    memory: np.ndarray, rho: Sequence[float], w_min: float = 0.03, rows=None, P=None,
                    rec_sketch=None, align=None, **kw):
    """Batched records with the library's layout: cand [R, max_cand] (-1 padded), horizon 1-based,
    memory [B, H, d]. Records are applied in order; a record whose (trajectory, horizon) slot was already
    used by an earlier record of the batch is skipped (applied = -1). ``rows`` restricts the computation
    to those records (the others are reported as None). With ``align`` [B, H, 4] (count, mean, M2 of the
    alignments, feedback count), an applied record adds one to the feedback count and, given P and the
    record's proposal-time memory sketch rec_sketch[r] (all zero = none), one alignment observation.
    Returns (new memory, list of dicts), or (new memory, list, new align) when ``align`` is given."""
    mem = np.array(memory, dtype=np.float64, copy=True)
    al = None if align is None else np.array(align, dtype=np.float64, copy=True)
    seen = set()
    out = []
    for r in range(cand.shape[0]):
        slot = (int(traj[r]), int(horizon[r]))
        if slot in seen:
            out.append(dict(applied=-1))
            continue
        seen.add(slot)
        if rows is not None and r not in rows:
            out.append(None)
            continue
        C = [int(c) for c in cand[r] if c >= 0]
        f = feedback(p_rows[int(p_row[r])], q_rows[int(q_row[r])], C, int(y_star[r]), W, **kw)
        f["applied"] = 1 if f["severity"] >= w_min else 0
        if f["applied"]:
            i, h = slot
            mem[i, h - 1] = ema_update(mem[i, h - 1], f["e"], rho[h - 1])
            if al is not None:
                al[i, h - 1, 3] += 1
                sr_ = None if rec_sketch is None else np.asarray(rec_sketch[r], dtype=np.float64)
                xi = None if P is None else sketch(f["e"], P)
                if sr_ is not None and np.any(sr_ != 0.0) and xi is not None:
                    f["alignment"] = float(sr_ @ xi)
                    al[i, h - 1, :3] = moments_update(tuple(al[i, h - 1, :3]), f["alignment"])
        out.append(f)
    return (mem, out) if al is None else (mem, out, al)


# ----------------------------------------------------------------------------- reliability gate
# Paper: Sec. 3.4, paragraphs "Reliability from delayed alignment" (Eq. (reliability-score)) and "Gated
# hidden-state correction" (Eq. (reflex-correction)); App. C, paragraph "Reflex configuration" and
# Tab. "reflex-hparams": rank-24 normalised random projections, exact online sample moments, minimum
# feedback counts (1, 2, 4), minimum alignment counts (6, 16, 48), correction intervals (1.0-2.5 %,
# 0.4-1.0 %, 0.25-0.6 %) of the head state's RMS, z_delta = 0.6.
#
# Readings taken here:
# * sketch(x) = P x / ||P x|| with the caller's projection P [r, d]; undefined (None) when P x = 0.
# * An alignment observation a = <s, sketch(e)> is taken when a record's feedback is applied, with s the
#   memory sketch stored when the record was proposed; none when either sketch is undefined.
# * Moments: count n, mean and M2 by the one-pass update; sample standard deviation sqrt(M2 / (n - 1)).
# * Rel = mean - z_delta * std / sqrt(n), defined for n >= 2.
# * The correction is applied iff n_fb >= n_fb_min, n >= n_align_min (and >= 2), Rel > 0 and
#   RMS(m) > m_floor; then alpha = a_min + (a_max - a_min) * min(Rel, 1) (the interval is spanned by
#   the reliability score), else alpha = 0.
# * Horizons past the listed ones reuse the last listed values.


def sketch(x: np.ndarray, P: np.ndarray):
    v = np.asarray(P, dtype=np.float64) @ np.asarray(x, dtype=np.float64)
    n = float(np.sqrt(np.sum(v * v)))
    return None if n == 0.0 else v / n


def moments_update(stats: Sequence[float], a: float):
    """One-pass (count, mean, M2) update with observation a."""
    n, mean, m2 = stats
    n1 = n + 1
    d = a - mean
    mean1 = mean + d / n1
    return (n1, mean1, m2 + d * (a - mean1))


def reliability(stats: Sequence[float], z_delta: float):
    n, mean, m2 = stats
    if n < 2:
        return None
    return mean - z_delta * np.sqrt(m2 / (n - 1)) / np.sqrt(n)


def correction(z: np.ndarray, m: np.ndarray, stats: Sequence[float], n_fb: int, a_min: float, a_max: float,
               n_fb_min: int, n_align_min: int, z_delta: float = 0.6, eps: float = 1e-6, m_floor: float = 1e-8):
    """Eq. (reflex-correction) for one (trajectory, horizon): returns (z + dz, alpha, Rel)."""
    z = np.asarray(z, dtype=np.float64)
    m = np.asarray(m, dtype=np.float64)
    rel = reliability(stats, z_delta)
    ok = (n_fb >= n_fb_min and stats[0] >= max(n_align_min, 2) and rel is not None and rel > 0.0
          and rms(m) > m_floor)
    if not ok:
        return z.copy(), 0.0, rel
    alpha = a_min + (a_max - a_min) * min(rel, 1.0)
    u = m / (rms(m) + eps)
    return z + alpha * rms(z) * u, alpha, rel
