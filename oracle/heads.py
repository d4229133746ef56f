"""Future-token heads on the Reflex-corrected hidden state (oracle; test infrastructure only).

Paper: Sec. 3.2, Eq. (heads) -- head h maps the target's last hidden state to
z_h and proposes q_h = softmax(W z_h) through the target's shared vocabulary
projection W. App. C ("Future-token proposer") gives the head as one residual
block, g(h) = h + SiLU(A_h LN(h) + b_h).

Readings taken here (the paper leaves them open):
* One residual, z_h = x + SiLU(A_h LN(x) + b_h): the algorithm in App. C
  writes z = g(h) with g already residual; Eq. (heads) adds h a second time.
* LN is LayerNorm without affine parameters, biased variance, eps = 1e-5 (an
  affine LN folds into A_h and b_h).
* The Reflex correction enters as one bounded vector per trajectory added to
  the hidden state before the heads: x = h + Delta * min(1, c / ||Delta||_2)
  when the trajectory's correction is active, else x = h.
* Precision contract for bf16 workloads: LN(x) and z_h are rounded to bf16
  where the GPU feeds them to its matrix cores; all else stays float64.
"""
from __future__ import annotations

from typing import Callable, Optional

import numpy as np


def clip_correction(delta: np.ndarray, active: np.ndarray, clip_norm: float) -> np.ndarray:
    """Delta' = Delta * min(1, c / ||Delta||_2) on active rows, 0 on inactive rows; a zero row stays zero."""
    delta = np.asarray(delta, dtype=np.float64)
    out = np.zeros_like(delta)
    for b in range(delta.shape[0]):
        if not active[b]:
            continue
        nrm = float(np.sqrt(np.sum(delta[b] * delta[b])))
        if nrm == 0.0:
            continue
        out[b] = delta[b] * min(1.0, clip_norm / nrm)
    return out


def layer_norm(x: np.ndarray, eps: float) -> np.ndarray:
    """(x - mean) / sqrt(var + eps) over the last axis, biased variance, no affine."""
    mu = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def silu(a: np.ndarray) -> np.ndarray:
    return a / (1.0 + np.exp(-a))


def heads_forward(hidden: np.ndarray, corr: Optional[np.ndarray], active: Optional[np.ndarray],
                  A: np.ndarray, bias: np.ndarray, W: np.ndarray, clip_norm: float = 1.0,
                  ln_eps: float = 1e-5, round_fn: Optional[Callable] = None,
                  with_logits: bool = True) -> dict:
    """All heads for all trajectories.

    hidden [B,d], corr [B,d] (None = no correction), active [B] (None = all active),
    A [H,d,d] with A[h][out][in], bias [H,d], W [V,d] (row = token).
    Returns x [B,d], n [B,d], z [B,H,d] and logits [B,H,V] (float64); ``z_exact`` is z before its
    rounding point (equal to z when ``round_fn`` is None).
    """
    hidden = np.asarray(hidden, dtype=np.float64)
    B, d = hidden.shape
    H = A.shape[0]
    if corr is None:
        x = hidden.copy()
    else:
        act = np.ones(B, dtype=bool) if active is None else np.asarray(active).astype(bool)
        x = hidden + clip_correction(corr, act, clip_norm)
    n = layer_norm(x, ln_eps)
    if round_fn is not None:
        n = round_fn(n)
    z = np.empty((B, H, d), dtype=np.float64)
    z_exact = np.empty((B, H, d), dtype=np.float64)
    for h in range(H):
        a = n @ np.asarray(A[h], dtype=np.float64).T + np.asarray(bias[h], dtype=np.float64)
        zh = x + silu(a)
        z_exact[:, h, :] = zh
        z[:, h, :] = round_fn(zh) if round_fn is not None else zh
    out = dict(x=x, n=n, z=z, z_exact=z_exact)
    if with_logits:
        W64 = np.asarray(W, dtype=np.float64)
        out["logits"] = np.einsum("bhd,vd->bhv", z, W64, optimize=True)
    return out
