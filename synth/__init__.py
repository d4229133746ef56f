"""Seeded synthetic workloads for the speculative verification step.

This module only draws inputs: shapes, value distributions, tree topologies,
paged-KV layouts and uniforms. It performs none of the method's arithmetic
(no normalisation, no head transform, no selection of draft tokens by the
heads, no attention, no acceptance). Both the CPU oracle (through the tests)
and the HIP path consume exactly the arrays produced here.

Every tensor is drawn from ``np.random.default_rng(SeedSequence([seed, cfg,
tensor_id, ...]))`` so that a tensor can be regenerated on its own.

bf16 tensors are returned as ``uint16`` bit patterns (round-to-nearest-even
from float32); ``bf16_bits_to_f32`` widens them exactly.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# tensor ids (fixed; changing one changes that tensor's stream only)
_TID = {
    "hidden": 1, "corr": 2, "active": 3, "A": 4, "bias": 5, "W": 6,
    "root": 7, "u_tree": 8,
    "q": 20, "kc": 21, "vc": 22, "kt": 23, "vt": 24, "ctx": 25, "perm": 26,
    "tlogits": 40, "dnoise": 41, "order": 42, "u_acc": 43, "u_fin": 44,
    "hlogits": 50,
    "ckc": 60, "cvc": 61, "ckt": 62, "cvt": 63, "cacc": 64, "cperm": 65,
    "rp": 70, "rq": 71, "rcand": 72, "rslot": 73, "rmem": 74, "ry": 75, "rW": 76,
    "gP": 80, "gmem": 81, "gsk": 82,
}


@dataclasses.dataclass(frozen=True)
class Config:
    """One workload shape. Field names follow the paper's notation."""
    name: str
    dtype: str                 # "f32" or "bf16"
    B: int                     # live trajectories
    T: int                     # tree nodes per trajectory, root included
    depth: int                 # maximum number of edges from the root
    Hq: int
    Hkv: int
    D: int                     # attention head dim
    d: int                     # hidden size
    H: int                     # future-token heads
    V: int                     # vocabulary
    ctx: Tuple                 # ("explicit", (L0, L1, ...)) | ("uniform", lo, hi) | ("lognormal", median, sigma, cap)
    parents: Optional[Tuple[int, ...]] = None   # explicit topology, else the level rule
    active_frac: float = 1.0   # fraction of trajectories with an active Reflex correction
    block_size: int = 16
    contiguous_pages: bool = False
    clip_norm: float = 1.0

    @property
    def max_ctx(self) -> int:
        kind = self.ctx[0]
        if kind == "explicit":
            return max(self.ctx[1])
        if kind == "uniform":
            return self.ctx[2]
        return self.ctx[3]

    @property
    def max_blocks(self) -> int:
        return max(1, -(-self.max_ctx // self.block_size))


_7B = dict(Hq=28, Hkv=4, D=128, d=3584, H=4, V=151936)

TINY_FP32 = Config("tiny-fp32", "f32", B=2, T=8, depth=3, Hq=4, Hkv=2, D=64, d=256, H=2, V=512,
                   ctx=("explicit", (100, 160)), parents=(-1, 0, 0, 1, 1, 2, 3, 4), contiguous_pages=True)
SHAPE_1P5B = Config("1.5B-shape", "bf16", B=64, T=16, depth=4, Hq=12, Hkv=2, D=128, d=1536, H=4,
                    V=151936, ctx=("uniform", 512, 4096))
SHAPE_7B = Config("7B-shape", "bf16", B=128, T=32, depth=5, ctx=("uniform", 1024, 8192), **_7B)
SHAPE_14B_TAIL = Config("14B-shape-tail", "bf16", B=8, T=64, depth=6, Hq=40, Hkv=8, D=128, d=5120, H=5,
                        V=151936, ctx=("uniform", 8192, 16384))
WORKLOADS: Dict[str, Config] = {c.name: c for c in (TINY_FP32, SHAPE_1P5B, SHAPE_7B, SHAPE_14B_TAIL)}

# Concurrency sweep at the 7B shape: live batch shrinks while the tree grows.
SWEEP_POINTS: List[Tuple[int, int]] = [(256, 8), (128, 12), (64, 16), (32, 24), (16, 32), (8, 64), (4, 96)]


def sweep_config(B: int, T: int) -> Config:
    return Config(f"7B-sweep-B{B}-T{T}", "bf16", B=B, T=T, depth=5,
                  ctx=("lognormal", 2048.0, 1.0, 16384), active_frac=0.5, **_7B)


def get_config(cfg) -> Config:
    if isinstance(cfg, Config):
        return cfg
    if isinstance(cfg, tuple):
        return sweep_config(*cfg)
    return WORKLOADS[cfg]


def scaled(cfg: Config, **over) -> Config:
    """A copy of ``cfg`` with some fields replaced (smaller parity cases)."""
    return dataclasses.replace(cfg, **over)


# ----------------------------------------------------------------------------- rng helpers

def _rng(seed: int, cfg_key, tid: str, *extra: int) -> np.random.Generator:
    key = [int(seed), _cfg_key(cfg_key), _TID[tid], *[int(e) for e in extra]]
    return np.random.default_rng(np.random.SeedSequence(key))


def _cfg_key(cfg: Config) -> int:
    # stable small integer derived from the shape, so scaled copies draw fresh streams
    h = 1000
    for v in (cfg.B, cfg.T, cfg.depth, cfg.Hq, cfg.Hkv, cfg.D, cfg.d, cfg.H, cfg.V):
        h = (h * 1000003 + int(v)) % (2 ** 31 - 1)
    return h


def normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    return (rng.standard_normal(shape, dtype=np.float32) * np.float32(std)).astype(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    out = ((u + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def as_dtype(x: np.ndarray, dtype: str) -> np.ndarray:
    """Store a float32 draw in the workload dtype (f32 array or bf16 bit patterns)."""
    return x.astype(np.float32) if dtype == "f32" else f32_to_bf16_bits(x)


def to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of a stored tensor to float64."""
    if dtype == "bf16" and x.dtype == np.uint16:
        return bf16_bits_to_f32(x).astype(np.float64)
    return np.asarray(x, dtype=np.float64)


def uniforms(rng: np.random.Generator, shape) -> np.ndarray:
    """U(0,1) values (2k+1)*2^-24, k uniform in [0, 2^23): exact in fp32, strictly inside (0,1)."""
    k = rng.integers(0, 2 ** 23, size=shape, dtype=np.int64)
    return ((2 * k + 1).astype(np.float64) * 2.0 ** -24).astype(np.float32)


# ----------------------------------------------------------------------------- topology

def level_sizes(T: int, depth: int) -> List[int]:
    """Nodes per level 1..depth: proportional to (depth-d+1), floored at 1, summing to T-1."""
    if T < 1:
        raise ValueError("T must be >= 1")
    n_spec = T - 1
    if n_spec == 0:
        return []
    depth = min(depth, n_spec)
    tot = depth * (depth + 1) // 2
    n = [max(1, (n_spec * (depth - d + 1)) // tot) for d in range(1, depth + 1)]
    s = sum(n)
    i = 0
    while s < n_spec:
        n[i % depth] += 1
        s += 1
        i += 1
    while s > n_spec:
        for j in range(depth - 1, -1, -1):
            if n[j] > 1:
                n[j] -= 1
                s -= 1
                break
    return n


def level_parents(T: int, depth: int) -> np.ndarray:
    """BFS-ordered parents array; child k of level d hangs under node floor(k*n_{d-1}/n_d) of level d-1."""
    sizes = level_sizes(T, depth)
    parents = [-1]
    prev_start, prev_n = 0, 1
    start = 1
    for n in sizes:
        for k in range(n):
            parents.append(prev_start + (k * prev_n) // n)
        prev_start, prev_n = start, n
        start += n
    out = np.asarray(parents, dtype=np.int32)
    assert out.shape[0] == T
    return out


def topology(cfg: Config) -> np.ndarray:
    p = np.asarray(cfg.parents, dtype=np.int32) if cfg.parents is not None else level_parents(cfg.T, cfg.depth)
    if p.shape[0] != cfg.T:
        raise ValueError("explicit parents do not match T")
    return p


def node_depths(parents: np.ndarray) -> np.ndarray:
    dep = np.zeros(parents.shape[0], dtype=np.int32)
    for c in range(1, parents.shape[0]):
        dep[c] = dep[parents[c]] + 1
    return dep


def max_children(parents: np.ndarray) -> int:
    if parents.shape[0] <= 1:
        return 0
    return int(np.bincount(parents[1:], minlength=parents.shape[0]).max())


# ----------------------------------------------------------------------------- workloads

def context_lengths(cfg: Config, seed: int = 0) -> np.ndarray:
    kind = cfg.ctx[0]
    if kind == "explicit":
        L = np.asarray(cfg.ctx[1], dtype=np.int32)
        assert L.shape[0] == cfg.B
        return L
    rng = _rng(seed, cfg, "ctx")
    if kind == "uniform":
        return rng.integers(cfg.ctx[1], cfg.ctx[2] + 1, size=cfg.B).astype(np.int32)
    med, sigma, cap = cfg.ctx[1], cfg.ctx[2], cfg.ctx[3]
    L = np.exp(np.log(med) + sigma * rng.standard_normal(cfg.B))
    return np.clip(np.rint(L), 1, cap).astype(np.int32)


def heads_inputs(cfg: Config, seed: int = 0, with_weights: bool = True) -> dict:
    """Inputs of the proposal step: hidden state, Reflex correction, head weights, tree topology, uniforms."""
    B, d, H, V, T = cfg.B, cfg.d, cfg.H, cfg.V, cfg.T
    out = dict(cfg=cfg, dtype=cfg.dtype)
    out["hidden"] = as_dtype(normal(_rng(seed, cfg, "hidden"), (B, d), 1.0), cfg.dtype)
    out["corr"] = normal(_rng(seed, cfg, "corr"), (B, d), 0.1)
    if cfg.active_frac >= 1.0:
        act = np.ones(B, dtype=np.uint8)
    else:
        act = (_rng(seed, cfg, "active").random(B) < cfg.active_frac).astype(np.uint8)
    out["active"] = act
    if with_weights:
        out["A"] = as_dtype(normal(_rng(seed, cfg, "A"), (H, d, d), 0.02), cfg.dtype)
        out["bias"] = as_dtype(normal(_rng(seed, cfg, "bias"), (H, d), 0.02), cfg.dtype)
        out["W"] = as_dtype(normal(_rng(seed, cfg, "W"), (V, d), 0.02), cfg.dtype)
    par = topology(cfg)
    out["parents"] = np.ascontiguousarray(np.broadcast_to(par, (B, T))).astype(np.int32)
    out["root_token"] = _rng(seed, cfg, "root").integers(0, V, size=B).astype(np.int32)
    out["u_tree"] = uniforms(_rng(seed, cfg, "u_tree"), (B, T))
    out["max_children"] = max_children(par)
    return out


def head_logits_inputs(cfg: Config, seed: int = 0, std: float = 1.5, tie_frac: float = 0.0) -> dict:
    """Inputs of the tree-build step on its own: fp32 head logits [B,H,V] plus topology and uniforms.

    ``tie_frac`` > 0 quantises that fraction of rows to a coarse grid so equal values occur.
    """
    B, H, V, T = cfg.B, cfg.H, cfg.V, cfg.T
    rng = _rng(seed, cfg, "hlogits")
    lg = normal(rng, (B, H, V), std)
    if tie_frac > 0:
        rows = rng.random((B, H)) < tie_frac
        lg[rows] = np.round(lg[rows] * 2.0) / 2.0
    par = topology(cfg)
    return dict(cfg=cfg, logits=lg,
                parents=np.ascontiguousarray(np.broadcast_to(par, (B, T))).astype(np.int32),
                root_token=_rng(seed, cfg, "root").integers(0, V, size=B).astype(np.int32),
                u_tree=uniforms(_rng(seed, cfg, "u_tree"), (B, T)),
                max_children=max_children(par))


def attn_inputs(cfg: Config, seed: int = 0, poison: bool = True) -> dict:
    """Inputs of the tree-verify attention: queries, paged prefix K/V, tree K/V, topology."""
    B, T, Hq, Hkv, D, bs = cfg.B, cfg.T, cfg.Hq, cfg.Hkv, cfg.D, cfg.block_size
    L = context_lengths(cfg, seed)
    nblk = -(-L // bs)
    num_blocks = max(1, int(nblk.sum()))
    max_blocks = cfg.max_blocks
    if (nblk > max_blocks).any():
        raise ValueError("context longer than max_blocks pages")
    if cfg.contiguous_pages:
        phys = np.arange(num_blocks, dtype=np.int32)
    else:
        phys = _rng(seed, cfg, "perm").permutation(num_blocks).astype(np.int32)
    table = np.full((B, max_blocks), -1, dtype=np.int32)
    off = 0
    for b in range(B):
        table[b, :nblk[b]] = phys[off:off + nblk[b]]
        off += nblk[b]
    kc = normal(_rng(seed, cfg, "kc"), (num_blocks, Hkv, bs, D), 1.0)
    vc = normal(_rng(seed, cfg, "vc"), (num_blocks, Hkv, bs, D), 1.0)
    if poison:
        # slots past the end of each trajectory's last page hold NaN: they must never be read
        for b in range(B):
            tail = L[b] % bs
            if nblk[b] > 0 and tail:
                blk = table[b, nblk[b] - 1]
                kc[blk, :, tail:, :] = np.nan
                vc[blk, :, tail:, :] = np.nan
    par = topology(cfg)
    return dict(
        cfg=cfg, dtype=cfg.dtype, ctx_len=L.astype(np.int32), block_table=table,
        num_blocks=num_blocks, max_blocks=max_blocks,
        q=as_dtype(normal(_rng(seed, cfg, "q"), (B, T, Hq, D), 1.0), cfg.dtype),
        k_cache=as_dtype(kc, cfg.dtype), v_cache=as_dtype(vc, cfg.dtype),
        k_tree=as_dtype(normal(_rng(seed, cfg, "kt"), (B, T, Hkv, D), 1.0), cfg.dtype),
        v_tree=as_dtype(normal(_rng(seed, cfg, "vt"), (B, T, Hkv, D), 1.0), cfg.dtype),
        parents=np.ascontiguousarray(np.broadcast_to(par, (B, T))).astype(np.int32),
        scale=1.0 / math.sqrt(D),
    )


def accept_inputs(cfg: Config, seed: int = 0, target_std: float = 4.0, noise_std: float = 1.0,
                  rows: Optional[Sequence[int]] = None) -> dict:
    """Inputs of the acceptance walk.

    Target logits ~ N(0, target_std) per node. A draft row per node is target + N(0, noise_std);
    the node's children take the draft row's largest entries as tokens in a random order (a
    permutation drawn here), and their draft values as ``child_logit``. Any ordered child list is
    a valid input to the walk; the draft law matters only for the exactness statistics, which
    build trees through the method's own tree builder instead.
    """
    B, T, V = cfg.B, cfg.T, cfg.V
    par = topology(cfg)
    kids = [[] for _ in range(T)]
    for c in range(1, T):
        kids[par[c]].append(c)
    tl = np.empty((B, T, V), dtype=np.float32)
    tokens = np.zeros((B, T), dtype=np.int32)
    child_logit = np.zeros((B, T), dtype=np.float32)
    root = _rng(seed, cfg, "root").integers(0, V, size=B).astype(np.int32)
    tokens[:, 0] = root
    rng_t = _rng(seed, cfg, "tlogits")
    for b in range(B):
        tl[b] = normal(rng_t, (T, V), target_std)
    tl_store = as_dtype(tl, cfg.dtype)
    del tl
    rng_n = _rng(seed, cfg, "dnoise")
    rng_o = _rng(seed, cfg, "order")
    for b in range(B):
        for u in range(T):
            m = len(kids[u])
            if m == 0:
                continue
            # children are picked from the stored (rounded) target values plus noise
            draft = to_f64(tl_store[b, u], cfg.dtype) + normal(rng_n, (V,), noise_std)
            top = np.argpartition(-draft, m - 1)[:m]
            perm = rng_o.permutation(m)
            for j, c in enumerate(kids[u]):
                tok = int(top[perm[j]])
                tokens[b, c] = tok
                child_logit[b, c] = np.float32(draft[tok])
    return dict(
        cfg=cfg, dtype=cfg.dtype, target_logits=tl_store, child_logit=child_logit, tokens=tokens,
        parents=np.ascontiguousarray(np.broadcast_to(par, (B, T))).astype(np.int32),
        u_acc=uniforms(_rng(seed, cfg, "u_acc"), (B, T)),
        u_fin=uniforms(_rng(seed, cfg, "u_fin"), (B,)),
        max_depth=int(node_depths(par).max()) if T > 1 else 0,
    )


def commit_inputs(cfg: Config, seed: int = 0, n_layers: int = 1, with_kv: bool = True) -> dict:
    """Inputs of the accepted-path cache extraction, stacked over ``n_layers`` layers.

    Each trajectory's page list has room for its prefix plus a full root path (depth + 1 rows).
    The accepted path is a random root path of a random target length 0..depth (at every step a
    uniformly chosen child among those whose subtree reaches that length, else among all children,
    stopping early at a leaf); out_len = 1 + its length. Cache slots past the prefix hold
    NaN, so a row that is not written stays visibly untouched. ``with_kv=False`` skips the cache and
    tree K/V draws (page lists, lengths and paths only).
    """
    B, T, Hkv, D, bs = cfg.B, cfg.T, cfg.Hkv, cfg.D, cfg.block_size
    par = topology(cfg)
    dep = node_depths(par)
    max_depth = int(dep.max()) if T > 1 else 0
    L = context_lengths(cfg, seed)
    nblk = -(-(L + max_depth + 1) // bs)
    num_blocks = int(nblk.sum())
    max_blocks = int(nblk.max())
    phys = (np.arange(num_blocks, dtype=np.int32) if cfg.contiguous_pages
            else _rng(seed, cfg, "cperm").permutation(num_blocks).astype(np.int32))
    table = np.full((B, max_blocks), -1, dtype=np.int32)
    off = 0
    for b in range(B):
        table[b, :nblk[b]] = phys[off:off + nblk[b]]
        off += nblk[b]
    if with_kv:
        kc = normal(_rng(seed, cfg, "ckc"), (n_layers, num_blocks, Hkv, bs, D), 1.0)
        vc = normal(_rng(seed, cfg, "cvc"), (n_layers, num_blocks, Hkv, bs, D), 1.0)
        for b in range(B):
            pos = np.arange(int(L[b]), int(nblk[b]) * bs)
            kc[:, table[b, pos // bs], :, pos % bs, :] = np.nan
            vc[:, table[b, pos // bs], :, pos % bs, :] = np.nan
    kids = [[] for _ in range(T)]
    for c in range(1, T):
        kids[par[c]].append(c)
    reach = dep.copy()                 # deepest depth inside each node's subtree
    for c in range(T - 1, 0, -1):
        reach[par[c]] = max(reach[par[c]], reach[c])
    rng = _rng(seed, cfg, "cacc")
    acc = np.full((B, max(1, max_depth)), -1, dtype=np.int32)
    out_len = np.empty(B, dtype=np.int32)
    for b in range(B):
        want = int(rng.integers(0, max_depth + 1))
        u, n = 0, 0
        while n < want and kids[u]:
            deep = [c for c in kids[u] if reach[c] >= want]
            pick = deep if deep else kids[u]
            u = pick[int(rng.integers(0, len(pick)))]
            acc[b, n] = u
            n += 1
        out_len[b] = n + 1
    out = dict(
        cfg=cfg, dtype=cfg.dtype, n_layers=n_layers, ctx_len=L.astype(np.int32), block_table=table,
        num_blocks=num_blocks, max_blocks=max_blocks, max_depth=max(1, max_depth),
        parents=np.ascontiguousarray(np.broadcast_to(par, (B, T))).astype(np.int32),
        acc_nodes=acc, out_len=out_len,
    )
    if with_kv:
        out.update(
            k_cache=as_dtype(kc, cfg.dtype), v_cache=as_dtype(vc, cfg.dtype),
            k_tree=as_dtype(normal(_rng(seed, cfg, "ckt"), (n_layers, B, T, Hkv, D), 1.0), cfg.dtype),
            v_tree=as_dtype(normal(_rng(seed, cfg, "cvt"), (n_layers, B, T, Hkv, D), 1.0), cfg.dtype))
    return out


def reflex_inputs(cfg: Config, seed: int = 0, R: Optional[int] = None, support: int = 48,
                  target_std: float = 4.0, boost: float = 8.0, with_W: bool = True) -> dict:
    """Matured proposal records for the Reflex feedback.

    One record per (trajectory, horizon) slot in a seeded order (the first R of them). Record r's
    candidate set has K_r = the tree's level size at depth h (capped at ``support``) distinct random
    tokens. Head logits ~ N(0, target_std) with the candidates raised by ``boost``; target logits
    ~ N(0, target_std) with a random half of the candidates and as many other random tokens raised by
    ``boost`` (so part of the target's important mass lies outside the candidates). The realised token is
    a random raised token. W ~ N(0, 0.02) as in the heads workload; memory ~ N(0, 0.1).
    """
    B, H, V, d = cfg.B, cfg.H, cfg.V, cfg.d
    sizes = level_sizes(cfg.T, cfg.depth) if cfg.T > 1 else [1]
    slots = [(i, h) for i in range(B) for h in range(1, H + 1)]
    order = _rng(seed, cfg, "rslot").permutation(len(slots))
    R = len(slots) if R is None else int(R)
    recs = [slots[int(j)] for j in order[:R]]
    K = [max(1, min(support, sizes[min(h, len(sizes)) - 1])) for (_, h) in recs]
    max_cand = max(K)
    rng_c, rng_y = _rng(seed, cfg, "rcand"), _rng(seed, cfg, "ry")
    rng_p, rng_q = _rng(seed, cfg, "rp"), _rng(seed, cfg, "rq")
    cand = np.full((R, max_cand), -1, dtype=np.int32)
    p = np.empty((R, V), dtype=np.float32)
    q = np.empty((R, V), dtype=np.float32)
    y = np.empty(R, dtype=np.int32)
    for r in range(R):
        k = K[r]
        ids = rng_c.choice(V, 2 * k, replace=False)
        c, other = ids[:k], ids[k:]
        cand[r, :k] = c
        q[r] = normal(rng_q, (V,), target_std)
        q[r, c] += boost
        p[r] = normal(rng_p, (V,), target_std)
        half = c[rng_c.permutation(k)[: max(1, k // 2)]]
        raised = np.concatenate([half, other])
        p[r, raised] += boost
        y[r] = int(raised[int(rng_y.integers(0, raised.shape[0]))])
    out = dict(cfg=cfg, dtype=cfg.dtype, R=R, support=support, p_logits=as_dtype(p, cfg.dtype), q_logits=q,
               p_row=np.arange(R, dtype=np.int32), q_row=np.arange(R, dtype=np.int32), cand=cand, y_star=y,
               traj=np.array([i for i, _ in recs], dtype=np.int32), horizon=np.array([h for _, h in recs], dtype=np.int32),
               memory=normal(_rng(seed, cfg, "rmem"), (B, H, d), 0.1))
    if with_W:
        out["W"] = as_dtype(normal(_rng(seed, cfg, "rW"), (V, d), 0.02), cfg.dtype)
    return out


def reflex_gate_inputs(cfg: Config, seed: int = 0, rank: int = 24) -> dict:
    """Reflex state for the gated correction: memory ~ N(0, 0.1) per (trajectory, head) (one row all zero),
    a projection P [rank, d] with unit rows, and alignment statistics (count, mean, M2, feedback count)
    cycling through five cases per (trajectory, head) slot: enough aligned evidence (gate open), too few
    observations, a negative mean, no feedback yet, and strong evidence (Rel near 1)."""
    B, H, d = cfg.B, cfg.H, cfg.d
    mem = normal(_rng(seed, cfg, "gmem"), (B, H, d), 0.1)
    mem[0, H - 1] = 0.0
    P = normal(_rng(seed, cfg, "gP"), (rank, d), 1.0)
    P /= np.sqrt((P.astype(np.float64) ** 2).sum(axis=1, keepdims=True)).astype(np.float32)
    cases = [(60, 0.5, 59 * 0.04, 10), (3, 0.5, 2 * 0.04, 10), (60, -0.1, 59 * 0.04, 10), (60, 0.5, 59 * 0.04, 0),
             (100, 0.95, 99 * 0.0025, 20)]
    align = np.array([cases[k % len(cases)] for k in range(B * H)], dtype=np.float32).reshape(B, H, 4)
    return dict(memory=mem, P=P.astype(np.float32), align=align)


def unit_sketches(n: int, rank: int, seed: int = 0, zero_every: int = 4) -> np.ndarray:
    """Stored memory sketches: random unit vectors, every ``zero_every``-th row all zero (no sketch)."""
    rng = np.random.default_rng(np.random.SeedSequence([int(seed), _TID["gsk"]]))
    s = rng.standard_normal((n, rank))
    s /= np.linalg.norm(s, axis=1, keepdims=True)
    s[::zero_every] = 0.0
    return s.astype(np.float32)
