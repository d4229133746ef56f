"""MI355X (gfx950) speculative verification step after SpecRoll (arXiv 2608.04962).

Thin torch-tensor binding over the C ABI of ``libspecroll.so`` (include/specroll.h):
argument marshalling only; every step runs in the HIP kernels. PyTorch supplies device
memory and the current stream.

    heads_propose     future-token heads + draft tree      (Sec. 3.2 Eq. (heads); App. B.1)
    tree_build        the tree-build half on given head logits
    tree_verify_attn  tree-masked attention over the paged prefix (App. B.1 Eq. (nodep))
    tree_accept       exact node-wise acceptance walk      (App. B.2)
    commit_path       accepted path's K/V appended to the paged cache, all layers in one launch
    tree_budget       per-response node budget and its tree (Sec. 3.2 Eq. (verification-budget),
                      Eq. (tree-budget)); host-only
    reflex_feedback   verifier feedback folded into the Reflex memory and its alignment statistics
                      (Sec. 3.3; Sec. 3.4)
    heads_propose_reflex  heads_propose with the gated Reflex correction of the head states
                      (Sec. 3.4 Eq. (reflex-correction))
"""
from __future__ import annotations

import ctypes as C
import math
from typing import Optional

import torch

from . import _lib
from ._lib import (AcceptDesc, AttnDesc, BudgetDesc, CommitDesc, HeadsDesc, ReflexDesc, ReflexGateDesc,  # noqa: F401
                   SpecRollError, check, lib)

__all__ = ["heads_propose", "tree_build", "tree_verify_attn", "tree_verify_attn_noalloc", "tree_accept", "commit_path", "tree_budget",
           "reflex_feedback", "heads_propose_reflex", "prof_begin", "prof_end",
           "kernel_names", "version", "SpecRollError", "library_path"]

_DT = {torch.float32: _lib.SR_F32, torch.bfloat16: _lib.SR_BF16}


def library_path() -> str:
    return _lib.LIB_PATH


def version() -> str:
    return lib().sr_version().decode()


def kernel_names():
    return lib().sr_kernel_names().decode().split(";")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(device) -> C.c_void_p:
    return C.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need(t, name, dtype, shape, device):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _workspace(nbytes: int, device, workspace: Optional[torch.Tensor]):
    if nbytes == 0:
        return None, 0
    if workspace is not None:
        if workspace.numel() * workspace.element_size() < nbytes:
            raise ValueError(f"workspace holds {workspace.numel() * workspace.element_size()} bytes, {nbytes} needed")
        return workspace, workspace.numel() * workspace.element_size()
    ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return ws, nbytes


def heads_workspace_bytes(B, d, H, V, T, max_children, dtype=torch.bfloat16) -> int:
    desc = HeadsDesc(B, d, H, V, T, max_children, _DT[dtype], 1.0, 1e-5)
    return int(lib().sr_heads_propose_workspace(C.byref(desc)))


def heads_propose(hidden, corr, corr_active, A, bias, W, parents, root_token, u_tree, max_children: int,
                  clip_norm: float = 1.0, ln_eps: float = 1e-5, logits: Optional[torch.Tensor] = None,
                  z: Optional[torch.Tensor] = None, tokens: Optional[torch.Tensor] = None,
                  child_logit: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
    """Heads on the corrected hidden state, shared-vocabulary logits and the draft tree.

    hidden [B,d] bf16|f32, corr [B,d] f32 or None, corr_active [B] uint8 or None, A [H,d,d],
    bias [H,d], W [V,d] (same dtype as hidden), parents [B,T] int32, root_token [B] int32,
    u_tree [B,T] f32. ``logits`` [B,H,V] f32 and ``z`` [B,H,d] are optional outputs.
    Returns (tokens [B,T] int32, child_logit [B,T] f32).
    """
    dev = hidden.device
    B, d = hidden.shape
    H = A.shape[0]
    V = W.shape[0]
    T = parents.shape[1]
    dt = hidden.dtype
    _need(hidden, "hidden", None, (B, d), dev)
    if dt not in _DT:
        raise TypeError("hidden must be float32 or bfloat16")
    if corr is not None:
        _need(corr, "corr", torch.float32, (B, d), dev)
    if corr_active is not None:
        _need(corr_active, "corr_active", torch.uint8, (B,), dev)
    _need(A, "A", dt, (H, d, d), dev)
    _need(bias, "bias", dt, (H, d), dev)
    _need(W, "W", dt, (V, d), dev)
    _need(parents, "parents", torch.int32, (B, T), dev)
    _need(root_token, "root_token", torch.int32, (B,), dev)
    _need(u_tree, "u_tree", torch.float32, (B, T), dev)
    if logits is not None:
        _need(logits, "logits", torch.float32, (B, H, V), dev)
    if z is not None:
        _need(z, "z", dt, (B, H, d), dev)
    tokens = torch.empty((B, T), dtype=torch.int32, device=dev) if tokens is None else tokens
    child_logit = torch.empty((B, T), dtype=torch.float32, device=dev) if child_logit is None else child_logit
    _need(tokens, "tokens", torch.int32, (B, T), dev)
    _need(child_logit, "child_logit", torch.float32, (B, T), dev)
    desc = HeadsDesc(B, d, H, V, T, int(max_children), _DT[dt], float(clip_norm), float(ln_eps))
    ws, wsb = _workspace(int(lib().sr_heads_propose_workspace(C.byref(desc))), dev, workspace)
    st = lib().sr_heads_propose(C.byref(desc), _ptr(hidden), _ptr(corr), _ptr(corr_active), _ptr(A), _ptr(bias),
                                _ptr(W), _ptr(parents), _ptr(root_token), _ptr(u_tree), _ptr(logits), _ptr(z),
                                _ptr(tokens), _ptr(child_logit), _ptr(ws), wsb, _stream(dev))
    check(st, "sr_heads_propose")
    return tokens, child_logit


def tree_build(logits, parents, root_token, u_tree, max_children: int, tokens=None, child_logit=None,
               workspace=None):
    """Draft tree from fp32 head logits [B,H,V]. Returns (tokens, child_logit)."""
    dev = logits.device
    B, H, V = logits.shape
    T = parents.shape[1]
    _need(logits, "logits", torch.float32, (B, H, V), dev)
    _need(parents, "parents", torch.int32, (B, T), dev)
    _need(root_token, "root_token", torch.int32, (B,), dev)
    _need(u_tree, "u_tree", torch.float32, (B, T), dev)
    tokens = torch.empty((B, T), dtype=torch.int32, device=dev) if tokens is None else tokens
    child_logit = torch.empty((B, T), dtype=torch.float32, device=dev) if child_logit is None else child_logit
    desc = HeadsDesc(B, 0, H, V, T, int(max_children), _lib.SR_F32, 1.0, 0.0)
    ws, wsb = _workspace(int(lib().sr_tree_build_workspace(C.byref(desc))), dev, workspace)
    st = lib().sr_tree_build(C.byref(desc), _ptr(logits), _ptr(parents), _ptr(root_token), _ptr(u_tree),
                             _ptr(tokens), _ptr(child_logit), _ptr(ws), wsb, _stream(dev))
    check(st, "sr_tree_build")
    return tokens, child_logit


def attn_desc(q, k_cache, block_table, scale=None) -> AttnDesc:
    B, T, Hq, D = q.shape
    NB, Hkv, bs, D2 = k_cache.shape
    return AttnDesc(B, T, Hq, Hkv, D, bs, block_table.shape[1], NB, _DT[q.dtype],
                    float(1.0 / math.sqrt(D) if scale is None else scale))


def attn_workspace_bytes(desc: AttnDesc) -> int:
    return int(lib().sr_tree_verify_attn_workspace(C.byref(desc)))


def tree_verify_attn(q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, parents, scale=None,
                     out=None, lse=None, want_lse: bool = True, workspace=None):
    """Tree-masked attention. q [B,T,Hq,D], caches [NB,Hkv,16,D], block_table [B,max_blocks] int32,
    ctx_len [B] int32, k_tree/v_tree [B,T,Hkv,D], parents [B,T] int32. Returns (out fp32, lse fp32 or None)."""
    dev = q.device
    B, T, Hq, D = q.shape
    NB, Hkv, bs, _ = k_cache.shape
    dt = q.dtype
    _need(q, "q", None, (B, T, Hq, D), dev)
    if dt not in _DT:
        raise TypeError("q must be float32 or bfloat16")
    _need(k_cache, "k_cache", dt, (NB, Hkv, bs, D), dev)
    _need(v_cache, "v_cache", dt, (NB, Hkv, bs, D), dev)
    _need(block_table, "block_table", torch.int32, (B, block_table.shape[1]), dev)
    _need(ctx_len, "ctx_len", torch.int32, (B,), dev)
    _need(k_tree, "k_tree", dt, (B, T, Hkv, D), dev)
    _need(v_tree, "v_tree", dt, (B, T, Hkv, D), dev)
    _need(parents, "parents", torch.int32, (B, T), dev)
    out = torch.empty((B, T, Hq, D), dtype=torch.float32, device=dev) if out is None else out
    _need(out, "out", torch.float32, (B, T, Hq, D), dev)
    if want_lse and lse is None:
        lse = torch.empty((B, T, Hq), dtype=torch.float32, device=dev)
    desc = attn_desc(q, k_cache, block_table, scale)
    ws, wsb = _workspace(attn_workspace_bytes(desc), dev, workspace)
    st = lib().sr_tree_verify_attn(C.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                                   _ptr(ctx_len), _ptr(k_tree), _ptr(v_tree), _ptr(parents), _ptr(out),
                                   _ptr(lse), _ptr(ws), wsb, _stream(dev))
    check(st, "sr_tree_verify_attn")
    return out, lse


def tree_verify_attn_noalloc(q, k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, parents, scale=None,
                             out=None, lse=None, want_lse: bool = True):
    """tree_verify_attn through sr_tree_verify_attn_noalloc: no workspace; the library's per-GPU scratch array
    holds the partial results (calls overlapping on one GPU race). Outputs as tree_verify_attn."""
    dev = q.device
    B, T, Hq, D = q.shape
    NB, Hkv, bs, _ = k_cache.shape
    dt = q.dtype
    _need(q, "q", None, (B, T, Hq, D), dev)
    if dt not in _DT:
        raise TypeError("q must be float32 or bfloat16")
    _need(k_cache, "k_cache", dt, (NB, Hkv, bs, D), dev)
    _need(v_cache, "v_cache", dt, (NB, Hkv, bs, D), dev)
    _need(block_table, "block_table", torch.int32, (B, block_table.shape[1]), dev)
    _need(ctx_len, "ctx_len", torch.int32, (B,), dev)
    _need(k_tree, "k_tree", dt, (B, T, Hkv, D), dev)
    _need(v_tree, "v_tree", dt, (B, T, Hkv, D), dev)
    _need(parents, "parents", torch.int32, (B, T), dev)
    out = torch.empty((B, T, Hq, D), dtype=torch.float32, device=dev) if out is None else out
    _need(out, "out", torch.float32, (B, T, Hq, D), dev)
    if want_lse and lse is None:
        lse = torch.empty((B, T, Hq), dtype=torch.float32, device=dev)
    desc = attn_desc(q, k_cache, block_table, scale)
    with torch.cuda.device(dev):
        st = lib().sr_tree_verify_attn_noalloc(C.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                               _ptr(block_table), _ptr(ctx_len), _ptr(k_tree), _ptr(v_tree),
                                               _ptr(parents), _ptr(out), _ptr(lse), _stream(dev))
    check(st, "sr_tree_verify_attn_noalloc")
    return out, lse


def tree_accept(target_logits, child_logit, tokens, parents, u_acc, u_fin, max_depth: int,
                temperature: float = 1.0, outputs: Optional[dict] = None, want_margin: bool = True,
                top_p: float = 1.0):
    """Exact acceptance walk. target_logits [B,T,V] bf16|f32; child_logit [B,T] f32; tokens, parents [B,T]
    int32; u_acc [B,T] f32; u_fin [B] f32; top_p < 1 cuts every target row to its nucleus.
    Returns dict(acc_nodes, out_tokens, out_len, final_kind, min_margin)."""
    dev = target_logits.device
    B, T, V = target_logits.shape
    dt = target_logits.dtype
    if dt not in _DT:
        raise TypeError("target_logits must be float32 or bfloat16")
    _need(target_logits, "target_logits", dt, (B, T, V), dev)
    _need(child_logit, "child_logit", torch.float32, (B, T), dev)
    _need(tokens, "tokens", torch.int32, (B, T), dev)
    _need(parents, "parents", torch.int32, (B, T), dev)
    _need(u_acc, "u_acc", torch.float32, (B, T), dev)
    _need(u_fin, "u_fin", torch.float32, (B,), dev)
    if outputs is None:
        outputs = dict(
            acc_nodes=torch.empty((B, max(max_depth, 1)), dtype=torch.int32, device=dev),
            out_tokens=torch.empty((B, max_depth + 1), dtype=torch.int32, device=dev),
            out_len=torch.empty((B,), dtype=torch.int32, device=dev),
            final_kind=torch.empty((B,), dtype=torch.uint8, device=dev),
            min_margin=torch.empty((B,), dtype=torch.float32, device=dev) if want_margin else None,
        )
    desc = AcceptDesc(B, T, V, int(max_depth), _DT[dt], float(temperature), float(top_p))
    st = lib().sr_tree_accept(C.byref(desc), _ptr(target_logits), _ptr(child_logit), _ptr(tokens), _ptr(parents),
                              _ptr(u_acc), _ptr(u_fin), _ptr(outputs["acc_nodes"]), _ptr(outputs["out_tokens"]),
                              _ptr(outputs["out_len"]), _ptr(outputs["final_kind"]), _ptr(outputs["min_margin"]),
                              None, 0, _stream(dev))
    check(st, "sr_tree_accept")
    if max_depth == 0:
        outputs["acc_nodes"] = outputs["acc_nodes"][:, :0]
    return outputs


def tree_budget(live: int, c_peak: int = 512, n_min: int = 1, n_max: int = 10, alloc=(5, 4, 0)):
    """Host rule of the node budget. Returns (N_t, per-horizon node counts, parents list of the tree)."""
    al = (C.c_int32 * max(1, len(alloc)))(*[int(a) for a in alloc])
    desc = BudgetDesc(int(c_peak), int(n_min), int(n_max), len(alloc), al)
    cap = max(int(n_max), 1)
    par = (C.c_int32 * cap)()
    cnt = (C.c_int32 * max(1, len(alloc)))()
    n_t, n_nodes = C.c_int32(), C.c_int32()
    check(lib().sr_tree_budget(C.byref(desc), int(live), C.byref(n_t), cnt, par, cap, C.byref(n_nodes)),
          "sr_tree_budget")
    counts = [int(cnt[h]) for h in range(len(alloc))]
    while counts and counts[-1] == 0:
        counts.pop()
    return int(n_t.value), counts, [int(par[i]) for i in range(n_nodes.value)]


def commit_path(k_cache, v_cache, block_table, ctx_len, k_tree, v_tree, acc_nodes, out_len, parents=None,
                new_ctx_len=None):
    """Append the root and accepted nodes' K/V rows to the paged caches (in place).

    k_cache/v_cache [n_layers,NB,Hkv,bs,D] (or [NB,Hkv,bs,D] for one layer), k_tree/v_tree
    [n_layers,B,T,Hkv,D] (or [B,T,Hkv,D]), block_table [B,max_blocks] int32, ctx_len [B] int32,
    acc_nodes [B,max_depth] int32, out_len [B] int32, parents [B,T] int32 or None.
    Returns new_ctx_len [B] int32 (-1 for a rejected trajectory)."""
    dev = k_cache.device
    one = k_cache.dim() == 4
    kc = k_cache.unsqueeze(0) if one else k_cache
    kt = k_tree.unsqueeze(0) if one else k_tree
    nl, NB, Hkv, bs, D = kc.shape
    _, B, T, _, _ = kt.shape
    dt = k_cache.dtype
    if dt not in _DT:
        raise TypeError("caches must be float32 or bfloat16")
    _need(k_cache, "k_cache", dt, tuple(k_cache.shape), dev)
    _need(v_cache, "v_cache", dt, tuple(k_cache.shape), dev)
    _need(k_tree, "k_tree", dt, ((B, T, Hkv, D) if one else (nl, B, T, Hkv, D)), dev)
    _need(v_tree, "v_tree", dt, tuple(k_tree.shape), dev)
    _need(block_table, "block_table", torch.int32, (B, block_table.shape[1]), dev)
    _need(ctx_len, "ctx_len", torch.int32, (B,), dev)
    _need(out_len, "out_len", torch.int32, (B,), dev)
    max_depth = int(acc_nodes.shape[1])
    _need(acc_nodes, "acc_nodes", torch.int32, (B, max_depth), dev)
    if parents is not None:
        _need(parents, "parents", torch.int32, (B, T), dev)
    if new_ctx_len is None:
        new_ctx_len = torch.empty((B,), dtype=torch.int32, device=dev)
    _need(new_ctx_len, "new_ctx_len", torch.int32, (B,), dev)
    desc = CommitDesc(nl, B, T, Hkv, D, bs, block_table.shape[1], NB, max_depth, _DT[dt])
    st = lib().sr_commit_path(C.byref(desc), _ptr(acc_nodes), _ptr(out_len), _ptr(parents), _ptr(k_tree),
                              _ptr(v_tree), _ptr(block_table), _ptr(ctx_len), _ptr(k_cache), _ptr(v_cache),
                              _ptr(new_ctx_len), _stream(dev))
    check(st, "sr_commit_path")
    return new_ctx_len


REFLEX_DEFAULTS = dict(temperature=1.0, support=48, w_dist=0.15, w_cov=1.25, sev_tv=0.3, sev_out=0.7, w_min=0.03,
                       eps=1e-6, n_boundary=4)
REFLEX_RHO = (0.85, 0.90, 0.95)


def reflex_feedback(target_logits, p_row, head_logits, q_row, cand, y_star, traj, horizon, W, memory, rho=None,
                    stats=None, e_out=None, want_e: bool = False, P=None, rec_sketch=None, align=None, **params):
    """Fold matured records' verifier feedback into the Reflex memory (in place).

    target_logits [Np,V] bf16|f32, p_row [R] int32, head_logits [Nq,V] f32, q_row [R] int32,
    cand [R,max_cand] int32 (-1 padded), y_star/traj/horizon [R] int32 (horizon 1-based),
    W [V,d] bf16|f32, memory [B,H,d] f32. ``rho`` defaults to the paper's (.85, .90, .95), the last value
    repeated for further horizons. With ``align`` [B,H,4] f32 (in place) the applied records update the
    alignment moments, given the sketch projection P [r,d] f32 and the records' stored memory sketches
    rec_sketch [R,r] f32. Returns (stats [R,8] f32, e [R,d] f32 or None)."""
    dev = target_logits.device
    Np, V = target_logits.shape
    Nq = head_logits.shape[0]
    R, MC = cand.shape
    Bm, Hm, d = memory.shape
    if target_logits.dtype not in _DT or W.dtype not in _DT:
        raise TypeError("target_logits and W must be float32 or bfloat16")
    _need(target_logits, "target_logits", None, (Np, V), dev)
    _need(head_logits, "head_logits", torch.float32, (Nq, V), dev)
    for t, n in ((p_row, "p_row"), (q_row, "q_row"), (y_star, "y_star"), (traj, "traj"), (horizon, "horizon")):
        _need(t, n, torch.int32, (R,), dev)
    _need(cand, "cand", torch.int32, (R, MC), dev)
    _need(W, "W", None, (V, d), dev)
    _need(memory, "memory", torch.float32, (Bm, Hm, d), dev)
    p = dict(REFLEX_DEFAULTS)
    p.update(params)
    rho = list(REFLEX_RHO if rho is None else rho)
    rho = (rho + [rho[-1]] * 8)[:8]
    if stats is None:
        stats = torch.empty((R, 8), dtype=torch.float32, device=dev)
    _need(stats, "stats", torch.float32, (R, 8), dev)
    if want_e and e_out is None:
        e_out = torch.empty((R, d), dtype=torch.float32, device=dev)
    if e_out is not None:
        _need(e_out, "e_out", torch.float32, (R, d), dev)
    rank = 0
    if P is not None:
        rank = P.shape[0]
        _need(P, "P", torch.float32, (rank, d), dev)
        if rec_sketch is not None:
            _need(rec_sketch, "rec_sketch", torch.float32, (R, rank), dev)
    if align is not None:
        _need(align, "align", torch.float32, (Bm, Hm, 4), dev)
    desc = ReflexDesc(R, V, d, Bm, Hm, Np, Nq, MC, int(p["support"]), int(p["n_boundary"]),
                      _DT[target_logits.dtype], _DT[W.dtype], float(p["temperature"]), float(p["w_dist"]),
                      float(p["w_cov"]), float(p["sev_tv"]), float(p["sev_out"]), float(p["w_min"]), float(p["eps"]),
                      (C.c_float * 8)(*rho), rank)
    st = lib().sr_reflex_feedback(C.byref(desc), _ptr(target_logits), _ptr(p_row), _ptr(head_logits), _ptr(q_row),
                                  _ptr(cand), _ptr(y_star), _ptr(traj), _ptr(horizon), _ptr(W), _ptr(memory),
                                  _ptr(stats), _ptr(e_out), _ptr(P), _ptr(rec_sketch), _ptr(align), _stream(dev))
    check(st, "sr_reflex_feedback")
    return stats, e_out


GATE_DEFAULTS = dict(z_delta=0.6, eps=1e-6, m_floor=1e-8, alpha_min=(0.010, 0.004, 0.0025),
                     alpha_max=(0.025, 0.010, 0.006), n_fb_min=(1, 2, 4), n_align_min=(6, 16, 48))


def _per_head(v, H):
    v = list(v)
    return (v + [v[-1]] * 8)[:8]


def reflex_gate_desc(rank: int = 0, **params) -> ReflexGateDesc:
    """Gate parameters (the paper's by default); per-head lists are extended with their last value."""
    p = dict(GATE_DEFAULTS)
    p.update(params)
    return ReflexGateDesc(int(rank), float(p["z_delta"]), float(p["eps"]), float(p["m_floor"]),
                          (C.c_float * 8)(*_per_head(p["alpha_min"], 8)), (C.c_float * 8)(*_per_head(p["alpha_max"], 8)),
                          (C.c_int32 * 8)(*_per_head(p["n_fb_min"], 8)), (C.c_int32 * 8)(*_per_head(p["n_align_min"], 8)))


def heads_propose_reflex(hidden, corr, corr_active, A, bias, W, parents, root_token, u_tree, max_children: int,
                         memory, align, P=None, clip_norm: float = 1.0, ln_eps: float = 1e-5,
                         logits: Optional[torch.Tensor] = None, z: Optional[torch.Tensor] = None,
                         tokens: Optional[torch.Tensor] = None, child_logit: Optional[torch.Tensor] = None,
                         sketch_out: Optional[torch.Tensor] = None, alpha_out: Optional[torch.Tensor] = None,
                         workspace: Optional[torch.Tensor] = None, **gate):
    """heads_propose with the gated Reflex correction of the head states. memory [B,H,d] f32,
    align [B,H,4] f32, P [r,d] f32 or None; sketch_out [B,H,r] and alpha_out [B,H] are optional outputs.
    Returns (tokens, child_logit)."""
    dev = hidden.device
    B, d = hidden.shape
    H = A.shape[0]
    V = W.shape[0]
    T = parents.shape[1]
    dt = hidden.dtype
    if dt not in _DT:
        raise TypeError("hidden must be float32 or bfloat16")
    _need(hidden, "hidden", None, (B, d), dev)
    _need(A, "A", dt, (H, d, d), dev)
    _need(bias, "bias", dt, (H, d), dev)
    _need(W, "W", dt, (V, d), dev)
    _need(parents, "parents", torch.int32, (B, T), dev)
    _need(root_token, "root_token", torch.int32, (B,), dev)
    _need(u_tree, "u_tree", torch.float32, (B, T), dev)
    _need(memory, "memory", torch.float32, (B, H, d), dev)
    _need(align, "align", torch.float32, (B, H, 4), dev)
    if corr is not None:
        _need(corr, "corr", torch.float32, (B, d), dev)
    if corr_active is not None:
        _need(corr_active, "corr_active", torch.uint8, (B,), dev)
    rank = 0
    if P is not None:
        rank = P.shape[0]
        _need(P, "P", torch.float32, (rank, d), dev)
    if logits is not None:
        _need(logits, "logits", torch.float32, (B, H, V), dev)
    if z is not None:
        _need(z, "z", dt, (B, H, d), dev)
    if sketch_out is not None:
        _need(sketch_out, "sketch_out", torch.float32, (B, H, rank), dev)
    if alpha_out is not None:
        _need(alpha_out, "alpha_out", torch.float32, (B, H), dev)
    tokens = torch.empty((B, T), dtype=torch.int32, device=dev) if tokens is None else tokens
    child_logit = torch.empty((B, T), dtype=torch.float32, device=dev) if child_logit is None else child_logit
    desc = HeadsDesc(B, d, H, V, T, int(max_children), _DT[dt], float(clip_norm), float(ln_eps))
    gdesc = reflex_gate_desc(rank, **gate)
    ws, wsb = _workspace(int(lib().sr_heads_propose_workspace(C.byref(desc))), dev, workspace)
    st = lib().sr_heads_propose_reflex(C.byref(desc), C.byref(gdesc), _ptr(hidden), _ptr(corr), _ptr(corr_active),
                                       _ptr(A), _ptr(bias), _ptr(W), _ptr(parents), _ptr(root_token), _ptr(u_tree),
                                       _ptr(memory), _ptr(align), _ptr(P), _ptr(logits), _ptr(z), _ptr(tokens),
                                       _ptr(child_logit), _ptr(sketch_out), _ptr(alpha_out), _ptr(ws), wsb,
                                       _stream(dev))
    check(st, "sr_heads_propose_reflex")
    return tokens, child_logit


def prof_begin(kernel_substr: str) -> None:
    check(lib().sr_prof_begin(kernel_substr.encode()), "sr_prof_begin")


def prof_end():
    """Returns (total_ms, launches) of the kernel selected by prof_begin."""
    ms = C.c_double()
    n = C.c_int32()
    check(lib().sr_prof_end(C.byref(ms), C.byref(n)), "sr_prof_end")
    return ms.value, n.value
