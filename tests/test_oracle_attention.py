"""Pins of the attention oracle (App. B.1, Eq. (nodep)): the tree-masked result at every node must equal
ordinary causal attention along that node's root path, computed here by torch's SDPA in float64."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth


def _causal_reference(inp, b, u, prefix_q_seed=0):
    """Causal SDPA over the token sequence prefix ++ path(u); returns the outputs at the path positions."""
    cfg = inp["cfg"]
    dt = cfg.dtype
    L = int(inp["ctx_len"][b])
    bs = cfg.block_size
    path = [u]
    while path[-1] != 0:
        path.append(int(inp["parents"][b][path[-1]]))
    path = path[::-1]
    kc = synth.to_f64(inp["k_cache"], dt)
    vc = synth.to_f64(inp["v_cache"], dt)
    pos = np.arange(L)
    kp = kc[inp["block_table"][b][pos // bs], :, pos % bs, :] if L else np.zeros((0, cfg.Hkv, cfg.D))
    vp = vc[inp["block_table"][b][pos // bs], :, pos % bs, :] if L else np.zeros((0, cfg.Hkv, cfg.D))
    K = np.concatenate([kp, synth.to_f64(inp["k_tree"], dt)[b, path]], 0)      # [S, Hkv, D]
    Vv = np.concatenate([vp, synth.to_f64(inp["v_tree"], dt)[b, path]], 0)
    # queries of the prefix positions are arbitrary (causality hides them from the path); the path
    # positions carry the nodes' queries
    qp = np.random.default_rng(prefix_q_seed).standard_normal((L, cfg.Hq, cfg.D))
    Q = np.concatenate([qp, synth.to_f64(inp["q"], dt)[b, path]], 0)           # [S, Hq, D]
    G = cfg.Hq // cfg.Hkv
    tq = torch.from_numpy(Q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    tv = torch.from_numpy(Vv).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    o = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True, scale=inp["scale"])
    s = (tq @ tk.transpose(-1, -2)) * inp["scale"]
    mask = torch.ones(s.shape[-2:], dtype=torch.bool).tril()
    lse = torch.logsumexp(s.masked_fill(~mask, -math.inf), dim=-1)
    return path, o[0].permute(1, 0, 2).numpy()[L:], lse[0].T.numpy()[L:]


def _check_all_nodes(inp):
    cfg = inp["cfg"]
    dt = cfg.dtype
    out, lse = oracle.tree_attention(synth.to_f64(inp["q"], dt), synth.to_f64(inp["k_cache"], dt),
                                     synth.to_f64(inp["v_cache"], dt), inp["block_table"], inp["ctx_len"],
                                     synth.to_f64(inp["k_tree"], dt), synth.to_f64(inp["v_tree"], dt),
                                     inp["parents"], inp["scale"], cfg.block_size)
    assert np.isfinite(out).all()
    for b in range(cfg.B):
        for u in range(cfg.T):
            path, ro, rl = _causal_reference(inp, b, u)
            # every node on u's path sits at its own causal position of the same sequence
            for i, w in enumerate(path):
                np.testing.assert_allclose(out[b, w], ro[i], rtol=1e-12, atol=1e-12)
                np.testing.assert_allclose(lse[b, w], rl[i], rtol=1e-12, atol=1e-12)


def test_masked_equals_per_path_causal_config0():
    _check_all_nodes(synth.attn_inputs(synth.TINY_FP32, seed=0))


def test_masked_equals_per_path_causal_scaled_bf16_paged():
    cfg = synth.scaled(synth.SHAPE_7B, B=3, T=12, depth=4, Hq=6, Hkv=2, D=32, ctx=("uniform", 1, 70))
    _check_all_nodes(synth.attn_inputs(cfg, seed=1))


def test_empty_prefix_and_single_node():
    cfg = synth.scaled(synth.TINY_FP32, ctx=("explicit", (0, 33)))
    _check_all_nodes(synth.attn_inputs(cfg, seed=2))
    cfg1 = synth.scaled(synth.TINY_FP32, T=1, parents=(-1,), ctx=("explicit", (17, 0)))
    inp = synth.attn_inputs(cfg1, seed=3)
    _check_all_nodes(inp)
    # T = 1 and L = 0: the root attends to itself only, so the output is its own value row
    out, lse = oracle.tree_attention(inp["q"], inp["k_cache"], inp["v_cache"], inp["block_table"], inp["ctx_len"],
                                     inp["k_tree"], inp["v_tree"], inp["parents"], inp["scale"])
    G = cfg1.Hq // cfg1.Hkv
    for h in range(cfg1.Hq):
        np.testing.assert_allclose(out[1, 0, h], inp["v_tree"][1, 0, h // G], rtol=1e-12)
        qk = inp["q"][1, 0, h].astype(np.float64) @ inp["k_tree"][1, 0, h // G].astype(np.float64)
        np.testing.assert_allclose(lse[1, 0, h], inp["scale"] * qk, rtol=1e-12)


def test_paging_is_transparent():
    # moving physical pages around (and rewriting the block table to match) must not change anything
    cfg = synth.scaled(synth.SHAPE_7B, B=2, T=4, depth=2, Hq=4, Hkv=2, D=16, ctx=("uniform", 20, 60),
                       dtype="f32")
    inp = synth.attn_inputs(cfg, seed=4)
    nb = inp["num_blocks"]
    pi = np.random.default_rng(9).permutation(nb)
    kc2 = np.empty_like(inp["k_cache"]); kc2[pi] = inp["k_cache"]
    vc2 = np.empty_like(inp["v_cache"]); vc2[pi] = inp["v_cache"]
    tab2 = np.where(inp["block_table"] >= 0, pi[np.maximum(inp["block_table"], 0)], -1)
    args = lambda kc, vc, tab: (inp["q"], kc, vc, tab, inp["ctx_len"], inp["k_tree"], inp["v_tree"],
                                inp["parents"], inp["scale"])
    o1, l1 = oracle.tree_attention(*args(inp["k_cache"], inp["v_cache"], inp["block_table"]))
    o2, l2 = oracle.tree_attention(*args(kc2, vc2, tab2))
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(l1, l2)
