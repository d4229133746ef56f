"""GPU parity of sr_tree_accept against the float64 oracle (App. B.2), plus exactness statistics of the
whole GPU proposal + acceptance path (App. B.3, Thm. "Exact target continuation")."""
import itertools

import numpy as np
import pytest
import torch
from scipy import stats

import oracle
import paper_2608_04962_amd as sr
import synth
from helpers import dev_tensor, f64

pytestmark = pytest.mark.gpu

MARGIN = 1e-6   # decisions closer than this to their threshold may legitimately differ


def _gpu_accept(inp, temperature=1.0, top_p=1.0):
    res = sr.tree_accept(dev_tensor(inp["target_logits"]), dev_tensor(inp["child_logit"]), dev_tensor(inp["tokens"]),
                         dev_tensor(inp["parents"]), dev_tensor(inp["u_acc"]), dev_tensor(inp["u_fin"]),
                         inp["max_depth"], temperature, top_p=top_p)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in res.items() if v is not None}


def _compare(inp, rows=None, temperature=1.0, top_p=1.0):
    cfg = inp["cfg"]
    print(f"[accept] {cfg.name} B={cfg.B} T={cfg.T} V={cfg.V} top_p={top_p}", flush=True)
    g = _gpu_accept(inp, temperature, top_p)
    rows = list(range(cfg.B)) if rows is None else [int(r) for r in rows]
    o = oracle.tree_accept(_Rows(inp["target_logits"], inp["dtype"]), inp["child_logit"], inp["tokens"],
                           inp["parents"], inp["u_acc"], inp["u_fin"], temperature, inp["max_depth"], rows=rows,
                           top_p=top_p)
    exempt = 0
    for b in rows:
        same = (np.array_equal(g["acc_nodes"][b], o["acc_nodes"][b])
                and np.array_equal(g["out_tokens"][b], o["out_tokens"][b])
                and g["out_len"][b] == o["out_len"][b] and g["final_kind"][b] == o["final_kind"][b])
        if not same:
            # only a near-threshold decision may differ
            assert min(o["min_margin"][b], g["min_margin"][b]) < MARGIN, (b, g["out_tokens"][b], o["out_tokens"][b])
            exempt += 1
        assert np.isfinite(g["min_margin"][b])
    print(f"[parity] accept {cfg.name} top_p={top_p}: {len(rows)} trajectories bit-exact except {exempt} "
          f"near-threshold (margin < {MARGIN})", flush=True)
    assert exempt <= max(1, len(rows) // 100), exempt
    return g, o


class _Rows:
    """float64 view of one trajectory's target logits at a time (bounds host memory at full size)."""

    def __init__(self, tl, dt):
        self.tl, self.dt = tl, dt

    def __getitem__(self, b):
        return f64(self.tl[b], self.dt)


def test_config0_parity():
    _compare(synth.accept_inputs(synth.TINY_FP32, seed=0))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_scaled_bf16_parity(seed):
    cfg = synth.scaled(synth.SHAPE_7B, B=48, V=4096)
    _compare(synth.accept_inputs(cfg, seed=seed))


def test_acceptance_happens_and_walks_deep():
    # drafts close to the target: most slots accept, walks reach the leaves
    cfg = synth.scaled(synth.SHAPE_1P5B, B=64, V=1024, dtype="f32")
    inp = synth.accept_inputs(cfg, seed=3, target_std=8.0, noise_std=0.05)
    g, _ = _compare(inp)
    assert (g["final_kind"] == 1).sum() > 0 and g["out_len"].mean() > 2.0


def test_temperature_power_of_two():
    cfg = synth.scaled(synth.SHAPE_7B, B=16, V=2048, dtype="f32")
    _compare(synth.accept_inputs(cfg, seed=4), temperature=0.5)


def test_single_node_tree_is_plain_sampling():
    cfg = synth.scaled(synth.TINY_FP32, T=1, parents=(-1,), B=8)
    g, o = _compare(synth.accept_inputs(cfg, seed=5))
    assert (g["out_len"] == 1).all() and (g["final_kind"] == 0).all()


def test_invalid_trajectories_are_flagged():
    cfg = synth.scaled(synth.TINY_FP32, B=4)
    inp = synth.accept_inputs(cfg, seed=6)
    inp["tokens"] = inp["tokens"].copy()
    inp["tokens"][1, 3] = cfg.V + 3            # token outside the vocabulary
    inp["tokens"][2, 2] = inp["tokens"][2, 1]  # duplicate sibling tokens
    inp["parents"] = inp["parents"].copy()
    inp["parents"][3, 4] = 6                   # not an earlier node
    g = _gpu_accept(inp)
    assert list(g["final_kind"][1:]) == [255, 255, 255]
    assert (g["out_len"][1:] == 0).all() and (g["out_tokens"][1:] == -1).all()
    assert g["final_kind"][0] in (0, 1)


@pytest.mark.parametrize("name,rseed", [("1.5B-shape", 1), ("7B-shape", 2), ("14B-shape-tail", 3)])
def test_full_size_sampled(name, rseed):
    cfg = synth.WORKLOADS[name]
    inp = synth.accept_inputs(cfg, seed=0)
    rows = np.random.default_rng(rseed).choice(cfg.B, size=min(8, cfg.B), replace=False)
    _compare(inp, rows=rows)


@pytest.mark.parametrize("point", synth.SWEEP_POINTS, ids=lambda p: f"B{p[0]}-T{p[1]}")
def test_sweep_points_sampled(point):
    # the concurrency sweep at full vocabulary: trees of 8 to 96 nodes (the 96-node root has 32 children)
    cfg = synth.sweep_config(*point)
    inp = synth.accept_inputs(cfg, seed=0)
    rows = np.random.default_rng(point[1]).choice(cfg.B, size=min(8, cfg.B), replace=False)
    _compare(inp, rows=rows)


@pytest.mark.parametrize("dt,top_p", [("bf16", 1.0), ("bf16", 0.95), ("f32", 1.0), ("f32", 0.95)])
def test_largest_vocabulary(dt, top_p):
    # V = 262144: 512 chunks of 512 tokens, the most a row may have; every trajectory compared
    cfg = synth.scaled(synth.SHAPE_7B, B=6, T=16, depth=4, V=262144, dtype=dt)
    _compare(synth.accept_inputs(cfg, seed=17), top_p=top_p)
    _compare(synth.accept_inputs(cfg, seed=18, target_std=8.0, noise_std=0.05), top_p=top_p)


def test_largest_tree():
    # SR_MAX_TREE = 128 nodes at depth 6 (the root has 43 children), every trajectory compared
    cfg = synth.scaled(synth.SHAPE_7B, B=24, T=128, depth=6, V=4096)
    _compare(synth.accept_inputs(cfg, seed=15))
    g, _ = _compare(synth.accept_inputs(cfg, seed=16, target_std=8.0, noise_std=0.05))
    assert g["out_len"].max() >= 3


def _peaked_inputs(B, V, seed, p_child=0.999, secondary=0):
    """Trajectories whose root target row puts mass ~p_child on the two drafted children, with slot uniforms above
    the acceptance ratios so both children are rejected: the fallback draws from the ~1 - p_child of mass outside
    the children, whose chunk sums must not be taken as differences of the large chunk sums holding the
    children. With ``secondary`` > 0 that many other tokens hold 90 % of the outside mass (so a nucleus cut can
    fall among them instead of among tail tokens of ~1e-8 mass each)."""
    rng = np.random.default_rng(seed)
    T = 3
    parents = np.tile(np.array([-1, 0, 0], dtype=np.int32), (B, 1))
    tl = (rng.standard_normal((B, T, V), dtype=np.float32) * 4.0).astype(np.float32)
    tokens = np.zeros((B, T), dtype=np.int32)
    child_logit = np.zeros((B, T), dtype=np.float32)
    u_acc = np.zeros((B, T), dtype=np.float32)
    for b in range(B):
        ids = rng.choice(V, size=2 + secondary, replace=False)
        ys, sec = ids[:2], ids[2:]
        tokens[b, 0] = int(rng.integers(V))
        tokens[b, 1:] = ys
        row = synth.to_f64(synth.as_dtype(tl[b, 0], "bf16"), "bf16")
        mx = row.max()
        w = np.exp(row - mx)
        w[ids] = 0.0
        s_out = w.sum()
        if secondary:
            share = 9.0 / secondary                      # each secondary token: 9/k of the tail's mass
            tl[b, 0, sec] = np.float32(mx + np.log(share * s_out))
            s_out *= 10.0
        # child masses: shares 0.8 and 0.2 of p_child (bf16 rounding of their logits moves them by < 7 %); the
        # first child's q is 0.95, so both slot ratios stay below 1
        mass = p_child / (1.0 - p_child) * s_out
        tl[b, 0, ys[0]] = np.float32(mx + np.log(0.8 * mass))
        tl[b, 0, ys[1]] = np.float32(mx + np.log(0.2 * mass))
        child_logit[b, 1] = np.float32(np.log(0.95))
        child_logit[b, 2] = np.float32(np.log(0.05))
        u_acc[b, 1:] = np.float32(1.0 - 2.0 ** -20)     # above every acceptance ratio below 1 - 1e-6
    u_fin = ((2 * rng.integers(0, 2 ** 23, size=B) + 1) * 2.0 ** -24).astype(np.float32)
    cfg = synth.scaled(synth.SHAPE_7B, B=B, T=T, depth=1, V=V)
    return dict(cfg=cfg, dtype="bf16", target_logits=synth.as_dtype(tl, "bf16"), child_logit=child_logit,
                tokens=tokens, parents=parents, u_acc=u_acc, u_fin=u_fin, max_depth=1)


@pytest.mark.parametrize("p_child", [0.999, 0.99999])
def test_peaked_rows_fallback_exact(p_child):
    inp = _peaked_inputs(64, 151936, seed=17, p_child=p_child)
    g, o = _compare(inp)
    assert (g["final_kind"] == 0).all() and (g["out_len"] == 1).all()
    _compare(inp, top_p=0.95)          # the nucleus is the two children: the second is accepted


def test_peaked_rows_nucleus_cut_outside_the_children():
    # children 0.999 of the mass, four secondary tokens 90 % of the rest: top_p 0.9995 keeps the children and
    # two or three secondary tokens, both children are rejected and the fallback draws among the kept ones
    inp = _peaked_inputs(64, 151936, seed=18, p_child=0.999, secondary=4)
    g, o = _compare(inp, top_p=0.9995)
    assert (g["final_kind"] == 0).all()
    _compare(inp)


def test_deterministic():
    cfg = synth.scaled(synth.SHAPE_7B, B=32, V=8192)
    inp = synth.accept_inputs(cfg, seed=7)
    a = _gpu_accept(inp)
    b = _gpu_accept(inp)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])


def test_nucleus_deterministic():
    # the cut's fixed-point histograms and the bin tallies (each cell written by the one wave owning its chunk)
    # give the same bits on every run, min_margin included; a flat row puts many tokens in the cut bin
    for kw in (dict(), dict(target_std=0.5)):
        inp = synth.accept_inputs(synth.scaled(synth.SHAPE_7B, B=24), seed=19, **kw)
        a = _gpu_accept(inp, top_p=0.95)
        b = _gpu_accept(inp, top_p=0.95)
        for k in a:
            np.testing.assert_array_equal(a[k].view(np.uint8), b[k].view(np.uint8), err_msg=k)


# ---------------------------------------------------------------- nucleus truncation
@pytest.mark.parametrize("top_p", [0.95, 0.5])
def test_nucleus_config0_and_scaled(top_p):
    _compare(synth.accept_inputs(synth.TINY_FP32, seed=10), top_p=top_p)
    _compare(synth.accept_inputs(synth.scaled(synth.SHAPE_7B, B=48, V=4096), seed=11), top_p=top_p)


def test_nucleus_deep_walks_and_temperature():
    cfg = synth.scaled(synth.SHAPE_1P5B, B=64, V=1024, dtype="f32")
    inp = synth.accept_inputs(cfg, seed=12, target_std=8.0, noise_std=0.05)
    g, _ = _compare(inp, top_p=0.9)
    assert (g["final_kind"] == 1).sum() > 0
    _compare(synth.accept_inputs(synth.scaled(synth.SHAPE_7B, B=16, V=2048), seed=13), temperature=0.5, top_p=0.95)


def test_nucleus_ties_cut_inside_equal_logits():
    """Rows whose logits take few distinct values (the cut falls among equal logits and is decided by id),
    a constant row and an all-negative row."""
    cfg = synth.scaled(synth.SHAPE_7B, B=24, V=4096)
    inp = synth.accept_inputs(cfg, seed=14)
    tl = synth.to_f64(inp["target_logits"], "bf16")
    tl = np.round(tl / 2.0) * 2.0                   # values on a coarse grid: heavy ties
    tl[0] = 0.0
    tl[1] = -np.abs(tl[1]) - 5.0
    inp["target_logits"] = synth.as_dtype(tl.astype(np.float32), "bf16")
    for top_p in (0.95, 0.37):
        _compare(inp, top_p=top_p)
    f32 = dict(inp, target_logits=tl.astype(np.float32), dtype="f32", cfg=synth.scaled(cfg, dtype="f32"))
    _compare(f32, top_p=0.6)


@pytest.mark.parametrize("name,rseed", [("7B-shape", 12), ("14B-shape-tail", 13)])
def test_nucleus_full_size_sampled(name, rseed):
    cfg = synth.WORKLOADS[name]
    inp = synth.accept_inputs(cfg, seed=1)
    rows = np.random.default_rng(rseed).choice(cfg.B, size=min(8, cfg.B), replace=False)
    _compare(inp, rows=rows, top_p=0.95)


# ---------------------------------------------------------------- exactness of the GPU path
@pytest.mark.parametrize("top_p", [1.0, 0.8])
def test_gpu_chi_square_exactness_1e6(top_p):
    """Tree build (sr_tree_build) + acceptance (sr_tree_accept), 1e6 independent trajectories with fresh
    uniforms: the first committed token must follow p_root and the first two tokens p(x1) p(x2|x1), where
    p is the (nucleus-truncated, for top_p < 1) target law."""
    V, H, N = 8, 2, 1_000_000
    parents = np.array([-1, 0, 0, 0, 1, 1, 2], dtype=np.int32)       # root 3 slots; node 1: 2; node 2: 1
    T = parents.shape[0]
    rng = np.random.default_rng(123)
    head = (rng.standard_normal((H, V)) * 1.2).astype(np.float32)
    # toy autoregressive target: logits of a node depend on its depth-1 token (the path)
    base = (rng.standard_normal(V) * 1.5).astype(np.float32)
    cond = (rng.standard_normal((V, V)) * 1.5).astype(np.float32)
    dev = "cuda"
    B = N
    logits = torch.from_numpy(np.broadcast_to(head, (B, H, V)).copy()).to(dev)
    par = torch.from_numpy(np.broadcast_to(parents, (B, T)).copy()).to(dev)
    root = torch.zeros(B, dtype=torch.int32, device=dev)
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    u_tree = torch.rand((B, T), generator=g, device=dev).clamp_(1e-7, 1 - 1e-7)
    tok, cl = sr.tree_build(logits, par, root, u_tree, max_children=3)
    # target logits per node: root -> base; depth-1 node with token a -> cond[a]; deeper nodes -> cond[a] too
    # (the toy target only looks at the first speculative token), so every node's row is a table lookup
    tokc = tok.long()
    first_tok = torch.zeros((B, T), dtype=torch.long, device=dev)
    anc1 = [0, 1, 2, 3, 1, 1, 2]                                        # depth-1 ancestor of each node (0 = root)
    for c in range(1, T):
        first_tok[:, c] = tokc[:, anc1[c]]
    condt = torch.from_numpy(cond).to(dev)
    tl = condt[first_tok]                                               # [B,T,V]
    tl[:, 0] = torch.from_numpy(base).to(dev)
    tl = tl.contiguous()
    u_acc = torch.rand((B, T), generator=g, device=dev).clamp_(1e-7, 1 - 1e-7)
    u_fin = torch.rand((B,), generator=g, device=dev).clamp_(1e-7, 1 - 1e-7)
    res = sr.tree_accept(tl, cl, tok, par, u_acc, u_fin, max_depth=2, top_p=top_p)
    out = res["out_tokens"].cpu().numpy()
    olen = res["out_len"].cpu().numpy()
    assert (res["final_kind"].cpu().numpy() != 255).all()
    p0, _ = oracle.accept._target_dist(base.astype(np.float64), 1.0, top_p)
    first = np.bincount(out[:, 0], minlength=V)
    assert (first[p0 == 0] == 0).all()
    keep = p0 > 0
    assert stats.chisquare(first[keep], p0[keep] * N).pvalue > 0.01
    # second token: where the round committed >= 2 tokens use it, else continue with a fresh draw from p(.|x1)
    pc = np.stack([oracle.accept._target_dist(cond[a].astype(np.float64), 1.0, top_p)[0] for a in range(V)])
    x1 = out[:, 0]
    x2 = out[:, 1].copy()
    need = olen < 2
    u2 = np.random.default_rng(9).random(need.sum())
    cdf = np.cumsum(pc[x1[need]], axis=1)
    x2[need] = (u2[:, None] * cdf[:, -1:] >= cdf).sum(1)
    joint = np.bincount(x1 * V + x2, minlength=V * V)
    exp = (p0[:, None] * pc).ravel()
    assert (joint[exp == 0] == 0).all()
    exp = exp / exp.sum() * N
    assert stats.chisquare(joint[exp > 0], exp[exp > 0]).pvalue > 0.01
