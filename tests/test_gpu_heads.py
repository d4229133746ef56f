"""GPU parity of sr_heads_propose / sr_tree_build against the float64 oracle
(Sec. 3.2 Eq. (heads); App. C future-token proposer; App. B.1 Eq. (slotq))."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_04962_amd as sr
import synth
from helpers import assert_z_bf16, dev_tensor, f64, row_rel_err, z_tolerance

pytestmark = pytest.mark.gpu


def _gpu_heads(inp):
    cfg = inp["cfg"]
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    B, H, V, d = cfg.B, cfg.H, cfg.V, cfg.d
    logits = torch.empty((B, H, V), dtype=torch.float32, device="cuda")
    z = torch.empty((B, H, d), dtype=dt, device="cuda")
    tok, cl = sr.heads_propose(dev_tensor(inp["hidden"]), dev_tensor(inp["corr"]), dev_tensor(inp["active"]),
                               dev_tensor(inp["A"]), dev_tensor(inp["bias"]), dev_tensor(inp["W"]),
                               dev_tensor(inp["parents"]), dev_tensor(inp["root_token"]), dev_tensor(inp["u_tree"]),
                               inp["max_children"], clip_norm=cfg.clip_norm, logits=logits, z=z)
    torch.cuda.synchronize()
    zf = z.float().cpu().numpy()
    return tok.cpu().numpy(), cl.cpu().numpy(), logits.cpu().numpy(), zf


def _oracle_heads(inp, rows=None, vocab=None):
    cfg = inp["cfg"]
    dt = cfg.dtype
    rows = np.arange(cfg.B) if rows is None else np.asarray(rows)
    W = f64(inp["W"], dt) if vocab is None else f64(inp["W"][vocab], dt)
    return oracle.heads_forward(f64(inp["hidden"], dt)[rows], inp["corr"][rows], inp["active"][rows],
                                f64(inp["A"], dt), f64(inp["bias"], dt), W, cfg.clip_norm, 1e-5,
                                round_fn=None if dt == "f32" else oracle.round_bf16)


def _check_fused_tree(inp, tok, cl, lg, rows):
    """App. B.1 Eq. (slotq), Eq. (childlist): the tree the GPU built inside sr_heads_propose (top-m supports from
    the vocabulary GEMM's group maxima, then the ordered draws) equals the oracle's tree build run on the
    GPU's own fp32 head logits, bit for bit (no logit tolerance enters); only a trajectory whose draws come
    closer than 1e-6 to a cumulative boundary may differ."""
    rows = np.asarray(list(rows))
    otok, ocl, mg = oracle.tree_build(lg[rows], inp["parents"][rows], inp["root_token"][rows], inp["u_tree"][rows])
    excused = 0
    for i, b in enumerate(rows):
        if mg[i] < 1e-6:
            excused += 1
            continue
        np.testing.assert_array_equal(tok[b], otok[i])
        np.testing.assert_array_equal(cl[b], ocl[i].astype(np.float32))
    assert excused <= max(1, len(rows) // 100), excused


def _check_z(inp, z_rows, ref):
    """bf16 head states: one ulp plus what the fp32 evaluation and a flipped LN rounding can move them."""
    tol = z_tolerance(ref["x"], f64(inp["A"], inp["dtype"]))
    assert_z_bf16(z_rows, ref["z_exact"], tol)


def test_config0_full():
    inp = synth.heads_inputs(synth.TINY_FP32, seed=0)
    tok, cl, lg, z = _gpu_heads(inp)
    ref = _oracle_heads(inp)
    assert row_rel_err(z.reshape(-1, inp["cfg"].d), ref["z"].reshape(-1, inp["cfg"].d)).max() <= 1e-5
    assert row_rel_err(lg.reshape(-1, inp["cfg"].V), ref["logits"].reshape(-1, inp["cfg"].V)).max() <= 1e-5
    _check_fused_tree(inp, tok, cl, lg, range(inp["cfg"].B))


# B*H rows 15, 96 and 132 take the 64-, 128- and 256-row vocabulary tiles; V = 262144 is the largest vocabulary
# of the grouped top-M (4096 groups of 64 columns); d = 64 is a single K-step of both GEMMs and d = 8192 the
# widest row the clip + LayerNorm holds in registers
@pytest.mark.parametrize("cfg_over", [dict(B=5, d=512, H=3, V=3000, T=16, depth=4),
                                      dict(B=24, d=512, H=4, V=5000, T=16, depth=4),
                                      dict(B=33, d=256, H=4, V=1000, T=32, depth=5, active_frac=0.5),
                                      dict(B=3, d=256, H=2, V=262144, T=24, depth=4),
                                      dict(B=66, d=256, H=2, V=262144, T=16, depth=4),
                                      dict(B=9, d=64, H=3, V=4104, T=16, depth=4),
                                      dict(B=3, d=8192, H=1, V=2048, T=8, depth=3)],
                         ids=["B5-V3000", "B24-V5000", "B33-V1000", "B3-V262144", "B66-V262144", "d64", "d8192"])
def test_bf16_scaled(cfg_over):
    cfg = synth.scaled(synth.SHAPE_7B, **cfg_over)
    inp = synth.heads_inputs(cfg, seed=1)
    tok, cl, lg, z = _gpu_heads(inp)
    ref = _oracle_heads(inp)
    _check_z(inp, z, ref)
    lerr = row_rel_err(lg.reshape(-1, cfg.V), ref["logits"].reshape(-1, cfg.V))
    assert lerr.max() <= 2e-3, lerr.max()
    _check_fused_tree(inp, tok, cl, lg, range(cfg.B))


def _full_size(cfg, rows, tree_rows):
    print(f"[heads] {cfg.name} B={cfg.B} T={cfg.T}", flush=True)
    inp = synth.heads_inputs(cfg, seed=0)
    tok, cl, lg, z = _gpu_heads(inp)
    ref = _oracle_heads(inp, rows=rows)
    _check_z(inp, z[rows], ref)
    lerr = row_rel_err(lg[rows].reshape(-1, cfg.V), ref["logits"].reshape(-1, cfg.V))
    print(f"[parity] heads {cfg.name}: {len(rows)} trajectories, max logits row rel err {lerr.max():.2e} (bar 2e-3)",
          flush=True)
    assert lerr.max() <= 2e-3, lerr.max()
    _check_fused_tree(inp, tok, cl, lg, tree_rows)
    return inp


@pytest.mark.parametrize("name,rseed", [("1.5B-shape", 1), ("7B-shape", 2), ("14B-shape-tail", 3)])
def test_full_size_sampled(name, rseed):
    cfg = synth.WORKLOADS[name]
    rng = np.random.default_rng(rseed)
    rows = rng.choice(cfg.B, size=min(3, cfg.B), replace=False)
    _full_size(cfg, rows, rng.choice(cfg.B, size=min(12, cfg.B), replace=False))


@pytest.mark.parametrize("point", synth.SWEEP_POINTS, ids=lambda p: f"B{p[0]}-T{p[1]}")
def test_sweep_points_sampled(point):
    # the concurrency sweep at full size: B*H from 1024 rows (four 256-row vocabulary tiles) down to 16, Reflex
    # corrections on a random half of the trajectories; sampled rows include both kinds and the last row
    cfg = synth.sweep_config(*point)
    act = synth.heads_inputs(cfg, seed=0, with_weights=False)["active"].astype(bool)
    rng = np.random.default_rng(point[0] * 1000 + point[1])
    on, off = np.flatnonzero(act), np.flatnonzero(~act)
    rows = [cfg.B - 1]
    for grp in (on, off):
        if len(grp):
            rows += list(rng.choice(grp, size=min(2, len(grp)), replace=False))
    rows = np.unique(np.asarray(rows))
    assert act[rows].any() and (~act[rows]).any()
    _full_size(cfg, rows, rng.choice(cfg.B, size=min(8, cfg.B), replace=False))


# ---------------------------------------------------------------- tree build alone: bit-exact
def _gpu_tree(inp):
    tok, cl = sr.tree_build(dev_tensor(inp["logits"]), dev_tensor(inp["parents"]), dev_tensor(inp["root_token"]),
                            dev_tensor(inp["u_tree"]), inp["max_children"])
    torch.cuda.synchronize()
    return tok.cpu().numpy(), cl.cpu().numpy()


@pytest.mark.parametrize("cfg", [synth.TINY_FP32, synth.scaled(synth.SHAPE_14B_TAIL, B=6, V=20000),
                                 synth.scaled(synth.sweep_config(4, 96), V=50000),
                                 synth.scaled(synth.SHAPE_7B, B=3, V=262144)], ids=lambda c: f"{c.name}-V{c.V}")
@pytest.mark.parametrize("tie_frac", [0.0, 0.5])
def test_tree_build_bit_exact(cfg, tie_frac):
    inp = synth.head_logits_inputs(cfg, seed=2, tie_frac=tie_frac)
    tok, cl = _gpu_tree(inp)
    otok, ocl, mg = oracle.tree_build(inp["logits"], inp["parents"], inp["root_token"], inp["u_tree"])
    for b in range(cfg.B):
        if mg[b] < 1e-12:           # a draw exactly on a cumulative boundary may go either way
            continue
        np.testing.assert_array_equal(tok[b], otok[b])
        np.testing.assert_array_equal(cl[b], ocl[b].astype(np.float32))


@pytest.mark.parametrize("fan", [16, 17, 64, 65, 127])
def test_tree_build_wide_nodes(fan):
    """A root with `fan` children and a chain below one of them: the draws of up to 16 candidates (one lane
    row), up to 64 (one slot per lane) and more (two slots per lane), bit-exact against the oracle."""
    T = min(fan + 1 + 3, 128)
    par = (-1,) + (0,) * fan + tuple(range(fan, fan + T - fan - 1))
    cfg = synth.scaled(synth.SHAPE_7B, B=6, T=T, depth=1 + (T - fan - 1), V=30000, parents=par)
    for tie_frac in (0.0, 0.5):
        inp = synth.head_logits_inputs(cfg, seed=7 + fan, tie_frac=tie_frac)
        assert inp["max_children"] == fan
        tok, cl = _gpu_tree(inp)
        otok, ocl, mg = oracle.tree_build(inp["logits"], inp["parents"], inp["root_token"], inp["u_tree"])
        for b in range(cfg.B):
            if mg[b] < 1e-12:           # a draw exactly on a cumulative boundary may go either way
                continue
            np.testing.assert_array_equal(tok[b], otok[b])
            np.testing.assert_array_equal(cl[b], ocl[b].astype(np.float32))


def test_tree_build_full_vocab_rows():
    inp = synth.head_logits_inputs(synth.scaled(synth.SHAPE_7B, B=16), seed=3)
    tok, cl = _gpu_tree(inp)
    otok, ocl, mg = oracle.tree_build(inp["logits"], inp["parents"], inp["root_token"], inp["u_tree"])
    ok = mg >= 1e-12
    assert ok.sum() >= len(ok) - 1
    np.testing.assert_array_equal(tok[ok], otok[ok])


def test_tree_build_invalid_topology():
    inp = synth.head_logits_inputs(synth.TINY_FP32, seed=4)
    inp["parents"] = inp["parents"].copy()
    inp["parents"][1, 5] = 7
    tok, cl = _gpu_tree(inp)
    assert (tok[1, 1:] == -1).all() and np.isnan(cl[1, 1:]).all()
    otok, _, _ = oracle.tree_build(inp["logits"][:1], inp["parents"][:1], inp["root_token"][:1], inp["u_tree"][:1])
    np.testing.assert_array_equal(tok[0], otok[0])


def test_heads_deterministic():
    cfg = synth.scaled(synth.SHAPE_7B, B=16, d=512, V=4000)
    inp = synth.heads_inputs(cfg, seed=5)
    a = _gpu_heads(inp)
    b = _gpu_heads(inp)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
