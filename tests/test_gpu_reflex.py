"""GPU parity of sr_reflex_feedback against the float64 oracle (Sec. 3.3; Sec. 3.4 Eq. (support) to
Eq. (ema)): per-record statistics, the feedback vector e and the updated memory, from the tiny case to the
7B shape at full size, the fallback selections (few groups, ties), gating, duplicates and invalid records."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_04962_amd as sr
import synth
from helpers import dev_tensor, row_rel_err

pytestmark = pytest.mark.gpu

RHO = (0.85, 0.90, 0.95, 0.95, 0.95)
MARGIN = 1e-6


class _Rows:
    """float64 rows of a stored (f32 or bf16-bits) matrix, converted on access."""

    def __init__(self, x, dt):
        self.x, self.dt = x, dt

    def __getitem__(self, idx):
        return synth.to_f64(self.x[idx], self.dt)


def _gpu(inp, W=None, **params):
    mem = dev_tensor(inp["memory"])
    stats, e = sr.reflex_feedback(dev_tensor(inp["p_logits"]), dev_tensor(inp["p_row"]), dev_tensor(inp["q_logits"]),
                                  dev_tensor(inp["q_row"]), dev_tensor(inp["cand"]), dev_tensor(inp["y_star"]),
                                  dev_tensor(inp["traj"]), dev_tensor(inp["horizon"]),
                                  dev_tensor(inp["W"]) if W is None else W, mem, rho=RHO, want_e=True,
                                  support=inp["support"], **params)
    torch.cuda.synchronize()
    return mem.cpu().numpy(), stats.cpu().numpy(), e.cpu().numpy()


def _oracle(inp, rows=None, **params):
    dt = inp["dtype"]
    kw = dict(params)
    w_min = kw.pop("w_min", 0.03)
    return oracle.reflex_feedback(_Rows(inp["p_logits"], dt), inp["p_row"], inp["q_logits"], inp["q_row"], inp["cand"],
                                  inp["y_star"], inp["traj"], inp["horizon"], _Rows(inp["W"], dt), inp["memory"],
                                  rho=RHO, w_min=w_min, rows=rows, support=inp["support"], **kw)


def _compare(inp, rows=None, **params):
    cfg = inp["cfg"]
    print(f"[reflex] {cfg.name} R={inp['R']} V={cfg.V} d={cfg.d} support={inp['support']} {params}", flush=True)
    gm, gs, ge = _gpu(inp, **params)
    om, info = _oracle(inp, rows, **params)
    exempt = 0
    touched = set()
    for r, f in enumerate(info):
        if f is None:
            continue
        if f["applied"] == -1:
            assert gs[r, 5] == -1 and np.isnan(ge[r]).all()
            continue
        slot = (int(inp["traj"][r]), int(inp["horizon"][r]) - 1)
        touched.add(slot)
        got = dict(d_dist=gs[r, 0], d_cov=gs[r, 1], tv_s=gs[r, 2], severity=gs[r, 3], p_C=gs[r, 6], p_star=gs[r, 7])
        for k, v in got.items():
            assert v == pytest.approx(f[k], rel=1e-5, abs=1e-7), (r, k, v, f[k])
        assert int(gs[r, 4]) == len(f["support"]), r
        if int(gs[r, 5]) != f["applied"]:
            assert abs(f["severity"] - params.get("w_min", 0.03)) < MARGIN, r
            exempt += 1
            continue
        assert row_rel_err(ge[r], f["e"]) < 1e-5, (r, row_rel_err(ge[r], f["e"]))
        i, h = slot
        if f["applied"]:
            assert row_rel_err(gm[i, h], om[i, h]) < 1e-5, r
        else:
            np.testing.assert_array_equal(gm[i, h], inp["memory"][i, h])
    assert exempt <= max(1, len(info) // 100)
    # memory rows no record touched are bit-identical
    B, H = inp["memory"].shape[:2]
    if rows is None:
        for i in range(B):
            for h in range(H):
                if (i, h) not in touched:
                    np.testing.assert_array_equal(gm[i, h], inp["memory"][i, h])
    return gm, gs, ge, info


def test_config0_all_records():
    # V = 512 has 8 groups, fewer than the 48 top entries: the full radix selection runs
    _compare(synth.reflex_inputs(synth.TINY_FP32, seed=0))


@pytest.mark.parametrize("support", [48, 8])
def test_bf16_1p5b_shape(support):
    cfg = synth.scaled(synth.SHAPE_1P5B, B=4)
    _compare(synth.reflex_inputs(cfg, seed=1, support=support))


def test_14b_shape_two_column_groups():
    cfg = synth.scaled(synth.SHAPE_14B_TAIL, B=2)          # d = 5120: two 8-column groups per lane
    _compare(synth.reflex_inputs(cfg, seed=2))


def test_full_size_7b_sampled():
    """B=128 trajectories x 4 horizons = 512 records at V=151936, d=3584; 24 records checked."""
    inp = synth.reflex_inputs(synth.SHAPE_7B, seed=3)
    rows = set(np.random.default_rng(0).choice(inp["R"], 24, replace=False).tolist())
    _compare(inp, rows=rows)


def test_temperature_and_parameters():
    cfg = synth.scaled(synth.SHAPE_1P5B, B=2, H=3)
    _compare(synth.reflex_inputs(cfg, seed=4, support=16), temperature=0.7, n_boundary=2, w_dist=0.5, w_cov=2.0,
             eps=1e-4)


def test_ties_take_the_full_selection():
    cfg = synth.scaled(synth.SHAPE_1P5B, B=2, H=2)
    inp = synth.reflex_inputs(cfg, seed=5)
    p = synth.to_f64(inp["p_logits"], "bf16")
    p[0] = 0.0                                      # a constant target row: every group ties
    p[1, : cfg.V // 2] = 1.0                        # half the row tied at the top
    inp["p_logits"] = synth.as_dtype(p.astype(np.float32), "bf16")
    inp["q_logits"][2] = 3.0                        # a constant proposal row
    _compare(inp)


def test_gate_duplicates_and_invalid_records():
    cfg = synth.scaled(synth.SHAPE_1P5B, B=6, H=2)
    inp = synth.reflex_inputs(cfg, seed=6)
    R = inp["R"]
    # record 1 becomes a low-severity record: candidates hold almost all target mass and q equals p
    p = synth.to_f64(inp["p_logits"], "bf16")
    p[1] = -20.0
    p[1, inp["cand"][1][inp["cand"][1] >= 0]] = 10.0
    inp["p_logits"] = synth.as_dtype(p.astype(np.float32), "bf16")
    inp["q_logits"][1] = p[1].astype(np.float32)
    # record R-1 repeats record 0's slot (skipped); the invalid ones get slots of their own
    inp["traj"][R - 1], inp["horizon"][R - 1] = inp["traj"][0], inp["horizon"][0]
    bad = {2: ("p_row", 10 ** 6), 3: ("horizon", 3), 4: ("y_star", cfg.V), 5: ("cand_dup", None),
           6: ("cand_gap", None), 7: ("cand_range", None)}
    inp_bad = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in inp.items()}
    for r, (what, val) in bad.items():
        if what == "cand_dup":
            inp_bad["cand"][r, 1] = inp_bad["cand"][r, 0]
        elif what == "cand_gap":
            inp_bad["cand"][r, 0] = -1
        elif what == "cand_range":
            inp_bad["cand"][r, 0] = cfg.V
        else:
            inp_bad[what][r] = val
    gm, gs, ge = _gpu(inp_bad)
    for r in bad:
        assert gs[r, 5] == -2 and np.isnan(gs[r, [0, 1, 2, 3, 4, 6, 7]]).all() and np.isnan(ge[r]).all()
    assert gs[R - 1, 5] == -1
    assert gs[1, 5] == 0 and gs[1, 3] < 0.03
    # the remaining records agree with the oracle run on them alone
    keep = [r for r in range(R) if r not in bad]
    sub = {k: (v[keep] if isinstance(v, np.ndarray) and v.shape[:1] == (R,) else v) for k, v in inp.items()}
    sub["p_row"] = np.arange(len(keep), dtype=np.int32)
    sub["q_row"] = np.arange(len(keep), dtype=np.int32)
    sub["R"] = len(keep)
    om, info = _oracle(sub)
    for j, r in enumerate(keep):
        f = info[j]
        assert int(gs[r, 5]) == f["applied"], r
        if f["applied"] >= 0:
            assert row_rel_err(ge[r], f["e"]) < 1e-5
    for i in range(cfg.B):
        for h in range(cfg.H):
            np.testing.assert_allclose(gm[i, h], om[i, h], rtol=1e-5, atol=1e-6)


# ----------------------------------------------------------------------------- gated correction
GATE = dict(z_delta=0.6, eps=1e-6, m_floor=1e-8, alpha_min=(0.010, 0.004, 0.0025), alpha_max=(0.025, 0.010, 0.006),
            n_fb_min=(1, 2, 4), n_align_min=(6, 16, 48))


def _per_head(v, h):
    return v[min(h, len(v) - 1)]


def _gpu_heads_reflex(inp, gin, P=True):
    cfg = inp["cfg"]
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    B, H, V, d = cfg.B, cfg.H, cfg.V, cfg.d
    rank = gin["P"].shape[0]
    logits = torch.empty((B, H, V), dtype=torch.float32, device="cuda")
    z = torch.empty((B, H, d), dtype=dt, device="cuda")
    sk = torch.empty((B, H, rank), dtype=torch.float32, device="cuda")
    al = torch.empty((B, H), dtype=torch.float32, device="cuda")
    tok, cl = sr.heads_propose_reflex(dev_tensor(inp["hidden"]), dev_tensor(inp["corr"]), dev_tensor(inp["active"]),
                                      dev_tensor(inp["A"]), dev_tensor(inp["bias"]), dev_tensor(inp["W"]),
                                      dev_tensor(inp["parents"]), dev_tensor(inp["root_token"]),
                                      dev_tensor(inp["u_tree"]), inp["max_children"], dev_tensor(gin["memory"]),
                                      dev_tensor(gin["align"]), dev_tensor(gin["P"]), clip_norm=cfg.clip_norm,
                                      logits=logits, z=z, sketch_out=sk, alpha_out=al, **GATE)
    torch.cuda.synchronize()
    return (tok.cpu().numpy(), cl.cpu().numpy(), logits.cpu().numpy(), z.float().cpu().numpy(), sk.cpu().numpy(),
            al.cpu().numpy())


@pytest.mark.parametrize("name,over", [("tiny-fp32", None), ("1.5B-shape", dict(B=5, V=20000))])
def test_gated_correction_parity(name, over):
    from helpers import assert_z_bf16, bf16_ulp, f64, z_tolerance
    cfg = synth.TINY_FP32 if over is None else synth.scaled(synth.SHAPE_1P5B, **over)
    inp = synth.heads_inputs(cfg, seed=7)
    gin = synth.reflex_gate_inputs(cfg, seed=7)
    print(f"[reflex-gate] {cfg.name} B={cfg.B} H={cfg.H} d={cfg.d} V={cfg.V}", flush=True)
    tok, cl, lg, z, sk, alpha = _gpu_heads_reflex(inp, gin)
    dt = cfg.dtype
    ref = oracle.heads_forward(f64(inp["hidden"], dt), inp["corr"], inp["active"], f64(inp["A"], dt),
                               f64(inp["bias"], dt), f64(inp["W"], dt), cfg.clip_norm, 1e-5,
                               round_fn=None if dt == "f32" else oracle.round_bf16)
    W64 = f64(inp["W"], dt)
    # the corrected state inherits the head state's deviation (one ulp plus the flipped-LN bound) on top of
    # its own rounding
    zin_tol = None if dt == "f32" else bf16_ulp(ref["z_exact"]) + z_tolerance(ref["x"], f64(inp["A"], dt))
    opened = 0
    for b in range(cfg.B):
        for h in range(cfg.H):
            st = tuple(float(x) for x in gin["align"][b, h, :3])
            zt, a, _ = oracle.correction(ref["z"][b, h], gin["memory"][b, h], st, float(gin["align"][b, h, 3]),
                                         _per_head(GATE["alpha_min"], h), _per_head(GATE["alpha_max"], h),
                                         _per_head(GATE["n_fb_min"], h), _per_head(GATE["n_align_min"], h),
                                         GATE["z_delta"], GATE["eps"], GATE["m_floor"])
            opened += a > 0
            assert alpha[b, h] == pytest.approx(a, abs=1e-7), (b, h)
            s = oracle.sketch(gin["memory"][b, h], gin["P"])
            np.testing.assert_allclose(sk[b, h], np.zeros(sk.shape[2]) if s is None else s, rtol=1e-5, atol=1e-6)
            if dt == "f32":
                assert row_rel_err(z[b, h], zt) <= 1e-5
                zr = zt
            else:
                assert_z_bf16(z[b, h][None], zt[None], zin_tol[b, h][None])
                zr = oracle.round_bf16(zt)
            assert row_rel_err(lg[b, h], W64 @ zr) <= (1e-5 if dt == "f32" else 2e-3)
    assert 0 < opened < cfg.B * cfg.H


def test_closed_gates_match_plain_proposal():
    cfg = synth.scaled(synth.SHAPE_1P5B, B=3, V=8000)
    inp = synth.heads_inputs(cfg, seed=8)
    gin = synth.reflex_gate_inputs(cfg, seed=8)
    gin["align"][:, :, 3] = 0.0                     # no feedback yet: every gate closed
    tok, cl, lg, z, sk, alpha = _gpu_heads_reflex(inp, gin)
    assert (alpha == 0).all()
    B, H, V, d = cfg.B, cfg.H, cfg.V, cfg.d
    logits = torch.empty((B, H, V), dtype=torch.float32, device="cuda")
    zz = torch.empty((B, H, d), dtype=torch.bfloat16, device="cuda")
    tok2, cl2 = sr.heads_propose(dev_tensor(inp["hidden"]), dev_tensor(inp["corr"]), dev_tensor(inp["active"]),
                                 dev_tensor(inp["A"]), dev_tensor(inp["bias"]), dev_tensor(inp["W"]),
                                 dev_tensor(inp["parents"]), dev_tensor(inp["root_token"]), dev_tensor(inp["u_tree"]),
                                 inp["max_children"], clip_norm=cfg.clip_norm, logits=logits, z=zz)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(tok, tok2.cpu().numpy())
    np.testing.assert_array_equal(cl, cl2.cpu().numpy())
    np.testing.assert_array_equal(lg, logits.cpu().numpy())
    np.testing.assert_array_equal(z, zz.float().cpu().numpy())


def test_feedback_alignment_moments():
    cfg = synth.scaled(synth.SHAPE_1P5B, B=6, H=3)
    inp = synth.reflex_inputs(cfg, seed=9)
    gin = synth.reflex_gate_inputs(cfg, seed=9)
    s_rec = synth.unit_sketches(inp["R"], gin["P"].shape[0], seed=9)
    align0 = gin["align"].copy()
    print(f"[reflex-align] {cfg.name} R={inp['R']}", flush=True)
    mem = dev_tensor(inp["memory"])
    al = dev_tensor(align0)
    stats, e = sr.reflex_feedback(dev_tensor(inp["p_logits"]), dev_tensor(inp["p_row"]), dev_tensor(inp["q_logits"]),
                                  dev_tensor(inp["q_row"]), dev_tensor(inp["cand"]), dev_tensor(inp["y_star"]),
                                  dev_tensor(inp["traj"]), dev_tensor(inp["horizon"]), dev_tensor(inp["W"]), mem,
                                  rho=RHO, want_e=True, P=dev_tensor(gin["P"]), rec_sketch=dev_tensor(s_rec), align=al,
                                  support=inp["support"])
    torch.cuda.synchronize()
    om, info, oal = oracle.reflex_feedback(_Rows(inp["p_logits"], "bf16"), inp["p_row"], inp["q_logits"], inp["q_row"],
                                           inp["cand"], inp["y_star"], inp["traj"], inp["horizon"],
                                           _Rows(inp["W"], "bf16"), inp["memory"], rho=RHO, support=inp["support"],
                                           P=gin["P"], rec_sketch=s_rec, align=align0)
    gal = al.cpu().numpy()
    st = stats.cpu().numpy()
    observed = 0
    for r, f in enumerate(info):
        assert int(st[r, 5]) == f["applied"]
        observed += "alignment" in f
    assert observed > 0
    np.testing.assert_allclose(gal, oal, rtol=1e-5, atol=1e-6)
