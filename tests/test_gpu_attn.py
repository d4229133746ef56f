"""GPU parity of sr_tree_verify_attn against the float64 oracle (App. B.1 Eq. (nodep))."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_04962_amd as sr
import synth
from helpers import dev_tensor, f64, row_rel_err, tol_for

pytestmark = pytest.mark.gpu


def _run_gpu(inp):
    t = {k: dev_tensor(inp[k]) for k in ("q", "k_cache", "v_cache", "k_tree", "v_tree")}
    out, lse = sr.tree_verify_attn(t["q"], t["k_cache"], t["v_cache"], dev_tensor(inp["block_table"]),
                                   dev_tensor(inp["ctx_len"]), t["k_tree"], t["v_tree"], dev_tensor(inp["parents"]),
                                   scale=inp["scale"])
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy()


def _oracle(inp, nodes=None):
    dt = inp["dtype"]
    return oracle.tree_attention(f64(inp["q"], dt), f64(inp["k_cache"], dt), f64(inp["v_cache"], dt),
                                 inp["block_table"], inp["ctx_len"], f64(inp["k_tree"], dt), f64(inp["v_tree"], dt),
                                 inp["parents"], inp["scale"], 16, nodes=nodes)


def _check(inp, nodes=None):
    print(f"[attn] {inp['cfg'].name} B={inp['cfg'].B} T={inp['cfg'].T}", flush=True)
    out, lse = _run_gpu(inp)
    ro, rl = _oracle(inp, nodes)
    tol = tol_for(inp["dtype"])
    sel = ~np.isnan(ro[..., 0])
    assert sel.any()
    err = row_rel_err(out[sel], ro[sel])
    assert err.max() <= tol, f"max row error {err.max():.3e} > {tol}"
    # lse (natural log of the softmax normaliser): absolute error within the same bar
    lerr = np.abs(lse[sel] - rl[sel]).max()
    print(f"[parity] attention {inp['cfg'].name}: {int(sel.sum() // inp['cfg'].Hq)} nodes, max row rel err "
          f"{err.max():.2e}, max lse abs err {lerr:.2e} (bar {tol})", flush=True)
    assert lerr <= tol, f"lse error {lerr:.3e} > {tol}"
    assert np.isfinite(out).all()
    return err.max()


def test_config0_all_nodes():
    _check(synth.attn_inputs(synth.TINY_FP32, seed=0))


@pytest.mark.parametrize("seed", [0, 1])
def test_bf16_multi_chunk_ragged(seed):
    # 10 (trajectory, KV head) pairs take 32-page (512-token) chunks: contexts up to 5000 tokens run the
    # split/combine path over up to ten chunks with ragged tails
    cfg = synth.scaled(synth.SHAPE_7B, B=5, T=12, depth=4, Hq=8, Hkv=2, ctx=("uniform", 1, 5000))
    inp = synth.attn_inputs(cfg, seed=seed)
    _check(inp)


def test_bf16_long_chunks_all_nodes():
    # 512 (trajectory, KV head) pairs select 256-page prefix chunks: contexts of 2900-9000 tokens take one
    # to three chunks, with ragged tails; every node of every trajectory is compared
    cfg = synth.scaled(synth.SHAPE_7B, B=128, T=2, depth=1, ctx=("uniform", 2900, 9000))
    _check(synth.attn_inputs(cfg, seed=5))


def test_bf16_rows_over_one_block_gqa7():
    # T*G = 40*7 = 280 > 256 query rows: two row groups
    cfg = synth.scaled(synth.SHAPE_7B, B=2, T=40, depth=5, ctx=("uniform", 100, 3000))
    _check(synth.attn_inputs(cfg, seed=3))


def test_fp32_d128_and_bf16_d64():
    _check(synth.attn_inputs(synth.scaled(synth.TINY_FP32, D=128, Hq=6, Hkv=3), seed=4))
    _check(synth.attn_inputs(synth.scaled(synth.SHAPE_1P5B, dtype="bf16", B=3, D=64, ctx=("uniform", 20, 300)),
                             seed=5))


def test_one_query_head_per_kv_head():
    # G = 1 (no grouping): one 32-row block per T nodes, split prefixes with ragged tails, bf16 and fp32
    _check(synth.attn_inputs(synth.scaled(synth.SHAPE_7B, B=6, T=32, Hq=4, Hkv=4, ctx=("uniform", 900, 5000)),
                             seed=11))
    _check(synth.attn_inputs(synth.scaled(synth.SHAPE_7B, dtype="f32", B=3, T=16, Hq=2, Hkv=2,
                                          ctx=("uniform", 100, 3000)), seed=12))


def test_empty_prefix_and_single_node_tree():
    _check(synth.attn_inputs(synth.scaled(synth.TINY_FP32, ctx=("explicit", (0, 17))), seed=6))
    _check(synth.attn_inputs(synth.scaled(synth.TINY_FP32, T=1, parents=(-1,), ctx=("explicit", (0, 2049))),
                             seed=7))
    _check(synth.attn_inputs(synth.scaled(synth.SHAPE_7B, B=2, T=128, depth=6, Hq=4, Hkv=4,
                                          ctx=("uniform", 0, 40)), seed=8))


def test_invalid_inputs_give_nan_rows_only_for_that_trajectory():
    cfg = synth.scaled(synth.SHAPE_7B, B=3, T=8, depth=3, Hq=8, Hkv=2, ctx=("uniform", 40, 3000))
    inp = synth.attn_inputs(cfg, seed=9)
    inp["block_table"] = inp["block_table"].copy()
    inp["block_table"][1, 0] = inp["num_blocks"] + 5      # page id out of range
    inp["ctx_len"] = inp["ctx_len"].copy()
    inp["ctx_len"][2] = cfg.max_blocks * 16 + 1           # longer than the table
    out, lse = _run_gpu(inp)
    assert np.isnan(out[1]).all() and np.isnan(out[2]).all()
    assert np.isnan(lse[1]).all() and np.isnan(lse[2]).all()
    assert np.isfinite(out[0]).all()
    inp2 = synth.attn_inputs(cfg, seed=9)
    inp2["parents"] = inp2["parents"].copy()
    inp2["parents"][0, 3] = 5                             # not an earlier node
    out2, _ = _run_gpu(inp2)
    assert np.isnan(out2[0]).all() and np.isfinite(out2[1:]).all()
    inp3 = synth.attn_inputs(cfg, seed=9)
    inp3["ctx_len"] = inp3["ctx_len"].copy()
    inp3["ctx_len"][1] = -1                               # negative length
    out3, lse3 = _run_gpu(inp3)
    assert np.isnan(out3[1]).all() and np.isnan(lse3[1]).all()
    assert np.isfinite(out3[0]).all() and np.isfinite(out3[2]).all()


def test_deterministic():
    cfg = synth.scaled(synth.SHAPE_7B, B=4, T=16, depth=4, ctx=("uniform", 1000, 4500))
    inp = synth.attn_inputs(cfg, seed=10)
    a, la = _run_gpu(inp)
    b, lb = _run_gpu(inp)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(la, lb)


def _sample_nodes(cfg, k, seed):
    rng = np.random.default_rng(seed)
    bs = rng.choice(cfg.B, size=min(k, cfg.B), replace=False)
    return [(int(b), int(u)) for b in bs for u in rng.choice(cfg.T, size=min(4, cfg.T), replace=False)]


@pytest.mark.parametrize("name,rseed", [("1.5B-shape", 1), ("7B-shape", 2), ("14B-shape-tail", 3)])
def test_full_size_sampled(name, rseed):
    cfg = synth.WORKLOADS[name]
    inp = synth.attn_inputs(cfg, seed=0)
    _check(inp, nodes=_sample_nodes(cfg, 6, rseed))


@pytest.mark.parametrize("point", synth.SWEEP_POINTS, ids=lambda p: f"B{p[0]}-T{p[1]}")
def test_sweep_points_sampled(point):
    cfg = synth.sweep_config(*point)
    inp = synth.attn_inputs(cfg, seed=0)
    _check(inp, nodes=_sample_nodes(cfg, 4, point[0]))


@pytest.mark.parametrize("T,Hq,Hkv", [(32, 32, 4), (29, 32, 4), (64, 16, 4)])
def test_bf16_rows_224_to_256(T, Hq, Hkv):
    # T*G of 256, 232 and 256 query rows per KV head: more than 224, so the rows split into two groups
    # (each keeps a wave free of query rows for the K/V transfers); contexts take one to several chunks
    cfg = synth.scaled(synth.SHAPE_7B, B=3, T=T, depth=5, Hq=Hq, Hkv=Hkv, ctx=("uniform", 100, 3000))
    _check(synth.attn_inputs(cfg, seed=11))


def _scale_values(inp, traj, fn):
    """Apply fn to the float values of trajectory traj's prefix V pages and tree V rows (bf16 bits kept)."""
    inp = dict(inp)
    vc = synth.to_f64(inp["v_cache"], "bf16")
    vt = synth.to_f64(inp["v_tree"], "bf16")
    L = int(inp["ctx_len"][traj])
    pages = inp["block_table"][traj, :-(-L // 16)]
    vc[pages] = fn(vc[pages])
    vt[traj] = fn(vt[traj])
    inp["v_cache"] = synth.as_dtype(vc.astype(np.float32), "bf16")
    inp["v_tree"] = synth.as_dtype(vt.astype(np.float32), "bf16")
    return inp


def test_bf16_v_outside_fp16_range():
    """bf16 V beyond what the fp16 product keeps: magnitudes around 1e5 (fp16 overflows past 65504), V scaled to
    around 1e-6 and 1e-30 (below fp16's normal range, so its subnormal step would dominate) and a mix of huge
    and tiny values in one trajectory. Those items are recomputed with fp32 V; the others (N(0,1) values, a
    few of them below 2^-14) keep the fp16 product; every trajectory matches the oracle."""
    cfg = synth.scaled(synth.SHAPE_7B, B=6, T=12, depth=4, Hq=8, Hkv=2, ctx=("uniform", 300, 2600))
    inp = synth.attn_inputs(cfg, seed=12)
    inp = _scale_values(inp, 1, lambda v: v * 1.0e5)
    inp = _scale_values(inp, 2, lambda v: v * 1.0e-6)
    inp = _scale_values(inp, 3, lambda v: np.where(np.arange(v.shape[-1]) % 2 == 0, v * 1.0e5, v * 1.0e-6))
    inp = _scale_values(inp, 4, lambda v: v * 1.0e-30)
    out, _ = _run_gpu(inp)
    assert np.isfinite(out).all()
    _check(inp)


def _scale_keys(inp, traj, fn):
    """Multiply trajectory traj's prefix K row of key position k by fn(k), and its tree K rows by fn(L + node)
    (bf16 bits kept)."""
    inp = dict(inp)
    kc = synth.to_f64(inp["k_cache"], "bf16")
    kt = synth.to_f64(inp["k_tree"], "bf16")
    L = int(inp["ctx_len"][traj])
    for k in range(L):
        kc[inp["block_table"][traj, k // 16], :, k % 16, :] *= fn(k)
    for u in range(kt.shape[1]):
        kt[traj, u] *= fn(L + u)
    inp["k_cache"] = synth.as_dtype(kc.astype(np.float32), "bf16")
    inp["k_tree"] = synth.as_dtype(kt.astype(np.float32), "bf16")
    return inp


def test_bf16_scores_growing_falling_and_spiking():
    """The running reference max under scores that move across tiles: keys scaled up along the context
    (every later tile's scores above the first's), scaled down along it, one key at 12x in the middle of a
    long context, and tree keys at 6x (the last tile holds the largest scores)."""
    cfg = synth.scaled(synth.SHAPE_7B, B=5, T=12, depth=4, Hq=8, Hkv=2, ctx=("uniform", 1500, 3000))
    inp = synth.attn_inputs(cfg, seed=21)
    L = inp["ctx_len"]
    inp = _scale_keys(inp, 0, lambda k: 0.05 + 5.0 * k / L[0])
    inp = _scale_keys(inp, 1, lambda k: 5.05 - 5.0 * k / L[1])
    inp = _scale_keys(inp, 2, lambda k: 12.0 if k == L[2] // 2 else 1.0)
    inp = _scale_keys(inp, 3, lambda k: 6.0 if k >= L[3] else 1.0)
    out, _ = _run_gpu(inp)
    assert np.isfinite(out).all()
    _check(inp)
