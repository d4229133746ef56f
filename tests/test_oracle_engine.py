"""Pins of the engine-glue oracle: the concurrency-aware node budget (Sec. 3.2, Eq. (verification-budget),
Eq. (tree-budget); App. C "Implementation and Reproducibility Details", paragraph "Concurrency-aware sparse
tree verification") and the accepted-path cache extraction."""
import numpy as np
import pytest

import oracle
import synth

# (live responses B_t, N_t, non-root nodes per horizon) worked out by hand from the paper's settings
# C_peak = 512, N_min = 1, N_max = 10 (root counted), nominal allocation (5, 4, 0).
PAPER_BUDGETS = [
    (1, 10, [5, 4]),
    (51, 10, [5, 4]),     # 512 // 51 = 10
    (52, 9, [5, 3]),      # 512 // 52 = 9
    (64, 8, [5, 2]),
    (73, 7, [5, 1]),      # 512 // 73 = 7
    (85, 6, [5]),         # 512 // 85 = 6: horizon 2 gets nothing, the tree stops there
    (86, 5, [4]),
    (128, 4, [3]),
    (256, 2, [1]),
    (257, 1, []),         # 512 // 257 = 1: the anchor alone
    (512, 1, []),
    (513, 1, []),         # floor gives 0, N_min lifts it to 1
    (100000, 1, []),
]


@pytest.mark.parametrize("live,n_t,counts", PAPER_BUDGETS)
def test_budget_paper_settings(live, n_t, counts):
    got_n, got_counts, parents = oracle.tree_budget(live)
    assert got_n == n_t
    assert got_counts == counts
    assert parents.shape[0] == 1 + sum(counts)


def test_budget_full_tree_shape():
    # (5, 4): the first four horizon-1 nodes each carry one horizon-2 node
    _, _, p = oracle.tree_budget(1)
    assert p.tolist() == [-1, 0, 0, 0, 0, 0, 1, 2, 3, 4]
    # (5, 2): horizon-2 nodes spread over the horizon-1 slots 0 and 2
    _, _, p = oracle.tree_budget(64)
    assert p.tolist() == [-1, 0, 0, 0, 0, 0, 1, 3]


@pytest.mark.parametrize("c_peak,n_min,n_max,alloc", [
    (512, 1, 10, (5, 4, 0)), (512, 2, 10, (5, 4, 0)), (1000, 1, 64, (8, 8, 8, 8, 8, 8, 8, 8)),
    (300, 3, 17, (1, 6, 2, 9)), (64, 1, 5, (0, 3)), (7, 1, 128, (100, 100))])
def test_budget_invariants_brute_force(c_peak, n_min, n_max, alloc):
    prev = None
    for live in range(1, 3 * c_peak + 3):
        n_t, counts, parents = oracle.tree_budget(live, c_peak, n_min, n_max, alloc)
        size = parents.shape[0]
        # Eq. (verification-budget): the clip of floor(C / B_t), checked against a search
        best = max([n for n in range(0, c_peak + 1) if n * live <= c_peak])
        assert n_t == min(max(best, n_min), n_max)
        # Eq. (tree-budget): anchor counted once, never above N_t
        assert size == 1 + sum(counts) <= n_t
        # truncation spends the whole budget unless the nominal tree is smaller or a zero horizon ends it
        nominal = 0
        for a in alloc:
            if a == 0:
                break
            nominal += a
        assert size == min(n_t, 1 + nominal)
        # the batch-wide envelope B_t |T| <= C holds wherever floor(C / B_t) >= N_min
        if c_peak // live >= n_min:
            assert live * size <= c_peak
        # N_t never grows as the live batch grows
        assert prev is None or n_t <= prev
        prev = n_t
        # a valid breadth-first topology whose horizon-h nodes sit at depth h, evenly spread
        depth, kids = oracle.tree_structure(parents)
        start = 1
        for h, n in enumerate(counts, 1):
            assert (depth[start:start + n] == h).all()
            if h > 1:
                par_lvl = [len(kids[w]) for w in range(start - counts[h - 2], start)]
                assert max(par_lvl) - min(par_lvl) <= 1
            start += n
        assert start == size


def test_budget_rejects_bad_arguments():
    with pytest.raises(ValueError):
        oracle.tree_budget(0)
    with pytest.raises(ValueError):
        oracle.tree_budget(4, n_min=0)
    with pytest.raises(ValueError):
        oracle.tree_budget(4, n_min=5, n_max=4)
    with pytest.raises(ValueError):
        oracle.tree_budget(4, alloc=(3, -1))


def _tiny_cache():
    # 2 trajectories, pages of 4 tokens, Hkv=1, D=2; every cache entry starts as -1
    kc = -np.ones((6, 1, 4, 2))
    vc = -np.ones((6, 1, 4, 2))
    table = np.array([[4, 1, 5], [0, 2, 3]], dtype=np.int32)
    ctx = np.array([3, 8], dtype=np.int32)
    T = 6
    kt = np.zeros((2, T, 1, 2))
    vt = np.zeros((2, T, 1, 2))
    for b in range(2):
        for u in range(T):
            kt[b, u, 0] = [100 * b + u, 0.5]
            vt[b, u, 0] = [-(100 * b + u), 0.25]
    return kc, vc, table, ctx, kt, vt


def test_commit_hand_example():
    kc, vc, table, ctx, kt, vt = _tiny_cache()
    acc = np.array([[2, 5, -1], [-1, -1, -1]], dtype=np.int32)
    out_len = np.array([3, 1], dtype=np.int32)
    nk, nv, nctx = oracle.commit_path(kc, vc, table, ctx, kt, vt, acc, out_len, block_size=4)
    assert nctx.tolist() == [6, 9]
    # trajectory 0: positions 3, 4, 5 -> (page 4, slot 3), (page 1, slot 0), (page 1, slot 1)
    assert nk[4, 0, 3].tolist() == [0, 0.5] and nv[4, 0, 3].tolist() == [0, 0.25]
    assert nk[1, 0, 0].tolist() == [2, 0.5] and nv[1, 0, 0].tolist() == [-2, 0.25]
    assert nk[1, 0, 1].tolist() == [5, 0.5] and nv[1, 0, 1].tolist() == [-5, 0.25]
    # trajectory 1: only the anchor, at position 8 -> (page 3, slot 0)
    assert nk[3, 0, 0].tolist() == [100, 0.5] and nv[3, 0, 0].tolist() == [-100, 0.25]
    changed = (nk != kc).any(axis=(1, 3))
    assert sorted(zip(*np.nonzero(changed))) == [(1, 0), (1, 1), (3, 0), (4, 3)]
    assert (kc == -1).all()                              # inputs are not modified


@pytest.mark.parametrize("name", ["tiny-fp32", "14B-shape-tail"])
def test_commit_cache_reads_back_as_prefix_plus_path(name):
    cfg = synth.get_config(name)
    if name == "14B-shape-tail":
        cfg = synth.scaled(cfg, B=4, ctx=("uniform", 30, 70), dtype="f32")
    inp = synth.commit_inputs(cfg, seed=3)
    kc, vc = inp["k_cache"][0].astype(np.float64), inp["v_cache"][0].astype(np.float64)
    kt, vt = inp["k_tree"][0].astype(np.float64), inp["v_tree"][0].astype(np.float64)
    nk, nv, nctx = oracle.commit_path(kc, vc, inp["block_table"], inp["ctx_len"], kt, vt,
                                      inp["acc_nodes"], inp["out_len"], cfg.block_size)
    assert (nctx == inp["ctx_len"] + inp["out_len"]).all()
    for b in range(cfg.B):
        n = int(inp["out_len"][b]) - 1
        path = [0] + inp["acc_nodes"][b, :n].tolist()
        # the accepted nodes form a root path (the walk moves from a node to one of its children)
        for i in range(1, len(path)):
            assert inp["parents"][b, path[i]] == path[i - 1]
        L = int(inp["ctx_len"][b])
        seq_k = oracle.gather_prefix(nk, inp["block_table"][b], int(nctx[b]), cfg.block_size)
        seq_v = oracle.gather_prefix(nv, inp["block_table"][b], int(nctx[b]), cfg.block_size)
        np.testing.assert_array_equal(seq_k[:L], oracle.gather_prefix(kc, inp["block_table"][b], L, cfg.block_size))
        np.testing.assert_array_equal(seq_k[L:], kt[b, path])
        np.testing.assert_array_equal(seq_v[L:], vt[b, path])
        # slots past the new length stay untouched (NaN in these inputs)
        pos = np.arange(int(nctx[b]), inp["block_table"].shape[1] * cfg.block_size)
        pos = pos[inp["block_table"][b, pos // cfg.block_size] >= 0]
        assert np.isnan(nk[inp["block_table"][b, pos // cfg.block_size], :, pos % cfg.block_size]).all()


def test_commit_then_attention_matches_tree_attention():
    """Eq. (nodep) across rounds: the next round's anchor query over the committed cache sees the same
    keys/values the tree-masked attention gave the deepest accepted node."""
    cfg = synth.scaled(synth.get_config("tiny-fp32"), B=2)
    inp = synth.commit_inputs(cfg, seed=5)
    rng = np.random.default_rng(11)
    q = rng.standard_normal((cfg.B, cfg.T, cfg.Hq, cfg.D))
    kc, vc = inp["k_cache"][0].astype(np.float64), inp["v_cache"][0].astype(np.float64)
    kt, vt = inp["k_tree"][0].astype(np.float64), inp["v_tree"][0].astype(np.float64)
    scale = cfg.D ** -0.5
    out, lse = oracle.tree_attention(q, kc, vc, inp["block_table"], inp["ctx_len"], kt, vt,
                                     inp["parents"], scale, cfg.block_size)
    nk, nv, nctx = oracle.commit_path(kc, vc, inp["block_table"], inp["ctx_len"], kt, vt,
                                      inp["acc_nodes"], inp["out_len"], cfg.block_size)
    for b in range(cfg.B):
        n = int(inp["out_len"][b]) - 1
        last = 0 if n == 0 else int(inp["acc_nodes"][b, n - 1])
        keys = oracle.gather_prefix(nk, inp["block_table"][b], int(nctx[b]), cfg.block_size)
        vals = oracle.gather_prefix(nv, inp["block_table"][b], int(nctx[b]), cfg.block_size)
        o2, l2 = oracle.tree_attention_node(q[b, last], keys, vals, scale)
        np.testing.assert_allclose(o2, out[b, last], rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(l2, lse[b, last], rtol=1e-13, atol=1e-13)


def test_commit_inputs_cover_edge_lengths():
    cfg = synth.get_config("7B-shape")
    cfg = synth.scaled(cfg, B=64, ctx=("uniform", 1, 40))
    inp = synth.commit_inputs(cfg, seed=0)
    assert (inp["out_len"] == 1).any() and (inp["out_len"] == cfg.depth + 1).any()
