"""Pins of the tree-build oracle (App. B.1, Eq. (slotq), Eq. (childlist))."""
import itertools
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import oracle
import synth


def test_tree_structure_config0():
    depth, kids = oracle.tree_structure(np.array([-1, 0, 0, 1, 1, 2, 3, 4]))
    assert depth.tolist() == [0, 1, 1, 2, 2, 2, 3, 3]
    assert kids == [[1, 2], [3, 4], [5], [6], [7], [], [], []]


@pytest.mark.parametrize("bad", [[0, 0], [-1, 1], [-1, 0, 3, 0], [-1, -1]])
def test_tree_structure_rejects_non_topological(bad):
    with pytest.raises(ValueError):
        oracle.tree_structure(np.array(bad))


def test_top_m_ties_break_to_lower_id():
    row = np.array([1.0, 3.0, 3.0, 2.0, 3.0, -1.0])
    assert oracle.top_m(row, 3).tolist() == [1, 2, 4]
    assert oracle.top_m(row, 4).tolist() == [1, 2, 4, 3]


def test_sample_hand_thresholds():
    # weights 3:1 -> cumulative (3, 4). U*4 < 3 picks the first candidate.
    ids = np.array([7, 9])
    lg = np.log([3.0, 1.0])
    assert oracle.sample_ordered_children(ids, lg, [0.5, 0.5])[0] == [7, 9]
    assert oracle.sample_ordered_children(ids, lg, [0.8, 0.5])[0] == [9, 7]
    # exactly on the boundary (U*S == 3) goes to the next candidate (strict '<')
    assert oracle.sample_ordered_children(ids, lg, [0.75, 0.1])[0] == [9, 7]


def _succ_prob(weights, order):
    """Successive-sampling probability of an ordered list, in exact rationals."""
    w = [Fraction(x) for x in weights]
    rem = list(range(len(w)))
    pr = Fraction(1)
    for i in order:
        pr *= w[i] / sum(w[j] for j in rem)
        rem.remove(i)
    return pr


def test_child_order_law_chi_square():
    # three candidates with weights 3:2:1; all 6 orders, frequencies vs successive sampling
    rng = np.random.default_rng(11)
    ids = np.arange(3)
    lg = np.log([3.0, 2.0, 1.0])
    N = 60000
    us = synth.uniforms(rng, (N, 3))
    counts = {}
    for n in range(N):
        order = tuple(oracle.sample_ordered_children(ids, lg, us[n])[0])
        counts[order] = counts.get(order, 0) + 1
    perms = list(itertools.permutations(range(3)))
    exp = np.array([float(_succ_prob([3, 2, 1], p)) for p in perms]) * N
    obs = np.array([counts.get(p, 0) for p in perms])
    assert abs(sum(float(_succ_prob([3, 2, 1], p)) for p in perms) - 1) < 1e-15
    assert stats.chisquare(obs, exp).pvalue > 0.01


def test_tree_build_uses_depth_head_and_topm_support():
    # V=6, H=2. Root children (depth-0 node -> head 1), grandchildren from head 2, deeper ones reuse head 2.
    parents = np.array([[-1, 0, 0, 1, 3]])
    logits = np.zeros((1, 2, 6))
    logits[0, 0] = [0, 5, 1, 4, -2, 0]     # head 1 top-2 support {1, 3}
    logits[0, 1] = [9, 0, 0, 0, 0, 1]      # head 2 top-1 support {0}
    u = np.full((1, 5), 0.5, dtype=np.float32)
    tok, cl, _ = oracle.tree_build(logits, parents, np.array([2]), u)
    assert tok[0, 0] == 2
    assert set(tok[0, 1:3].tolist()) == {1, 3}
    assert tok[0, 3] == 0 and tok[0, 4] == 0   # node 4 hangs under a depth-2 node: head min(2 + 1, H) = 2
    assert cl[0, 3] == 9.0
    # e^5 : e^4 -> first slot takes token 1 when U*S < e^5, i.e. U < 0.731
    assert tok[0, 1] == 1


def test_tree_build_on_generator_topologies():
    for base in (synth.TINY_FP32, synth.SHAPE_1P5B):
        cfg = synth.scaled(base, B=3, V=300)
        inp = synth.head_logits_inputs(cfg, seed=3)
        tok, cl, _ = oracle.tree_build(inp["logits"], inp["parents"], inp["root_token"], inp["u_tree"])
        depth, kids = oracle.tree_structure(inp["parents"][0])
        for b in range(cfg.B):
            for u, ch in enumerate(kids):
                if not ch:
                    continue
                k = min(depth[u] + 1, cfg.H)
                row = inp["logits"][b, k - 1].astype(np.float64)
                got = tok[b, ch]
                assert len(set(got.tolist())) == len(ch)                  # distinct siblings
                assert sorted(got.tolist()) == sorted(oracle.top_m(row, len(ch)).tolist())
                np.testing.assert_array_equal(cl[b, ch], row[got])
