"""Pins of the acceptance oracle (App. B.2 Eq. (nodeaccept), Eq. (noderesidual), Alg. "Exact node-wise tree
verification"; App. B.3 Prop. "One-node correction", Thm. "Exact target continuation"; App. A Prop.
"Candidate-support acceptance certificate" and the support-mismatch worked example; App. B.4 Eq.
(verifier-sandwich))."""
import itertools
import json
import math
import os
from concurrent.futures import ProcessPoolExecutor
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "support_mismatch.json")


def _run_node(p, cand_tokens, draft_w, n_draws, seed):
    """Root with one leaf child per candidate; returns (first-slot accepted, any accepted, emitted token) per draw."""
    V = len(p)
    m = len(cand_tokens)
    parents = np.array([-1] + [0] * m)
    head = np.full((1, V), -1e30)                    # head logits: support only on the candidates
    head[0, cand_tokens] = np.log(draft_w)
    rng = np.random.default_rng(seed)
    tl = np.tile(np.log(np.asarray(p, dtype=np.float64)), (m + 1, 1))
    out = np.zeros((n_draws, 3), dtype=np.int64)
    for n in range(n_draws):
        u = synth.uniforms(rng, (2 * (m + 1) + 1,))
        tok, cl, _ = oracle.tree_build(head[None], parents[None], np.array([0]), u[None, :m + 1])
        res = oracle.tree_accept_one(tl, cl[0], tok[0], parents, u[m + 1:2 * (m + 1)], float(u[-1]))
        first = 1 if res["acc_nodes"][:1] == [1] else 0
        out[n] = (first, 1 if res["acc_nodes"] else 0, res["out_tokens"][0])
    return out


def test_support_mismatch_worked_example():
    g = json.load(open(GOLDEN))
    p = [float(Fraction(x)) for x in g["p"]]
    C = g["C"]
    for ukey, qkey, akey in (("u", "q_C", "A1_q"), ("u_prime", "q_C_prime", "A1_q_prime")):
        u = [float(Fraction(x)) for x in g[ukey]]
        w = [u[c] for c in C]
        # the draft law restricted to C is the paper's q_C
        np.testing.assert_allclose(np.asarray(w) / sum(w), [float(Fraction(x)) for x in g[qkey]], rtol=1e-15)
        N = 40000
        res = _run_node(p, C, w, N, seed={"u": 101, "u_prime": 202}[ukey])
        A1 = float(Fraction(g[akey]))
        se = math.sqrt(A1 * (1 - A1) / N)
        assert abs(res[:, 0].mean() - A1) < 4.5 * se, (ukey, res[:, 0].mean(), A1)
        # trying every candidate of C (m_u = |C|) makes node acceptance exactly p(C) = 3/5 for both drafts
        pC = p[0] + p[2]
        assert abs(res[:, 1].mean() - pC) < 4.5 * math.sqrt(pC * (1 - pC) / N)
        # and the emitted token follows p
        obs = np.bincount(res[:, 2], minlength=3)
        assert stats.chisquare(obs, np.asarray(p) * N).pvalue > 0.01


def test_single_candidate_hand_thresholds():
    # p = (.5, .3, .2); one child (token 0) so q is a point mass and A = min(1, .5 / 1) = .5.
    tl = np.tile(np.log([0.5, 0.3, 0.2]), (2, 1))
    parents = np.array([-1, 0])
    tokens = np.array([2, 0])
    cl = np.array([0.0, 1.7])
    acc = lambda U, uf: oracle.tree_accept_one(tl, cl, tokens, parents, np.array([0.0, U]), uf)
    r = acc(0.49, 0.45)
    assert r["acc_nodes"] == [1] and r["kind"] == oracle.BONUS
    assert r["out_tokens"] == [0, 0]                 # bonus from the leaf's p: .45 < .5 -> token 0
    # rejected: residual [p - q]_+ / Z = (0, .6, .4); inverse CDF: U*1 < .6 -> token 1, else token 2
    r = acc(0.51, 0.5)
    assert r["acc_nodes"] == [] and r["kind"] == oracle.FALLBACK and r["out_tokens"] == [1]
    r = acc(0.51, 0.7)
    assert r["out_tokens"] == [2]
    # bonus draw at the leaf uses the leaf's p: U = .3 -> .3 < .5 -> token 0; U = .6 -> token 1; U = .9 -> 2
    assert acc(0.2, 0.3)["out_tokens"] == [0, 0]
    assert acc(0.2, 0.6)["out_tokens"] == [0, 1]
    assert acc(0.2, 0.9)["out_tokens"] == [0, 2]


def test_inverse_cdf_hand_values():
    r = np.array([0.0, 0.25, 0.0, 0.75])
    assert oracle.inverse_cdf(r, 0.1)[0] == 1
    assert oracle.inverse_cdf(r, 0.25)[0] == 3        # U*S == boundary -> next token (strict '<')
    assert oracle.inverse_cdf(r, 0.999)[0] == 3
    v, mg = oracle.inverse_cdf(r, 0.2)
    assert v == 1 and abs(mg - 0.05) < 1e-15


def _exact_node_law(p, cand, w):
    """Exact law of (slot accepted or 0 for fallback, emitted token) for one node, from the paper's formulas,
    enumerating every ordered child list (Eq. (childlist)) in rational arithmetic."""
    V = len(p)
    law = {}
    for order in itertools.permutations(range(len(cand))):
        pr_order = Fraction(1)
        rem = list(range(len(cand)))
        for i in order:
            pr_order *= w[i] / sum(w[j] for j in rem)
            rem.remove(i)
        r = list(p)
        reach = pr_order
        rem = list(range(len(cand)))
        for j, i in enumerate(order):
            tot = sum(w[k] for k in rem)
            q = [Fraction(0)] * V
            for k in rem:
                q[cand[k]] = w[k] / tot
            y = cand[i]
            A = min(Fraction(1), r[y] / q[y])
            law[(j + 1, y)] = law.get((j + 1, y), 0) + reach * A
            reach *= 1 - A
            pos = [max(r[v] - q[v], Fraction(0)) for v in range(V)]
            Z = sum(pos)
            r = [x / Z for x in pos] if Z > 0 else pos
            rem.remove(i)
        for v in range(V):
            if r[v]:
                law[(0, v)] = law.get((0, v), 0) + reach * r[v]
    return law


def test_brute_force_one_node_exact_and_oracle_matches():
    p = [Fraction(1, 2), Fraction(1, 4), Fraction(1, 8), Fraction(1, 8)]
    cand = [1, 0, 3]
    w = [Fraction(3), Fraction(2), Fraction(1)]
    law = _exact_node_law(p, cand, w)
    # Prop. "One-node correction": the emitted token is distributed exactly as p
    for v in range(4):
        assert sum(pr for (s, t), pr in law.items() if t == v) == p[v]
    # the oracle's joint (slot, token) frequencies match the enumerated law
    N = 30000
    tl = np.tile(np.log([float(x) for x in p]), (len(cand) + 1, 1))
    parents = np.array([-1] + [0] * len(cand))
    head = np.full((1, 1, 4), -1e30)
    head[0, 0, cand] = np.log([float(x) for x in w])
    rng = np.random.default_rng(21)
    counts = {}
    for n in range(N):
        u = synth.uniforms(rng, (2 * len(cand) + 3,))
        tok, cl, _ = oracle.tree_build(head, parents[None], np.array([0]), u[None, :len(cand) + 1])
        res = oracle.tree_accept_one(tl, cl[0], tok[0], parents, u[len(cand) + 1:2 * len(cand) + 2], float(u[-1]))
        slot = res["acc_nodes"][0] if res["acc_nodes"] else 0     # children 1..m are slots 1..m
        key = (slot, res["out_tokens"][0])
        counts[key] = counts.get(key, 0) + 1
    keys = sorted(k for k in law if law[k] > 0)
    assert set(counts) <= set(keys)
    exp = np.array([float(law[k]) * N for k in keys])
    obs = np.array([counts.get(k, 0) for k in keys])
    assert stats.chisquare(obs, exp).pvalue > 0.01


# ------------------------------------------------------------------- exactness over a two-level tree

_V = 4
_PARENTS = np.array([-1, 0, 0, 1, 1, 2])        # root: 2 slots; node 1: 2 slots; node 2: 1 slot
_ANCHOR = 0


def _ar_logits(prefix):
    """A fixed toy autoregressive target: logits depend on the whole prefix."""
    seed = 7
    for t in prefix:
        seed = seed * 31 + int(t) + 1
    return np.random.default_rng(seed).standard_normal(_V) * 1.3


def _ar_probs(prefix):
    l = _ar_logits(prefix)
    e = np.exp(l - l.max())
    return e / e.sum()


def _draws(args):
    seed, n = args
    rng = np.random.default_rng(seed)
    head = np.random.default_rng(99).standard_normal((1, 2, _V)) * 1.1   # two heads, path-independent
    T = _PARENTS.shape[0]
    depth, kids = oracle.tree_structure(_PARENTS)
    first = np.zeros(_V, dtype=np.int64)
    seq3 = np.zeros(_V ** 3, dtype=np.int64)
    for _ in range(n):
        u = synth.uniforms(rng, (2 * T + 1 + 3,))
        tok, cl, _ = oracle.tree_build(head, _PARENTS[None], np.array([_ANCHOR]), u[None, :T])
        paths = {0: (_ANCHOR,)}
        for c in range(1, T):
            paths[c] = paths[int(_PARENTS[c])] + (int(tok[0, c]),)
        tl = np.stack([_ar_logits(paths[c]) for c in range(T)])
        res = oracle.tree_accept_one(tl, cl[0], tok[0], _PARENTS, u[T:2 * T], float(u[2 * T]))
        committed = list(res["out_tokens"])
        first[committed[0]] += 1
        k = 0
        while len(committed) < 3:                     # exact autoregressive continuation
            pr = _ar_probs((_ANCHOR, *committed))
            committed.append(int(np.searchsorted(np.cumsum(pr), u[2 * T + 1 + k] * pr.sum(), side="right")))
            k += 1
        c3 = committed[:3]
        seq3[(c3[0] * _V + c3[1]) * _V + c3[2]] += 1
    return first, seq3


def test_chi_square_exactness_1e6_draws():
    n_total = 1_000_000
    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    chunks = [(1000 + i, n_total // 64) for i in range(64)]
    first = np.zeros(_V, dtype=np.int64)
    seq3 = np.zeros(_V ** 3, dtype=np.int64)
    with ProcessPoolExecutor(workers) as ex:
        for f, s in ex.map(_draws, chunks):
            first += f
            seq3 += s
    N = first.sum()
    assert stats.chisquare(first, _ar_probs((_ANCHOR,)) * N).pvalue > 0.01
    exp = np.zeros(_V ** 3)
    for a, b, c in itertools.product(range(_V), repeat=3):
        exp[(a * _V + b) * _V + c] = (_ar_probs((_ANCHOR,))[a] * _ar_probs((_ANCHOR, a))[b]
                                      * _ar_probs((_ANCHOR, a, b))[c])
    assert abs(exp.sum() - 1) < 1e-12
    assert stats.chisquare(seq3, exp * N).pvalue > 0.01


def test_first_slot_closed_form_and_sandwich():
    # A_1 = sum_v min(p(v), q_C(v)) (App. A) and p(C) * Omega_C <= A_ver <= p(C) (App. B.4),
    # on random instances with a strict subset C of the vocabulary
    rng = np.random.default_rng(5)
    for trial in range(4):
        V = 6
        p = rng.dirichlet(np.ones(V))
        C = rng.choice(V, size=3, replace=False)
        w = rng.uniform(0.2, 2.0, size=3)
        N = 20000
        res = _run_node(p, C, w, N, seed=100 + trial)
        qC = np.zeros(V)
        qC[C] = w / w.sum()
        A1 = np.minimum(p, qC).sum()
        assert abs(res[:, 0].mean() - A1) < 4.5 * math.sqrt(A1 * (1 - A1) / N)
        pC = p[C].sum()
        omega = np.minimum(p[C] / pC, w / w.sum()).sum()
        acc = res[:, 1].mean()
        tol = 4.5 * math.sqrt(0.25 / N)
        assert pC * omega - tol <= acc <= pC + tol


# ------------------------------------------------------------------- nucleus truncation of the target law
def test_nucleus_hand_examples():
    lg = np.log([0.5, 0.3, 0.15, 0.05])
    p, _ = oracle.accept._target_dist(lg, 1.0, 0.79)       # mass before: 0, 0.5, 0.8 -> keep 2
    np.testing.assert_allclose(p, [0.625, 0.375, 0.0, 0.0], rtol=1e-14)
    p, _ = oracle.accept._target_dist(lg, 1.0, 0.81)       # 0.8 < 0.81 -> keep 3
    np.testing.assert_allclose(p, [0.5 / 0.95, 0.3 / 0.95, 0.15 / 0.95, 0.0], rtol=1e-14)
    # ties rank the lower id first: four equal logits, top_p 0.5 keeps ids 0 and 1
    p, _ = oracle.accept._target_dist(np.zeros(4), 1.0, 0.5)
    np.testing.assert_allclose(p, [0.5, 0.5, 0.0, 0.0], rtol=1e-14)
    p, _ = oracle.accept._target_dist(np.array([0.0, 2.0, 0.0, 2.0]), 1.0, 0.6)
    np.testing.assert_array_equal(p > 0, [False, True, False, True])
    # top_p = 1 is the plain softmax
    p1, m1 = oracle.accept._target_dist(lg, 1.0, 1.0)
    np.testing.assert_allclose(p1, [0.5, 0.3, 0.15, 0.05], rtol=1e-14)
    assert m1 == np.inf


@pytest.mark.parametrize("seed", range(5))
def test_nucleus_smallest_ranked_prefix(seed):
    rng = np.random.default_rng(seed)
    V = 40
    lg = np.round(rng.standard_normal(V) * 2, 1)          # rounded: ties occur
    base = np.exp(lg - lg.max())
    base /= base.sum()
    rank = sorted(range(V), key=lambda v: (-lg[v], v))
    prev = 0
    for top_p in (0.3, 0.6, 0.9, 0.95, 0.999):
        p, _ = oracle.accept._target_dist(lg, 1.0, top_p)
        kept = [v for v in rank if p[v] > 0]
        n = len(kept)
        assert kept == rank[:n]                            # a prefix of the ranking
        assert base[kept].sum() >= top_p - 1e-12           # reaches top_p ...
        assert base[kept[:-1]].sum() < top_p               # ... and no shorter prefix does
        np.testing.assert_allclose(p[kept], base[kept] / base[kept].sum(), rtol=1e-13)
        assert n >= prev                                   # grows with top_p
        prev = n


def test_nucleus_one_node_exactness():
    """The committed token of one node follows the truncated target law (the exactness argument holds for
    any target distribution): p = (1/2, 1/4, 1/8, 1/8) at top_p 0.7 keeps tokens 0 and 1 with (2/3, 1/3)."""
    p = [0.5, 0.25, 0.125, 0.125]
    cand = [1, 2, 3]
    w = [3.0, 2.0, 1.0]
    N = 30000
    tl = np.tile(np.log(p), (len(cand) + 1, 1))
    parents = np.array([-1] + [0] * len(cand))
    head = np.full((1, 1, 4), -1e30)
    head[0, 0, cand] = np.log(w)
    rng = np.random.default_rng(23)
    counts = np.zeros(4)
    for n in range(N):
        u = synth.uniforms(rng, (2 * len(cand) + 3,))
        tok, cl, _ = oracle.tree_build(head, parents[None], np.array([0]), u[None, :len(cand) + 1])
        res = oracle.tree_accept_one(tl, cl[0], tok[0], parents, u[len(cand) + 1:2 * len(cand) + 2], float(u[-1]),
                                     top_p=0.7)
        counts[res["out_tokens"][0]] += 1
    assert counts[2] == 0 and counts[3] == 0
    assert stats.chisquare(counts[:2], np.array([2 / 3, 1 / 3]) * N).pvalue > 0.01
