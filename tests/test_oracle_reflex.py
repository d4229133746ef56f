"""Pins of the Reflex feedback oracle (Sec. 3.3; Sec. 3.4 Eq. (support) to Eq. (ema); App. A.1
Prop. "Pointwise surrogate representation"; App. A.2 Eq. (analysis-ema-unrolled),
Eq. (analysis-effective-age), Eq. (analysis-weight-mass); App. C "Verifier-derived feedback")."""
import itertools

import numpy as np
import pytest
import torch

import oracle


def _record(seed, V=40, d=8, K=4, tau=1.0, spread=2.0):
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((V, d))
    z0 = rng.standard_normal(d)
    q_logits = W @ z0
    p_logits = rng.standard_normal(V) * spread
    # candidates: the proposal's own top-K shifted by one rank, so that O is not empty in general
    cand = oracle.top_list(q_logits, K + 1)[1:].tolist()
    y_star = int(rng.integers(0, V))
    return W, z0, q_logits, p_logits, cand, y_star


@pytest.mark.parametrize("seed,tau", [(0, 1.0), (1, 0.7), (2, 1.3)])
def test_dist_direction_is_scaled_negative_kl_gradient(seed, tau):
    """Eq. (analysis-dist-gradient): r_dist = -tau * grad_z KL(p_S || softmax(W_S z / tau)) at z0."""
    W, z0, q_logits, p_logits, cand, y = _record(seed, tau=tau)
    f = oracle.feedback(p_logits, q_logits, cand, y, W, temperature=tau, support=12)
    S = f["support"]
    p = np.exp(p_logits / tau - (p_logits / tau).max())
    p /= p.sum()
    pS = torch.tensor(p[S] / p[S].sum(), dtype=torch.float64)
    z = torch.tensor(z0, dtype=torch.float64, requires_grad=True)
    WS = torch.tensor(W[S], dtype=torch.float64)
    logq = torch.log_softmax(WS @ z / tau, dim=0)
    kl = (pS * (torch.log(pS) - logq)).sum()
    kl.backward()
    np.testing.assert_allclose(f["r_dist"], -tau * z.grad.numpy(), rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("seed,gamma", [(3, 0.0), (4, 0.2), (5, -1.5)])
def test_cov_direction_is_negative_surrogate_gradient(seed, gamma):
    """Eq. (analysis-cov-gradient) with omega_y = p_S(y) and equal weights over the boundary set."""
    W, z0, q_logits, p_logits, cand, y = _record(seed, K=6)
    f = oracle.feedback(p_logits, q_logits, cand, y, W, support=20)
    S, O, Bset = f["support"], f["O"], f["boundary"]
    assert O, "the case must have omitted target-important tokens"
    p = np.exp(p_logits - p_logits.max())
    pS = p[S] / p[S].sum()
    Wt = torch.tensor(W, dtype=torch.float64)
    z = torch.tensor(z0, dtype=torch.float64, requires_grad=True)
    loss = torch.zeros((), dtype=torch.float64)
    for yy in O:
        for b in Bset:
            c0 = gamma + float(W[b] @ z0 - W[yy] @ z0)
            kappa = pS[S.index(yy)] / len(Bset) / (1.0 / (1.0 + np.exp(-c0)))
            c = gamma + Wt[b] @ z - Wt[yy] @ z
            loss = loss + kappa * torch.nn.functional.softplus(c)
    loss.backward()
    np.testing.assert_allclose(f["r_cov"], -z.grad.numpy(), rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_gap_decomposition_and_brute_force_ceiling(seed):
    """Eq. (optimal-candidates) by enumeration of every K-subset, Eq. (conditional-overlap) and the exact
    decomposition Eq. (acceptance-gap-decomposition)."""
    rng = np.random.default_rng(100 + seed)
    V, K = 9, 3
    p_logits = rng.standard_normal(V) * 1.5
    q_logits = rng.standard_normal(V) * 1.5
    cand = rng.choice(V, K, replace=False).tolist()
    W = rng.standard_normal((V, 5))
    f = oracle.feedback(p_logits, q_logits, cand, 0, W, support=9)
    p = np.exp(p_logits - p_logits.max()); p /= p.sum()
    q = np.exp(q_logits - q_logits.max()); q /= q.sum()
    best = max(p[list(A)].sum() for A in itertools.combinations(range(V), K))
    assert f["p_star"] == pytest.approx(best, rel=1e-14)
    pC, qC = p[cand] / p[cand].sum(), q[cand] / q[cand].sum()
    omega = np.minimum(pC, qC).sum()
    assert f["tv_c"] == pytest.approx(1.0 - omega, abs=1e-14)
    assert best - p[cand].sum() * omega == pytest.approx(f["d_dist"] + f["d_cov"], abs=1e-14)
    assert f["d_cov"] >= -1e-15 and f["d_dist"] >= 0.0


def test_support_order_dedup_and_cap():
    # candidates, then Top_K(p), then y*, then alternately the next of Top_k(p) and of Top_k(q)
    S = oracle.build_support([5, 9], [9, 2, 7, 1], [3, 5, 8], 4, K=2, cap=7)
    assert S == [5, 9, 2, 4, 7, 3, 1]
    assert oracle.build_support([5, 9], [9, 2, 7, 1], [3, 5, 8], 4, K=2, cap=3) == [5, 9, 2]
    assert oracle.build_support([5], [5, 6], [6, 5], 5, K=1, cap=10) == [5, 6]


def test_top_list_ties_to_lower_id():
    assert oracle.top_list(np.array([1.0, 3.0, 3.0, 2.0, 3.0]), 4).tolist() == [1, 2, 4, 3]


def test_special_cases():
    rng = np.random.default_rng(7)
    V, d = 30, 6
    W = rng.standard_normal((V, d))
    lg = rng.standard_normal(V) * 2
    top = oracle.top_list(lg, 4).tolist()
    # proposal equal to the target and candidates equal to the target's top-K: no feedback at all
    f = oracle.feedback(lg, lg, top, top[0], W, support=10)
    assert f["tv_s"] == pytest.approx(0.0, abs=1e-15) and f["d_dist"] == pytest.approx(0.0, abs=1e-15)
    assert f["d_cov"] == 0.0 and f["O"] == []
    assert np.abs(f["r_dist"]).max() < 1e-14 and not f["r_cov"].any()
    assert np.abs(f["e"]).max() < 1e-8
    # the combined feedback has RMS d_dist + d_cov (up to eps)
    f = oracle.feedback(lg, rng.standard_normal(V) * 2, top[1:] + [top[-1] + 1 if top[-1] + 1 < V else 0], 3, W)
    assert oracle.reflex.rms(f["e"]) == pytest.approx(f["d_dist"] + f["d_cov"], rel=1e-5)


@pytest.mark.parametrize("rho", [0.85, 0.9, 0.95])
def test_ema_unrolled_and_weight_closed_forms(rho):
    """Eq. (analysis-ema-unrolled): from zero, H updates give (1 - rho) sum_j rho^j X_{t-j}; the implied
    normalised weights have the closed forms Eq. (analysis-effective-age) and Eq. (analysis-weight-mass)."""
    rng = np.random.default_rng(int(rho * 100))
    H, d0 = 7, 3
    X = rng.standard_normal((H, 5))
    m = np.zeros(5)
    for s in range(H):
        m = oracle.ema_update(m, X[s], rho)
    expect = (1 - rho) * sum(rho ** j * X[H - 1 - j] for j in range(H))
    np.testing.assert_allclose(m, expect, rtol=1e-13)
    # weights of each record, read off by feeding unit impulses through the recursion
    a = []
    for j in range(H):
        m = np.zeros(1)
        for s in range(H):
            m = oracle.ema_update(m, np.array([1.0 if s == H - 1 - j else 0.0]), rho)
        a.append(m[0] / (1 - rho ** H))
    a = np.array(a)
    assert a.sum() == pytest.approx(1.0, rel=1e-13)
    ell = (a * (d0 + np.arange(H))).sum()
    assert ell == pytest.approx(d0 + rho / (1 - rho) - H * rho ** H / (1 - rho ** H), rel=1e-12)
    nu = (a ** 2).sum()
    assert nu == pytest.approx((1 - rho) ** 2 * (1 - rho ** (2 * H)) / ((1 - rho ** H) ** 2 * (1 - rho ** 2)),
                               rel=1e-12)


def test_batched_gate_duplicates_and_memory():
    rng = np.random.default_rng(9)
    V, d, B, H = 50, 8, 3, 2
    W = rng.standard_normal((V, d))
    p_rows = rng.standard_normal((4, V)) * 2
    q_rows = rng.standard_normal((4, V)) * 2
    q_rows[3] = p_rows[3]                       # record 3: proposal == target ...
    cand = np.full((5, 3), -1)
    cand[0, :3] = [1, 2, 3]
    cand[1, :2] = [4, 5]
    cand[2, :3] = [6, 7, 8]
    cand[3, :3] = oracle.top_list(p_rows[3], 3)  # ... and C = Top_K(p): severity = 0.7 (1 - p(C))
    cand[4, :1] = [9]
    traj = np.array([0, 1, 0, 2, 0])
    hor = np.array([1, 1, 1, 2, 2])              # record 2 repeats slot (0, 1): skipped
    mem0 = rng.standard_normal((B, H, d))
    mem, info = oracle.reflex_feedback(p_rows, np.array([0, 1, 2, 3, 0]), q_rows, np.array([0, 1, 2, 3, 1]), cand,
                                       np.array([1, 2, 3, 4, 5]), traj, hor, W, mem0, rho=(0.85, 0.9))
    assert info[2]["applied"] == -1
    for r in (0, 1, 4):
        assert info[r]["applied"] == (1 if info[r]["severity"] >= 0.03 else 0)
    np.testing.assert_allclose(mem[0, 0], 0.85 * mem0[0, 0] + 0.15 * info[0]["e"], rtol=1e-14)
    np.testing.assert_allclose(mem[0, 1], 0.9 * mem0[0, 1] + 0.1 * info[4]["e"], rtol=1e-14)
    # the high-mass record: severity below w_min only when the candidates hold > 1 - 0.03/0.7 of p
    p3 = np.exp(p_rows[3] - p_rows[3].max()); p3 /= p3.sum()
    assert info[3]["severity"] == pytest.approx(0.7 * (1 - p3[cand[3]].sum()), abs=1e-14)
    np.testing.assert_array_equal(mem[1, 1], mem0[1, 1])
    np.testing.assert_array_equal(mem[2, 0], mem0[2, 0])


def test_low_severity_record_leaves_memory():
    V, d = 20, 4
    W = np.eye(V, d)
    lg = np.full(V, -30.0)
    lg[:3] = [5.0, 4.0, 3.0]                     # the three candidates hold all but ~1e-14 of the mass
    mem0 = np.ones((1, 1, d))
    mem, info = oracle.reflex_feedback(lg[None], np.array([0]), lg[None], np.array([0]), np.array([[0, 1, 2]]),
                                       np.array([0]), np.array([0]), np.array([1]), W, mem0, rho=(0.85,))
    assert info[0]["severity"] < 0.03 and info[0]["applied"] == 0
    np.testing.assert_array_equal(mem, mem0)


# ----------------------------------------------------------------------------- reliability gate
def test_moments_match_two_pass_statistics():
    """The one-pass moments against numpy's two-pass mean and sample variance."""
    a = np.random.default_rng(3).uniform(-1, 1, 37)
    st = (0, 0.0, 0.0)
    for k, x in enumerate(a, 1):
        st = oracle.moments_update(st, x)
        assert st[0] == k
        assert st[1] == pytest.approx(a[:k].mean(), abs=1e-14)
        if k >= 2:
            assert st[2] / (k - 1) == pytest.approx(a[:k].var(ddof=1), rel=1e-12)


def test_reliability_score_hand_example():
    # alignments 0.5, 0.7, 0.9: mean 0.7, sample std 0.2, n = 3
    st = (0, 0.0, 0.0)
    for x in (0.5, 0.7, 0.9):
        st = oracle.moments_update(st, x)
    assert oracle.reliability(st, 0.6) == pytest.approx(0.7 - 0.6 * 0.2 / np.sqrt(3), rel=1e-12)
    assert oracle.reliability(oracle.moments_update((0, 0.0, 0.0), 0.3), 0.6) is None


def test_sketch_is_unit_and_scale_invariant():
    rng = np.random.default_rng(4)
    P = rng.standard_normal((24, 40))
    x = rng.standard_normal(40)
    s = oracle.sketch(x, P)
    assert np.linalg.norm(s) == pytest.approx(1.0, rel=1e-14)
    np.testing.assert_allclose(oracle.sketch(3.5 * x, P), s, rtol=1e-13)
    np.testing.assert_allclose(oracle.sketch(-x, P), -s, rtol=1e-13)
    assert oracle.sketch(np.zeros(40), P) is None


def _reliable_stats(n=50, mean=0.6, spread=0.1):
    st = (0, 0.0, 0.0)
    for k in range(n):
        st = oracle.moments_update(st, mean + spread * (1 if k % 2 else -1))
    return st


def test_correction_magnitude_direction_and_gates():
    """Eq. (reflex-correction): dz = alpha RMS(z) m / (RMS(m) + eps), alpha spanned by Rel; every gate
    condition switches it off."""
    rng = np.random.default_rng(5)
    z, m = rng.standard_normal(64), rng.standard_normal(64) * 0.3
    st = _reliable_stats()
    rel = oracle.reliability(st, 0.6)
    zc, alpha, r = oracle.correction(z, m, st, n_fb=5, a_min=0.01, a_max=0.025, n_fb_min=1, n_align_min=6)
    assert r == pytest.approx(rel) and alpha == pytest.approx(0.01 + 0.015 * rel)
    dz = zc - z
    np.testing.assert_allclose(dz / np.linalg.norm(dz), m / np.linalg.norm(m), rtol=1e-12)
    rms = lambda v: np.sqrt(np.mean(v * v))  # noqa: E731
    assert rms(dz) == pytest.approx(alpha * rms(z) * rms(m) / (rms(m) + 1e-6), rel=1e-12)
    # the shadow correction of App. E, Eq. (shadow-correction), has the same form with a fixed ratio
    zs, a_s, _ = oracle.correction(z, m, st, n_fb=5, a_min=0.005, a_max=0.005, n_fb_min=1, n_align_min=6)
    np.testing.assert_allclose(zs, z + 0.005 * rms(z) * m / (rms(m) + 1e-6), rtol=1e-13)
    off = [dict(n_fb=0), dict(n_align_min=51), dict(st=_reliable_stats(mean=-0.2)), dict(m=np.zeros(64))]
    for o in off:
        args = dict(z=z, m=m, st=st, n_fb=5, a_min=0.01, a_max=0.025, n_fb_min=1, n_align_min=6)
        args.update(o)
        zc, alpha, _ = oracle.correction(args["z"], args["m"], args["st"], args["n_fb"], args["a_min"],
                                         args["a_max"], args["n_fb_min"], args["n_align_min"])
        assert alpha == 0.0 and np.array_equal(zc, z)


def test_feedback_alignment_observations():
    rng = np.random.default_rng(6)
    V, d, B, H = 60, 16, 2, 2
    W = rng.standard_normal((V, d))
    P = rng.standard_normal((24, d))
    p_rows, q_rows = rng.standard_normal((3, V)) * 2, rng.standard_normal((3, V)) * 2
    cand = np.array([[1, 2, -1], [3, 4, 5], [6, -1, -1]])
    s_rec = np.zeros((3, 24))
    s_rec[0] = oracle.sketch(rng.standard_normal(d), P)
    s_rec[2] = oracle.sketch(rng.standard_normal(d), P)       # record 1 has no stored sketch
    align0 = np.zeros((B, H, 4))
    mem, info, al = oracle.reflex_feedback(p_rows, np.arange(3), q_rows, np.arange(3), cand, np.array([7, 8, 9]),
                                           np.array([0, 1, 0]), np.array([1, 1, 2]), W, np.zeros((B, H, d)),
                                           rho=(0.85, 0.9), P=P, rec_sketch=s_rec, align=align0)
    assert all(f["applied"] == 1 for f in info)
    a0 = float(s_rec[0] @ oracle.sketch(info[0]["e"], P))
    assert info[0]["alignment"] == pytest.approx(a0, rel=1e-14) and "alignment" not in info[1]
    np.testing.assert_allclose(al[0, 0], [1, a0, 0.0, 1])
    np.testing.assert_allclose(al[1, 0], [0, 0.0, 0.0, 1])
    assert al[0, 1, 0] == 1 and al[0, 1, 3] == 1
