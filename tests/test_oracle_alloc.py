"""Pins for the allocation oracle (Sec. 4.3-4.4): the contrast-graph proxy,
the vertex term's bound (App. A "Variance upper bound and convexity"), and
the design solver's optimum checked independently of the solver -- KKT
conditions, closed forms, feasible alternatives -- plus the paper's trace
bound tying the proxy to the exact HT covariance of the estimator oracle."""
import numpy as np
import pytest

import oracle
from oracle import alloc


def _instance(rng, g):
    p = rng.uniform(0.02, 0.98, g)
    c = rng.lognormal(np.log(1000.0), 0.8, g)
    return p, c


def test_disagreement_is_expected_squared_reward_gap():
    rng = np.random.default_rng(1)
    p = rng.random(7)
    d = alloc.disagreement(p)
    # E[(r_i - r_j)^2] for independent binary rewards = p_i + p_j - 2 p_i p_j
    want = p[:, None] + p[None, :] - 2.0 * p[:, None] * p[None, :]
    np.fill_diagonal(want, 0.0)
    assert np.allclose(d, want, rtol=0, atol=1e-15)
    m = rng.random(7) + 0.5
    a = alloc.edge_proxy(p, m)
    assert np.allclose(a, want * (m[:, None] + m[None, :]) ** 2 / 4, rtol=1e-15, atol=0)


def test_vertex_term_bounds_shared_edge_cross_products():
    rng = np.random.default_rng(2)
    g, D = 7, 11
    r = rng.random(g)
    s = rng.standard_normal((g, D))
    h = {(i, j): 0.5 * (r[i] - r[j]) * (s[i] - s[j]) for i in range(g) for j in range(g) if i != j}
    a = np.zeros((g, g))
    for (i, j), v in h.items():
        a[i, j] = v @ v
    b = alloc.vertex_term(a)
    for i in range(g):
        cross = sum(abs(h[i, j] @ h[i, k]) for j in range(g) for k in range(j + 1, g)
                    if i not in (j, k))
        assert 2.0 * cross <= b[i] * (1 + 1e-12)
        assert b[i] >= 0.0


def test_proxy_bounds_the_exact_ht_covariance():
    """With a_ij = ||h_ij||^2 the design objective bounds M^2 tr Cov(g_PAIR)
    for any probabilities (the covariance from the estimator oracle)."""
    rng = np.random.default_rng(3)
    g, D = 6, 9
    r = rng.random(g).astype(np.float32)
    s = rng.standard_normal((g, D)).astype(np.float32)
    rd, sd = r.astype(np.float64), s.astype(np.float64)
    a = np.zeros((g, g))
    for i in range(g):
        for j in range(g):
            if i != j:
                hv = 0.5 * (rd[i] - rd[j]) * (sd[i] - sd[j])
                a[i, j] = hv @ hv
    b = alloc.vertex_term(a)
    M = g * (g - 1) / 2
    for _ in range(5):
        pi = (rng.integers(8, 65, size=g) / 64.0).astype(np.float32)
        ex = oracle.audit_exact(np.array([0, g]), s, r, pi)
        assert M * M * ex["mse"][0] <= alloc.objective_pi(pi.astype(np.float64), a, b) * (1 + 1e-12)


@pytest.mark.parametrize("g", [4, 16, 64])
def test_solver_satisfies_kkt(g):
    rng = np.random.default_rng(10 + g)
    for ratio in (0.25, 0.5, 0.75):
        p, c = _instance(rng, g)
        budget = ratio * c.sum()
        out = alloc.solve(p, c, budget, 0.08)
        pi = out["pi"]
        assert np.all(pi >= 0.08 * (1 - 1e-12)) and np.all(pi <= 1 + 1e-12)
        assert c @ pi <= budget * (1 + 1e-8)
        assert out["success"]
        res, lam = alloc.kkt_residual(pi, out["a"], out["b"], c, budget, 0.08)
        assert res <= 2e-6, (ratio, res)
        assert lam >= 0.0


def test_two_vertices_closed_form():
    # One edge, b = 0: maximise pi_1 pi_2 under c_1 pi_1 + c_2 pi_2 = budget.
    p = np.array([0.3, 0.6])
    c = np.array([1000.0, 3000.0])
    budget = 1500.0
    out = alloc.solve(p, c, budget, 0.05)
    assert np.allclose(out["pi"], budget / (2 * c), rtol=1e-6)


def test_symmetric_graph_gives_the_uniform_design():
    g = 12
    out = alloc.solve(np.full(g, 0.4), np.full(g, 800.0), 0.37 * g * 800.0, 0.08)
    assert np.allclose(out["pi"], 0.37, rtol=1e-7)


def test_slack_and_tight_budgets():
    rng = np.random.default_rng(4)
    p, c = _instance(rng, 9)
    assert np.all(alloc.solve(p, c, 1.01 * c.sum(), 0.08)["pi"] == 1.0)
    assert np.allclose(alloc.solve(p, c, 0.08 * c.sum(), 0.08)["pi"], 0.08)
    with pytest.raises(ValueError):
        alloc.solve(p, c, 0.05 * c.sum(), 0.08)


def test_optimum_beats_feasible_alternatives():
    rng = np.random.default_rng(5)
    for g in (8, 16):
        p, c = _instance(rng, g)
        budget = 0.5 * c.sum()
        best = alloc.solve(p, c, budget, 0.08)
        uni = alloc.solve(p, c, budget, 0.08, design=alloc.UNIFORM)
        pw = alloc.solve(p, c, budget, 0.08, design=alloc.POINTWISE)
        assert best["objective"] <= uni["objective"] * (1 + 1e-10)
        assert best["objective"] <= pw["objective"] * (1 + 1e-10)
        for _ in range(200):   # random feasible points never do better
            q = np.clip(best["pi"] * np.exp(0.2 * rng.standard_normal(g)), 0.08, 1.0)
            q *= min(1.0, budget / (c @ q))
            q = np.clip(q, 0.08, 1.0)
            if c @ q <= budget * (1 - 1e-7):
                assert alloc.objective_pi(q, best["a"], best["b"]) >= best["objective"] * (1 - 1e-9)


def test_pointwise_design_is_water_filling():
    rng = np.random.default_rng(6)
    p, c = _instance(rng, 10)
    budget = 0.4 * c.sum()
    pi = alloc.solve(p, c, budget, 0.08, design=alloc.POINTWISE)["pi"]
    v = p * (1 - p)
    # pi_i = clip(sqrt(v_i / (lam c_i)), pi_min, 1) for one lam, spending the budget
    inner = (pi > 0.08 * (1 + 1e-6)) & (pi < 1 - 1e-6)
    lam = np.median(v[inner] / (c[inner] * pi[inner] ** 2))
    assert np.allclose(pi, np.clip(np.sqrt(v / (lam * c)), 0.08, 1.0), rtol=1e-5)
    assert abs(c @ pi - budget) <= 1e-8 * budget


def test_uniform_design_spends_the_budget():
    rng = np.random.default_rng(7)
    p, c = _instance(rng, 10)
    pi = alloc.solve(p, c, 0.3 * c.sum(), 0.08, design=alloc.UNIFORM)["pi"]
    assert np.allclose(pi, 0.3) and abs(c @ pi - 0.3 * c.sum()) <= 1e-9 * c.sum()
