"""Pins for the oracle's edge-weight rules (the estimator variants of the
frozen-policy audit and ablation tables).  Each rule is checked against what
the paper states about it, by exhaustive enumeration of every independent
Bernoulli design outcome (exact expectations), with targets and edge terms
computed here directly from Eq. (pair-kernel):

  - unweighted (naive selection, App. A): E[g~_0] - g = (1/M) sum (rho - 1) h
  - clipped weights (App. B): bias multiplier min(1, w_max rho) - 1
  - ratio over the observed-edge count (App. A): equals the uniform pair
    average in expectation given K_E > 0 for a self-weighting design
  - self-normalised (App. B): a ratio estimator; with a constant rho it is
    the observed-edge average draw by draw
  - marginal-only (named in Tables 4 and 5 without a formula; reading: each
    half of h_ij is weighted by its own endpoint's 1/pi): its enumeration
    expectation (1/M) sum 1/2 (r_i - r_j)(pi_j s_i - pi_i s_j)
  - every rule reduces to the leave-one-out form (Theorem 1) when every
    vertex completes with rho = 1
  - ESS = (sum w)^2 / sum w^2 (App. D metrics) special cases.
"""
import itertools

import numpy as np
import pytest

import oracle

RULES = [oracle.RULE_HT, oracle.RULE_UNWEIGHTED, oracle.RULE_RATIO_KE, oracle.RULE_CLIPPED,
         oracle.RULE_SELFNORM, oracle.RULE_MARGINAL]


def _prompt(rng, g, D):
    r = rng.random(g).astype(np.float32)
    s = rng.standard_normal((g, D)).astype(np.float32)
    # multiples of 1/64 in [1/8, 1]: products p_i p_j are exact in fp32
    p = (rng.integers(8, 65, size=g) / 64.0).astype(np.float32)
    return r, s, p


def _block(p):
    blk = (p[:, None].astype(np.float64) * p[None, :].astype(np.float64)).astype(np.float32)
    np.fill_diagonal(blk, p)
    return blk


def _h(r, s, i, j):
    return 0.5 * (float(r[i]) - float(r[j])) * (s[i].astype(np.float64) - s[j].astype(np.float64))


def _target(r, s):
    g = s.shape[0]
    M = g * (g - 1) / 2
    return sum(_h(r, s, i, j) for i in range(g) for j in range(i + 1, g)) / M


def _enumerate(r, s, p, rule, wmax=0.0):
    g, D = s.shape
    masks = np.array(list(itertools.product([0, 1], repeat=g)), dtype=np.uint8)
    n = masks.shape[0]
    offsets = np.arange(0, (n + 1) * g, g, dtype=np.int64)
    out = oracle.pair_grad_rule(offsets, np.tile(s, (n, 1)), np.tile(r, n),
                                mask=masks.reshape(-1), pi=np.repeat(_block(p)[None], n, axis=0),
                                rule=rule, wmax=wmax)
    pd = p.astype(np.float64)
    probs = np.prod(np.where(masks == 1, pd[None, :], 1.0 - pd[None, :]), axis=1)
    return masks, probs, out


def _close(a, b, scale):
    return np.max(np.abs(a - b)) <= 1e-12 * max(scale, 1e-300)


@pytest.mark.parametrize("g", [3, 6, 8])
def test_unweighted_rule_bias(g):
    rng = np.random.default_rng(10 + g)
    r, s, p = _prompt(rng, g, 6)
    _, probs, out = _enumerate(r, s, p, oracle.RULE_UNWEIGHTED)
    M = g * (g - 1) / 2
    pd = p.astype(np.float64)
    bias = sum((pd[i] * pd[j] - 1.0) * _h(r, s, i, j) for i in range(g) for j in range(i + 1, g)) / M
    t = _target(r, s)
    assert _close(probs @ out["out"] - t, bias, np.abs(t).max())


@pytest.mark.parametrize("g,wmax", [(5, 2.0), (7, 5.0), (8, 10.0)])
def test_clipped_rule_multiplier(g, wmax):
    rng = np.random.default_rng(20 + g)
    r, s, p = _prompt(rng, g, 6)
    p[:2] = 0.125                                       # 1/rho_01 = 64: clipped
    _, probs, out = _enumerate(r, s, p, oracle.RULE_CLIPPED, wmax)
    M = g * (g - 1) / 2
    pd = p.astype(np.float64)
    bias = sum((min(1.0, wmax * pd[i] * pd[j]) - 1.0) * _h(r, s, i, j)
               for i in range(g) for j in range(i + 1, g)) / M
    t = _target(r, s)
    assert any(1.0 / (pd[i] * pd[j]) > wmax for i in range(g) for j in range(i + 1, g))
    assert _close(probs @ out["out"] - t, bias, np.abs(t).max())


def test_clipped_rule_above_every_weight_is_ht():
    rng = np.random.default_rng(3)
    r, s, p = _prompt(rng, 6, 4)
    _, _, ht = _enumerate(r, s, p, oracle.RULE_HT)
    _, _, cl = _enumerate(r, s, p, oracle.RULE_CLIPPED, 1e6)
    assert np.array_equal(ht["out"], cl["out"])


@pytest.mark.parametrize("g", [4, 7])
def test_ratio_rule_recovers_target_under_self_weighting_design(g):
    rng = np.random.default_rng(30 + g)
    r, s, _ = _prompt(rng, g, 5)
    p = np.full(g, 0.625, dtype=np.float32)           # constant p: self-weighting
    masks, probs, out = _enumerate(r, s, p, oracle.RULE_RATIO_KE)
    ke = masks.sum(axis=1) * (masks.sum(axis=1) - 1) // 2
    pos = ke > 0
    cond = probs[pos] @ out["out"][pos] / probs[pos].sum()
    t = _target(r, s)
    assert _close(cond, t, np.abs(t).max())
    assert np.all(out["out"][~pos] == 0.0)


def test_ratio_rule_is_not_the_target_under_unequal_design():
    rng = np.random.default_rng(41)
    r, s, p = _prompt(rng, 6, 5)
    masks, probs, out = _enumerate(r, s, p, oracle.RULE_RATIO_KE)
    pos = masks.sum(axis=1) >= 2
    cond = probs[pos] @ out["out"][pos] / probs[pos].sum()
    t = _target(r, s)
    assert np.max(np.abs(cond - t)) > 1e-3 * np.abs(t).max()


def test_selfnorm_equals_observed_edge_average_for_constant_rho():
    rng = np.random.default_rng(5)
    r, s, _ = _prompt(rng, 6, 5)
    p = np.full(6, 0.75, dtype=np.float32)
    _, _, sn = _enumerate(r, s, p, oracle.RULE_SELFNORM)
    _, _, ra = _enumerate(r, s, p, oracle.RULE_RATIO_KE)
    assert np.max(np.abs(sn["out"] - ra["out"])) <= 1e-13 * np.abs(ra["out"]).max()


def test_selfnorm_draw_by_draw_definition():
    """One draw, by hand: sum_e (I_e / rho_e) h_e / sum_e (I_e / rho_e)."""
    rng = np.random.default_rng(8)
    r, s, p = _prompt(rng, 5, 4)
    J = np.array([1, 0, 1, 1, 1], dtype=np.uint8)
    out = oracle.pair_grad_rule(np.array([0, 5]), s, r, mask=J, pi=_block(p)[None],
                                rule=oracle.RULE_SELFNORM)["out"][0]
    pd = p.astype(np.float64)
    num, den = 0.0, 0.0
    for i in range(5):
        for j in range(i + 1, 5):
            if J[i] and J[j]:
                w = 1.0 / (pd[i] * pd[j])
                num = num + w * _h(r, s, i, j)
                den += w
    assert _close(out, num / den, np.abs(out).max())


@pytest.mark.parametrize("g", [4, 7])
def test_marginal_rule_expectation(g):
    rng = np.random.default_rng(50 + g)
    r, s, p = _prompt(rng, g, 5)
    _, probs, out = _enumerate(r, s, p, oracle.RULE_MARGINAL)
    M = g * (g - 1) / 2
    pd = p.astype(np.float64)
    sd = s.astype(np.float64)
    want = sum(0.5 * (float(r[i]) - float(r[j])) * (pd[j] * sd[i] - pd[i] * sd[j])
               for i in range(g) for j in range(i + 1, g)) / M
    assert _close(probs @ out["out"], want, np.abs(want).max())
    # it is biased whenever some p < 1 (the paper's point: joint inclusion is needed)
    assert np.max(np.abs(probs @ out["out"] - _target(r, s))) > 1e-3 * np.abs(want).max()


@pytest.mark.parametrize("rule", RULES)
def test_every_rule_reduces_to_leave_one_out_when_all_complete(rule):
    rng = np.random.default_rng(60 + rule)
    g, D = 6, 5
    r, s, _ = _prompt(rng, g, D)
    out = oracle.pair_grad_rule(np.array([0, g]), s, r, rule=rule, wmax=3.0)["out"][0]
    loo = ((r.astype(np.float64) - r.astype(np.float64).mean()) / (g - 1)) @ s.astype(np.float64)
    assert _close(out, loo, np.abs(loo).max())
    co = oracle.pair_coeffs_rule(np.array([0, g]), r, rule=rule, wmax=3.0)["coeff"]
    assert np.max(np.abs(co - (r - r.astype(np.float64).mean()) / (g - 1))) <= 1e-15


@pytest.mark.parametrize("rule", RULES)
def test_coefficients_reproduce_the_rule_estimate(rule):
    rng = np.random.default_rng(70 + rule)
    sizes = [5, 2, 9, 3]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    nv, gm = int(off[-1]), max(sizes)
    r = rng.random(nv).astype(np.float32)
    s = rng.standard_normal((nv, 7)).astype(np.float32)
    p = (rng.integers(8, 65, size=nv) / 64.0).astype(np.float32)
    J = (rng.random(nv) < 0.7).astype(np.uint8)
    pi = np.zeros((len(sizes), gm, gm), dtype=np.float32)
    for b, g in enumerate(sizes):
        pi[b, :g, :g] = _block(p[off[b]:off[b + 1]])
    est = oracle.pair_grad_rule(off, s, r, mask=J, pi=pi, rule=rule, wmax=4.0)
    co = oracle.pair_coeffs_rule(off, r, mask=J, pi=pi, rule=rule, wmax=4.0)
    for b in range(len(sizes)):
        lo, hi = off[b], off[b + 1]
        via = co["coeff"][lo:hi] @ s[lo:hi].astype(np.float64)
        assert _close(via, est["out"][b], np.abs(est["out"][b]).max() + 1e-300)
    assert np.array_equal(co["edge_count"], est["edge_count"])
    assert np.allclose(co["ess"], est["ess"], rtol=1e-14)
    assert np.array_equal(co["max_weight"], est["max_weight"])


def test_ess_and_max_weight_special_cases():
    rng = np.random.default_rng(9)
    g = 6
    r, _, p = _prompt(rng, g, 1)
    pi = _block(p)[None]
    J = np.array([1, 1, 1, 0, 1, 0], dtype=np.uint8)        # K_E = 6
    un = oracle.pair_coeffs_rule(np.array([0, g]), r, mask=J, pi=pi, rule=oracle.RULE_UNWEIGHTED)
    assert un["edge_count"][0] == 6 and un["ess"][0] == 6.0 and un["max_weight"][0] == 1.0
    one = np.array([0, 1, 0, 0, 1, 0], dtype=np.uint8)      # one observed edge
    ht1 = oracle.pair_coeffs_rule(np.array([0, g]), r, mask=one, pi=pi, rule=oracle.RULE_HT)
    assert ht1["ess"][0] == 1.0
    assert ht1["max_weight"][0] == 1.0 / (float(p[1]) * float(p[4]))
    two = np.array([1, 1, 0, 0, 0, 0], dtype=np.uint8)
    J3 = np.array([1, 1, 1, 0, 0, 0], dtype=np.uint8)       # edges (0,1), (0,2), (1,2)
    ht3 = oracle.pair_coeffs_rule(np.array([0, g]), r, mask=J3, pi=pi, rule=oracle.RULE_HT)
    pd = p.astype(np.float64)
    w = [1 / (pd[0] * pd[1]), 1 / (pd[0] * pd[2]), 1 / (pd[1] * pd[2])]
    assert abs(ht3["ess"][0] - sum(w) ** 2 / sum(x * x for x in w)) <= 1e-12 * sum(w)
    assert ht3["max_weight"][0] == max(w)
    none = oracle.pair_coeffs_rule(np.array([0, g]), r, mask=np.zeros(g, np.uint8), pi=pi)
    assert none["ess"][0] == 0.0 and none["max_weight"][0] == 0.0
    assert np.all(none["coeff"] == 0.0)
    cl = oracle.pair_coeffs_rule(np.array([0, g]), r, mask=two, pi=pi, rule=oracle.RULE_CLIPPED,
                                 wmax=1.5)
    assert cl["max_weight"][0] == min(1.5, 1 / (pd[0] * pd[1]))


def test_rule_errors():
    r = np.array([0.0, 1.0, 0.5], dtype=np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.pair_coeffs_rule(np.array([0, 3]), r, rule=9)
    with pytest.raises(oracle.OracleError):
        oracle.pair_coeffs_rule(np.array([0, 3]), r, rule=oracle.RULE_CLIPPED, wmax=0.0)
    pi = _block(np.array([0.5, 0.5, 0.5], dtype=np.float32))[None].copy()
    pi[0, 1, 1] = 0.0                                         # marginal pi_1 = 0
    with pytest.raises(oracle.OracleError):
        oracle.pair_coeffs_rule(np.array([0, 3]), r, pi=pi, rule=oracle.RULE_MARGINAL)


def test_audit_rules_agree_with_equivalent_estimators():
    rng = np.random.default_rng(12)
    sizes = [6, 4, 8]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    nv = int(off[-1])
    r = rng.random(nv).astype(np.float32)
    s = rng.standard_normal((nv, 16)).astype(np.float32)
    p = rng.uniform(0.2, 1.0, nv).astype(np.float32)
    ones = np.ones((3, 8, 8), dtype=np.float32)
    a_un = oracle.audit(off, s, r, p, 5, 0, 40, gmax=8, rule=oracle.RULE_UNWEIGHTED)
    a_ht1 = oracle.audit(off, s, r, p, 5, 0, 40, pi_w=ones)
    for k in ("mse", "bias_norm", "rep_sqerr", "edge_count"):
        assert np.array_equal(a_un[k], a_ht1[k])
    a_cl = oracle.audit(off, s, r, p, 5, 0, 40, gmax=8, rule=oracle.RULE_CLIPPED, wmax=1e9)
    a_ht = oracle.audit(off, s, r, p, 5, 0, 40, gmax=8)
    for k in ("mse", "bias_norm", "rep_sqerr"):
        assert np.array_equal(a_cl[k], a_ht[k])
