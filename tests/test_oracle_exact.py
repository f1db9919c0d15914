"""Pins for the oracle's exact design audit (Prop. 1 and App. A "Design
covariance"): the closed-form MSE and bias of every rule that is linear in
the edge indicators are checked against exhaustive enumeration of all 2^G
independent Bernoulli design outcomes (the definition E||g^ - t||^2 written
out), against Theorem 2 (HT has zero design bias), against Prop. 1's
unweighted bias vector, and against the Monte-Carlo audit (a z-test).
"""
import itertools

import numpy as np
import pytest

import oracle

LINEAR = [(oracle.RULE_HT, 0.0), (oracle.RULE_UNWEIGHTED, 0.0), (oracle.RULE_CLIPPED, 4.0),
          (oracle.RULE_MARGINAL, 0.0)]


def _prompt(rng, g, D):
    r = rng.random(g).astype(np.float32)
    s = rng.standard_normal((g, D)).astype(np.float32)
    p = (rng.integers(8, 65, size=g) / 64.0).astype(np.float32)   # exact products
    return r, s, p


def _block(p):
    blk = (p[:, None].astype(np.float64) * p[None, :].astype(np.float64)).astype(np.float32)
    np.fill_diagonal(blk, p)
    return blk


def _target(r, s):
    g = s.shape[0]
    M = g * (g - 1) / 2
    sd = s.astype(np.float64)
    return sum(0.5 * (float(r[i]) - float(r[j])) * (sd[i] - sd[j])
               for i in range(g) for j in range(i + 1, g)) / M


def _enumerated(r, s, p, rule, wmax):
    g, D = s.shape
    masks = np.array(list(itertools.product([0, 1], repeat=g)), dtype=np.uint8)
    n = masks.shape[0]
    off = np.arange(0, (n + 1) * g, g, dtype=np.int64)
    est = oracle.pair_grad_rule(off, np.tile(s, (n, 1)), np.tile(r, n), mask=masks.reshape(-1),
                                pi=np.repeat(_block(p)[None], n, axis=0), rule=rule,
                                wmax=wmax)["out"]
    pd = p.astype(np.float64)
    probs = np.prod(np.where(masks == 1, pd[None, :], 1.0 - pd[None, :]), axis=1)
    t = _target(r, s)
    dev = est - t[None, :]
    return float(probs @ np.sum(dev * dev, axis=1)), float(np.linalg.norm(probs @ est - t))


@pytest.mark.parametrize("rule,wmax", LINEAR)
@pytest.mark.parametrize("g", [3, 5, 7])
def test_exact_audit_matches_enumeration(rule, wmax, g):
    rng = np.random.default_rng(100 * rule + g)
    r, s, p = _prompt(rng, g, 6)
    ex = oracle.audit_exact(np.array([0, g]), s, r, p, rule=rule, wmax=wmax)
    mse, bias = _enumerated(r, s, p, rule, wmax)
    assert abs(ex["mse"][0] - mse) <= 1e-11 * mse
    assert abs(ex["bias_norm"][0] - bias) <= 1e-9 * max(bias, 1e-6 * np.sqrt(mse))


def test_exact_audit_with_logged_block_and_batch():
    rng = np.random.default_rng(7)
    sizes = [4, 6, 5]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    nv = int(off[-1])
    r = rng.random(nv).astype(np.float32)
    s = rng.standard_normal((nv, 5)).astype(np.float32)
    p = (rng.integers(8, 65, size=nv) / 64.0).astype(np.float32)
    pi = np.zeros((3, 6, 6), dtype=np.float32)
    for b, g in enumerate(sizes):
        pi[b, :g, :g] = _block(p[off[b]:off[b + 1]])
    for rule, wmax in LINEAR:
        a = oracle.audit_exact(off, s, r, p, rule=rule, wmax=wmax, gmax=6)
        bw = oracle.audit_exact(off, s, r, p, pi_w=pi, rule=rule, wmax=wmax)
        assert np.allclose(a["mse"], bw["mse"], rtol=1e-14, atol=0)
        for b, g in enumerate(sizes):
            lo, hi = off[b], off[b + 1]
            mse, _ = _enumerated(r[lo:hi], s[lo:hi], p[lo:hi], rule, wmax)
            assert abs(a["mse"][b] - mse) <= 1e-11 * mse


def test_ht_has_zero_design_bias_and_unweighted_has_prop1_bias():
    rng = np.random.default_rng(3)
    g = 8
    r, s, p = _prompt(rng, g, 9)
    ht = oracle.audit_exact(np.array([0, g]), s, r, p)
    assert ht["bias_norm"][0] <= 1e-12 * np.sqrt(ht["mse"][0])
    un = oracle.audit_exact(np.array([0, g]), s, r, p, rule=oracle.RULE_UNWEIGHTED)
    M = g * (g - 1) / 2
    pd = p.astype(np.float64)
    sd = s.astype(np.float64)
    bias = sum((pd[i] * pd[j] - 1.0) * 0.5 * (float(r[i]) - float(r[j])) * (sd[i] - sd[j])
               for i in range(g) for j in range(i + 1, g)) / M
    assert abs(un["bias_norm"][0] - np.linalg.norm(bias)) <= 1e-12 * np.linalg.norm(bias)


@pytest.mark.parametrize("rule,wmax", LINEAR)
def test_certain_design_has_zero_error(rule, wmax):
    rng = np.random.default_rng(5)
    r, s, _ = _prompt(rng, 6, 4)
    ex = oracle.audit_exact(np.array([0, 6]), s, r, np.ones(6, np.float32), rule=rule,
                            wmax=max(wmax, 1.0))
    assert ex["mse"][0] == 0.0 and ex["bias_norm"][0] == 0.0


def test_monte_carlo_audit_agrees_with_exact_audit():
    rng = np.random.default_rng(11)
    sizes = [10, 12]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    nv = int(off[-1])
    r = (rng.random(nv) < 0.5).astype(np.float32)
    s = rng.standard_normal((nv, 32)).astype(np.float32)
    p = rng.uniform(0.2, 1.0, nv).astype(np.float32)
    R = 6000
    for rule, wmax in ((oracle.RULE_HT, 0.0), (oracle.RULE_UNWEIGHTED, 0.0)):
        mc = oracle.audit(off, s, r, p, 17, 0, R, gmax=12, rule=rule, wmax=wmax)
        ex = oracle.audit_exact(off, s, r, p, gmax=12, rule=rule, wmax=wmax)
        for b in range(2):
            sd = mc["rep_sqerr"][b].std() / np.sqrt(R)
            assert abs(mc["mse"][b] - ex["mse"][b]) <= 4.5 * sd


def test_nonlinear_rules_are_rejected():
    r = np.array([0.0, 1.0, 0.5], dtype=np.float32)
    s = np.ones((3, 2), dtype=np.float32)
    p = np.full(3, 0.5, dtype=np.float32)
    for rule in (oracle.RULE_RATIO_KE, oracle.RULE_SELFNORM):
        with pytest.raises(oracle.OracleError):
            oracle.audit_exact(np.array([0, 3]), s, r, p, rule=rule)
