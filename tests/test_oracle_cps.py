"""Pins for the oracle's conditional Poisson (fixed-size) design (App. B
"Fixed-size and exact-cost designs"; Hajek 1964): inclusion probabilities
against brute force over every sample of size n, the fixed-size identities,
simple random sampling as the equal-odds special case, the fit reproducing
its target, the sequential draw's sample distribution (exact sample size and
a chi-square test against prod w / e_n), and Theorem 2 with the design's
exact non-factorising joint probabilities (HT unbiased by enumeration)."""
import itertools
import math

import numpy as np
import pytest

import oracle


def _brute(w, n):
    g = w.size
    subsets = list(itertools.combinations(range(g), n))
    wt = np.array([np.prod(w[list(S)]) for S in subsets])
    P = wt / wt.sum()
    pi = np.zeros(g)
    pij = np.zeros((g, g))
    for p, S in zip(P, subsets):
        for i in S:
            pi[i] += p
            for j in S:
                pij[i, j] += p
    return pi, pij, subsets, P


@pytest.mark.parametrize("g,n", [(4, 2), (6, 1), (6, 3), (8, 5), (10, 4)])
def test_inclusion_probabilities_match_brute_force(g, n):
    rng = np.random.default_rng(g * 10 + n)
    w = rng.lognormal(0.0, 1.0, g)
    pi, pij = oracle.cps_inclusion(w, n)
    bpi, bpij, _, _ = _brute(w, n)
    assert np.allclose(pi, bpi, rtol=1e-12, atol=0)
    assert np.allclose(pij, bpij, rtol=1e-12, atol=1e-300)
    assert abs(pi.sum() - n) <= 1e-12 * n
    off = pij.sum(axis=1) - np.diag(pij)
    assert np.allclose(off, (n - 1) * pi, rtol=1e-12)


def test_equal_odds_is_simple_random_sampling():
    g, n = 9, 4
    pi, pij = oracle.cps_inclusion(np.full(g, 2.5), n)
    assert np.allclose(pi, n / g, rtol=1e-14)
    iu = np.triu_indices(g, 1)
    assert np.allclose(pij[iu], n * (n - 1) / (g * (g - 1)), rtol=1e-14)
    assert np.all(pij[iu] < (n / g) ** 2)          # joint inclusion does not factorise


@pytest.mark.parametrize("g,n", [(5, 2), (16, 8), (40, 13), (64, 30)])
def test_fit_reproduces_target(g, n):
    rng = np.random.default_rng(g)
    t = rng.uniform(0.1, 0.9, g)
    t = t * n / t.sum()
    while t.max() >= 0.97:                     # keep the target strictly inside (0, 1)
        t = np.minimum(t, 0.95)
        t = t * n / t.sum()
    w, it = oracle.cps_fit(t, n)
    assert it > 0
    pi, _ = oracle.cps_inclusion(w, n)
    assert np.max(np.abs(pi / t - 1)) <= 1e-11
    assert abs(np.sum(np.log(w))) <= 1e-9 * g


@pytest.mark.parametrize("g,n", [(2, 1), (7, 3), (16, 15)])
def test_fit_of_equal_targets_is_equal_odds_with_unit_geometric_mean(g, n):
    # Equal targets n/g are met by equal odds at once (simple random
    # sampling); the returned odds still carry the scale convention.
    w, it = oracle.cps_fit(np.full(g, n / g), n)
    assert it == 0
    np.testing.assert_allclose(w, 1.0, rtol=0, atol=1e-15)


def test_draw_has_the_design_distribution():
    g, n, R = 6, 3, 60000
    rng = np.random.default_rng(1)
    w = rng.lognormal(0.0, 0.8, g)
    mask = oracle.cps_draw(np.array([0, g]), w, [n], 11, 0, R)
    assert np.all(mask.sum(axis=1) == n)
    _, _, subsets, P = _brute(w, n)
    idx = {S: k for k, S in enumerate(subsets)}
    counts = np.zeros(len(subsets))
    for row in mask:
        counts[idx[tuple(np.flatnonzero(row))]] += 1
    expected = R * P
    chi2 = float(np.sum((counts - expected) ** 2 / expected))
    dof = len(subsets) - 1
    # 5-sigma bound of the chi-square distribution
    assert chi2 <= dof + 5 * math.sqrt(2 * dof), (chi2, dof)


def test_draw_frequencies_match_inclusion_probabilities():
    rng = np.random.default_rng(2)
    sizes = [12, 7, 20]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    w = rng.lognormal(0.0, 1.0, int(off[-1]))
    n = [5, 3, 11]
    R = 20000
    mask = oracle.cps_draw(off, w, n, 7, 100, R).astype(np.float64)
    for b, g in enumerate(sizes):
        m = mask[:, off[b]:off[b + 1]]
        assert np.all(m.sum(axis=1) == n[b])
        pi, pij = oracle.cps_inclusion(w[off[b]:off[b + 1]], n[b])
        f1 = m.mean(axis=0)
        assert np.all(np.abs(f1 - pi) <= 5 * np.sqrt(pi * (1 - pi) / R) + 1e-12)
        f2 = (m.T @ m) / R
        iu = np.triu_indices(g, 1)
        sd = np.sqrt(pij[iu] * (1 - pij[iu]) / R)
        assert np.all(np.abs(f2[iu] - pij[iu]) <= 5.5 * sd + 1e-12)


def test_ht_with_exact_joint_probabilities_is_unbiased():
    """Theorem 2 under the fixed-size design: averaging the HT estimate over
    every sample with its probability gives the complete-pair average."""
    rng = np.random.default_rng(3)
    g, n, D = 7, 4, 5
    w = rng.lognormal(0.0, 0.7, g)
    r = rng.random(g).astype(np.float32)
    s = rng.standard_normal((g, D)).astype(np.float32)
    _, pij = oracle.cps_inclusion(w, n)
    blk = pij.astype(np.float32)
    _, _, subsets, P = _brute(w, n)
    masks = np.zeros((len(subsets), g), dtype=np.uint8)
    for k, S in enumerate(subsets):
        masks[k, list(S)] = 1
    N = len(subsets)
    est, _ = oracle.pair_grad(np.arange(0, (N + 1) * g, g, dtype=np.int64), np.tile(s, (N, 1)),
                              np.tile(r, N), mask=masks.reshape(-1),
                              pi=np.repeat(blk[None], N, axis=0))
    # weights use the fp32-logged rho; the design's own rho is fp64: expected
    # value = sum_e (rho_e / fl32(rho_e)) h_e / M, within 2^-24 of the target
    mean = P @ est
    sd, rd = s.astype(np.float64), r.astype(np.float64)
    M = g * (g - 1) / 2
    target = sum(0.5 * (rd[i] - rd[j]) * (sd[i] - sd[j]) for i in range(g)
                 for j in range(i + 1, g)) / M
    assert np.max(np.abs(mean - target)) <= 1e-6 * np.abs(target).max()
    exact = sum((pij[i, j] / float(blk[i, j])) * 0.5 * (rd[i] - rd[j]) * (sd[i] - sd[j])
                for i in range(g) for j in range(i + 1, g)) / M
    assert np.max(np.abs(mean - exact)) <= 1e-12 * np.abs(exact).max()
