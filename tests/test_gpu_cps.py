"""GPU parity for the fixed-size conditional Poisson design (App. B) through
the C ABI, against the oracle.

Bars: odds within 1e-9 relative (both sides converge to 1e-12), sample sizes
exact, the fp32 joint block within 1e-6 relative; draws bit-exact given the
same odds (the thresholds are computed the same way in fp64 on both sides);
the fixed-size chain's gradients within 2e-3 relative L2 (bf16 scores);
draw frequencies within 5 standard errors of the exact probabilities.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11368_amd as pair
import workloads as wl
from tests.gpu_util import DEV, log, rel_l2, scores_to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pair.lib()
    yield
    torch.cuda.synchronize()


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


@pytest.mark.parametrize("B,G", [(24, None), (16, 16), (8, 33)])
def test_fit_vs_oracle(B, G):
    w_ = wl.WORKLOADS["ragged"].replace(B=B) if G is None else wl.WORKLOADS["b128"].replace(B=B, G=G)
    meta = wl.host_meta(w_)
    tgt = wl.cps_targets(meta.offsets)
    log(f"cps fit B={B} gmax={meta.gmax}")
    got = pair.cps_fit(_t(meta.offsets), _t(tgt), meta.gmax, nv=meta.nv)
    torch.cuda.synchronize()
    assert int(got["status"].item()) == 0
    w, n = got["w"].cpu().numpy(), got["n"].cpu().numpy()
    pj = got["pi_joint"].cpu().numpy()
    assert np.all(got["iters"].cpu().numpy() > 0)
    worst_w, worst_p = 0.0, 0.0
    for b in range(meta.B):
        lo, hi = meta.offsets[b], meta.offsets[b + 1]
        g = hi - lo
        nb = int(round(float(tgt[lo:hi].astype(np.float64).sum())))
        assert n[b] == nb
        ow, it = oracle.cps_fit(tgt[lo:hi], nb)
        assert it > 0
        worst_w = max(worst_w, float(np.max(np.abs(w[lo:hi] / ow - 1))))
        _, opij = oracle.cps_inclusion(ow, nb)
        worst_p = max(worst_p, float(np.max(np.abs(pj[b, :g, :g] - opij) / opij)))
        assert np.all(pj[b, g:, :] == 0) and np.all(pj[b, :, g:] == 0)
    log(f"  max w rel {worst_w:.2e}, max pi_ij rel {worst_p:.2e}")
    assert worst_w <= 1e-9 and worst_p <= 1e-6


def _hard_targets():
    """Targets that stress the fit: all equal (the start is already the
    answer), a few tied values, a wide spread, and half the units near 0 with
    half near 1; sample sizes 1, 2, G/2 and G - 1; G from 2 to 64."""
    r = np.random.default_rng(17)
    out = []
    for g in (2, 3, 7, 16, 40, 64):
        for n in sorted({1, 2, g // 2, g - 1}):
            if not 1 <= n < g:
                continue
            cands = [np.full(g, n / g), r.choice([0.2, 0.5, 0.7], g), r.uniform(0.001, 0.999, g),
                     np.where(np.arange(g) % 2 == 0, r.uniform(1e-3, 1e-2, g), r.uniform(0.9, 1.0, g))]
            if g % 2 == 0 and n == g // 2:
                cands.append(np.where(np.arange(g) % 2 == 0, r.uniform(0.01, 0.03, g),
                                      r.uniform(0.97, 0.99, g)))
            for t in cands:
                t = t * (n / t.sum())
                if 0 < t.min() and t.max() < 0.999:
                    out.append(t.astype(np.float32))
    return out


def test_fit_hard_targets_vs_oracle():
    groups = _hard_targets()
    sizes = np.array([t.size for t in groups])
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    tgt = np.concatenate(groups)
    nv = int(offsets[-1])
    log(f"cps fit hard targets: B={len(groups)} nv={nv}")
    got = pair.cps_fit(_t(offsets), _t(tgt), 64, nv=nv)
    torch.cuda.synchronize()
    assert int(got["status"].item()) == 0
    w, n, its = got["w"].cpu().numpy(), got["n"].cpu().numpy(), got["iters"].cpu().numpy()
    pj = got["pi_joint"].cpu().numpy()
    assert np.all(its >= 0)
    worst_w, worst_p = 0.0, 0.0
    for b in range(len(groups)):
        lo, hi = offsets[b], offsets[b + 1]
        g = hi - lo
        nb = int(round(float(tgt[lo:hi].astype(np.float64).sum())))
        assert n[b] == nb
        ow, it = oracle.cps_fit(tgt[lo:hi], nb, max_iter=100000)
        assert it >= 0
        worst_w = max(worst_w, float(np.max(np.abs(w[lo:hi] / ow - 1))))
        _, opij = oracle.cps_inclusion(ow, nb)
        off = ~np.eye(g, dtype=bool)
        if nb >= 2:
            worst_p = max(worst_p, float(np.max(np.abs(pj[b, :g, :g] - opij)[off] / opij[off])))
        else:
            assert np.all(np.abs(pj[b, :g, :g][off]) <= 1e-12)
        assert np.max(np.abs(np.diag(pj[b, :g, :g]) - np.diag(opij)) / np.diag(opij)) <= 1e-6
    log(f"  max w rel {worst_w:.2e}, max pi_ij rel {worst_p:.2e}, evaluations max {its.max()}")
    assert worst_w <= 1e-9 and worst_p <= 1e-6
    assert its.max() <= 40


@pytest.mark.parametrize("R", [1, 300])
def test_draw_bit_exact(R):
    w_ = wl.WORKLOADS["ragged"].replace(B=40)
    meta = wl.host_meta(w_)
    odds, n = wl.cps_odds(meta.offsets)
    log(f"cps draw B=40 R={R}")
    got = pair.cps_draw(_t(meta.offsets), _t(odds), _t(n), 99, 5, R, meta.gmax, nv=meta.nv)
    torch.cuda.synchronize()
    assert int(got["status"].item()) == 0
    want = oracle.cps_draw(meta.offsets, odds, n, 99, 5, R)
    assert np.array_equal(got["mask"].cpu().numpy(), want)
    ec = got["edge_count"].cpu().numpy()
    assert np.all(ec == (n * (n - 1) // 2)[None, :])


def test_draw_all_or_none_and_bad_input():
    offsets = np.array([0, 5, 9], dtype=np.int64)
    odds = np.ones(9)
    got = pair.cps_draw(_t(offsets), _t(odds), _t(np.array([5, 0], np.int32)), 1, 0, 3, 5, nv=9)
    torch.cuda.synchronize()
    m = got["mask"].cpu().numpy()
    assert np.all(m[:, :5] == 1) and np.all(m[:, 5:] == 0)
    bad = pair.cps_draw(_t(offsets), _t(odds), _t(np.array([6, 1], np.int32)), 1, 0, 3, 5, nv=9)
    torch.cuda.synchronize()
    assert int(bad["status"].item()) & pair.ST_P_RANGE


def test_fixed_size_chain_vs_oracle_chain():
    """targets -> fit -> draw -> coefficients with the exact non-factorising
    joint block -> weighted gradient, on the GPU and, independently, in the
    oracle."""
    w_ = wl.WORKLOADS["b128"].replace(B=32, D=2048 + 24)
    meta = wl.host_meta(w_)
    tgt = wl.cps_targets(meta.offsets, seed=11)
    dm_off, dm_rew = _t(meta.offsets), _t(meta.rewards)
    fit = pair.cps_fit(dm_off, _t(tgt), meta.gmax, nv=meta.nv)
    dr = pair.cps_draw(dm_off, fit["w"], fit["n"], 31, 0, 1, meta.gmax, nv=meta.nv)
    c = pair.edge_coeffs(dm_off, dm_rew, dr["mask"][0], fit["pi_joint"], meta.gmax, nv=meta.nv)
    s = wl.host_scores(w_, meta.nv)
    g = pair.weighted_grad(dm_off, scores_to_device(s, w_), c["coeff"], nv=meta.nv)
    torch.cuda.synchronize()
    assert int(fit["status"].item()) == 0 and int(c["status"].item()) == 0
    # the oracle's own chain
    B, gm = meta.B, meta.gmax
    ow = np.zeros(meta.nv)
    on = np.zeros(B, dtype=np.int32)
    opi = np.zeros((B, gm, gm), dtype=np.float32)
    for b in range(B):
        lo, hi = meta.offsets[b], meta.offsets[b + 1]
        on[b] = int(round(float(tgt[lo:hi].astype(np.float64).sum())))
        ow[lo:hi], _ = oracle.cps_fit(tgt[lo:hi], on[b])
        _, pij = oracle.cps_inclusion(ow[lo:hi], on[b])
        opi[b, :hi - lo, :hi - lo] = pij.astype(np.float32)
    omask = oracle.cps_draw(meta.offsets, ow, on, 31, 0, 1)
    assert np.array_equal(dr["mask"].cpu().numpy(), omask)
    est, ec = oracle.pair_grad(meta.offsets, s, meta.rewards, mask=omask[0], pi=opi)
    assert np.array_equal(c["edge_count"].cpu().numpy(), ec)
    err = rel_l2(g["out"].cpu().numpy(), est)
    log(f"  fixed-size chain grad rel L2 {err:.2e}")
    assert err <= 2e-3


@pytest.mark.timeout(300)
def test_full_ragged_draw_frequencies():
    """B = 512 ragged prompts, R = 4096 draws: per-unit and per-pair
    frequencies against the exact probabilities of the GPU fit."""
    w_ = wl.WORKLOADS["ragged"]
    meta = wl.host_meta(w_)
    tgt = wl.cps_targets(meta.offsets, seed=5)
    off = _t(meta.offsets)
    fit = pair.cps_fit(off, _t(tgt), meta.gmax, nv=meta.nv)
    R = 4096
    dr = pair.cps_draw(off, fit["w"], fit["n"], 1234, 0, R, meta.gmax, nv=meta.nv)
    torch.cuda.synchronize()
    assert int(fit["status"].item()) == 0 and int(dr["status"].item()) == 0
    m = dr["mask"].cpu().numpy().astype(np.float64)
    pj = fit["pi_joint"].cpu().numpy().astype(np.float64)
    n = fit["n"].cpu().numpy()
    zmax = 0.0
    for b in np.random.default_rng(0).choice(meta.B, 40, replace=False):
        lo, hi = meta.offsets[b], meta.offsets[b + 1]
        g = hi - lo
        mb = m[:, lo:hi]
        assert np.all(mb.sum(axis=1) == n[b])
        pi = np.diag(pj[b, :g, :g])
        assert abs(pi.sum() - n[b]) <= 1e-4 * n[b]
        f2 = (mb.T @ mb) / R
        iu = np.triu_indices(g, 1)
        sd = np.sqrt(np.maximum(pj[b][iu] * (1 - pj[b][iu]), 1e-12) / R)
        z = np.abs(f2[iu] - pj[b][iu]) / sd
        zmax = max(zmax, float(z.max()))
        f1 = mb.mean(axis=0)
        assert np.all(np.abs(f1 - pi) <= 5 * np.sqrt(pi * (1 - pi) / R) + 1e-9)
    log(f"  max pair z {zmax:.2f}")
    assert zmax <= 6.0
