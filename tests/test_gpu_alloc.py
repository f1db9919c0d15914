"""GPU parity for the probability design (Sec. 4.3-4.4) through the C ABI,
against the allocation oracle (SLSQP in fp64 on the same program).

Bars: the design is an optimisation, so the GPU result is checked as an
optimum -- its objective within 1e-6 relative of the oracle's (and never
worse by more), its own KKT residual (the oracle's checker) at most 1e-5,
the budget spent to 1e-6 -- and the probabilities within 1e-3 relative of
the oracle's (the oracle's solver stops at KKT residuals of ~1e-7).
The uniform design is compared exactly up to fp32 rounding.
"""
import numpy as np
import pytest
import torch

import paper_2608_11368_amd as pair
import workloads as wl
from oracle import alloc
from tests.gpu_util import DEV, log

pytestmark = pytest.mark.gpu

PI_MIN = 0.08


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pair.lib()
    yield
    torch.cuda.synchronize()


def _run(offsets, inp, design, gmax, m_hat=None, pi_min=PI_MIN):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    out = pair.design_alloc(t(offsets), t(inp.p_hat), t(inp.c_hat), t(inp.budget), gmax,
                            pi_min=pi_min, design=design,
                            m_hat=None if m_hat is None else t(m_hat))
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


@pytest.mark.parametrize("design", [pair.DESIGN_PAIR, pair.DESIGN_POINTWISE])
@pytest.mark.parametrize("ratio,scaled", [(0.5, False), (0.25, False), (0.75, True)])
def test_design_vs_oracle(design, ratio, scaled):
    w = wl.WORKLOADS["ragged"].replace(B=48)
    meta = wl.host_meta(w)
    inp = wl.alloc_inputs(w, meta.offsets, ratio=ratio)
    m_hat = None
    if scaled:
        m_hat = np.random.default_rng(5).uniform(0.5, 2.0, meta.nv).astype(np.float32)
    log(f"design {design} ratio {ratio} scaled {scaled} B={meta.B}")
    got = _run(meta.offsets, inp, design, meta.gmax, m_hat)
    assert got["status"][0] == 0
    want = alloc.solve_batch(meta.offsets, inp.p_hat.astype(np.float64),
                             inp.c_hat.astype(np.float64), inp.budget.astype(np.float64), PI_MIN,
                             design=design, m_hat=None if m_hat is None else m_hat.astype(np.float64))
    assert want["success"].all()
    worst_obj, worst_pi, worst_kkt = 0.0, 0.0, 0.0
    for b in range(meta.B):
        lo, hi = meta.offsets[b], meta.offsets[b + 1]
        pg = got["pi"][lo:hi].astype(np.float64)
        po = want["pi"][lo:hi]
        c = inp.c_hat[lo:hi].astype(np.float64)
        bud = float(inp.budget[b])
        assert np.all(pg >= np.float32(PI_MIN)) and np.all(pg <= 1.0)
        assert c @ pg <= bud * (1 + 1e-6)
        rel_obj = (got["objective"][b] - want["objective"][b]) / want["objective"][b]
        worst_obj = max(worst_obj, abs(rel_obj))
        assert rel_obj <= 1e-6
        worst_pi = max(worst_pi, float(np.max(np.abs(pg / po - 1.0))))
        a = alloc.edge_proxy(inp.p_hat[lo:hi].astype(np.float64),
                             None if m_hat is None else m_hat[lo:hi].astype(np.float64))
        if design == pair.DESIGN_POINTWISE:
            pv = inp.p_hat[lo:hi].astype(np.float64)
            kk = alloc.kkt_residual(pg, np.zeros_like(a), pv * (1 - pv), c, bud, PI_MIN)[0]
        else:
            kk = alloc.kkt_residual(pg, a, alloc.vertex_term(a), c, bud, PI_MIN)[0]
        worst_kkt = max(worst_kkt, kk)
    log(f"  max |obj rel| {worst_obj:.2e}, max pi rel {worst_pi:.2e}, max KKT {worst_kkt:.2e}, "
        f"sweeps max {got['iters'].max()}")
    assert worst_obj <= 1e-6 and worst_pi <= 1e-3 and worst_kkt <= 1e-5


def test_uniform_design_and_budget_edges():
    w = wl.WORKLOADS["ragged"].replace(B=16)
    meta = wl.host_meta(w)
    inp = wl.alloc_inputs(w, meta.offsets)
    got = _run(meta.offsets, inp, pair.DESIGN_UNIFORM, meta.gmax)
    for b in range(meta.B):
        lo, hi = meta.offsets[b], meta.offsets[b + 1]
        want = np.float32(np.clip(float(inp.budget[b]) / inp.c_hat[lo:hi].astype(np.float64).sum(),
                                  PI_MIN, 1.0))
        assert np.allclose(got["pi"][lo:hi], want, rtol=1e-6, atol=0)
    # slack budget: every vertex continues; tight budget: every vertex at the floor
    slack = wl.AllocInputs(inp.p_hat, inp.c_hat, inp.budget * 2.5)
    assert np.all(_run(meta.offsets, slack, pair.DESIGN_PAIR, meta.gmax)["pi"] == 1.0)
    tight = wl.AllocInputs(inp.p_hat, inp.c_hat, np.array(
        [PI_MIN * inp.c_hat[meta.offsets[b]:meta.offsets[b + 1]].astype(np.float64).sum()
         for b in range(meta.B)], dtype=np.float32) * np.float32(1.0000001))
    tg = _run(meta.offsets, tight, pair.DESIGN_PAIR, meta.gmax)
    assert np.allclose(tg["pi"], PI_MIN, rtol=1e-3)   # 1e-7 of slack may go to one vertex
    bad = wl.AllocInputs(inp.p_hat, inp.c_hat, inp.budget * np.float32(0.1))
    out = _run(meta.offsets, bad, pair.DESIGN_PAIR, meta.gmax)
    assert out["status"][0] & pair.ST_BUDGET
    assert np.all(out["pi"] == np.float32(PI_MIN))


def test_two_vertex_closed_form_and_design_feeds_the_draw():
    offsets = np.array([0, 2, 4], dtype=np.int64)
    inp = wl.AllocInputs(np.array([0.3, 0.6, 0.5, 0.5], np.float32),
                         np.array([1000, 3000, 2000, 2000], np.float32),
                         np.array([1500, 2000], np.float32))
    got = _run(offsets, inp, pair.DESIGN_PAIR, 2, pi_min=0.05)
    # one edge, b = 0: maximise pi_1 pi_2 on the budget line: pi_i = budget / (2 c_i)
    assert np.allclose(got["pi"], [0.75, 0.25, 0.5, 0.5], rtol=1e-6)
    t = lambda a: torch.from_numpy(a).to(DEV)
    d = pair.design_inclusion(t(offsets), t(got["pi"]), 3, 0, 64, 2)
    torch.cuda.synchronize()
    assert int(d["status"].item()) == 0
    assert np.allclose(d["pi"].cpu().numpy()[0, 0, 1], np.float32(0.75) * np.float32(0.25))


@pytest.mark.timeout(300)
def test_full_ragged_batch_sampled_against_oracle():
    """B = 512 prompts, G_b ~ U{2..64}, in the launch configuration the bench
    times; 24 sampled prompts against the oracle."""
    w = wl.WORKLOADS["ragged"]
    meta = wl.host_meta(w)
    inp = wl.alloc_inputs(w, meta.offsets)
    log(f"full ragged design B={meta.B} nv={meta.nv}")
    got = _run(meta.offsets, inp, pair.DESIGN_PAIR, meta.gmax)
    assert got["status"][0] == 0
    rng = np.random.default_rng(2)
    for b in rng.choice(meta.B, 24, replace=False):
        lo, hi = meta.offsets[b], meta.offsets[b + 1]
        want = alloc.solve(inp.p_hat[lo:hi].astype(np.float64), inp.c_hat[lo:hi].astype(np.float64),
                           float(inp.budget[b]), PI_MIN)
        rel = (got["objective"][b] - want["objective"]) / want["objective"]
        assert rel <= 1e-6 and abs(rel) <= 1e-6, (b, rel)
    log(f"  sweeps: mean {got['iters'].mean():.1f}, max {got['iters'].max()}")


def _run_ex(offsets, inp, design, gmax, pi_prev=None, max_sweeps=0, pi_min=PI_MIN):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    out = pair.design_alloc(t(offsets), t(inp.p_hat), t(inp.c_hat), t(inp.budget), gmax,
                            pi_min=pi_min, design=design,
                            pi_prev=None if pi_prev is None else t(pi_prev),
                            max_sweeps=max_sweeps)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


@pytest.mark.parametrize("design", [pair.DESIGN_PAIR, pair.DESIGN_POINTWISE, pair.DESIGN_UNIFORM])
def test_solver_residual_against_oracle_kkt(design):
    """The residual the solver logs (App. C) is the KKT residual of the
    design's program at the returned fp32 probabilities: the oracle's
    checker on the same probabilities gives the same value."""
    w = wl.WORKLOADS["ragged"].replace(B=40)
    meta = wl.host_meta(w)
    inp = wl.alloc_inputs(w, meta.offsets)
    log(f"solver residual, design {design}")
    got = _run_ex(meta.offsets, inp, design, meta.gmax)
    assert got["status"][0] == 0 and np.all(got["iters"] >= 0)
    pmin = float(np.float32(PI_MIN))
    worst = 0.0
    for b in range(meta.B):
        lo, hi = meta.offsets[b], meta.offsets[b + 1]
        pg = got["pi"][lo:hi].astype(np.float64)
        pv = inp.p_hat[lo:hi].astype(np.float64)
        c = inp.c_hat[lo:hi].astype(np.float64)
        a = alloc.edge_proxy(pv)
        if design == pair.DESIGN_POINTWISE:
            want = alloc.kkt_residual(pg, np.zeros_like(a), pv * (1 - pv), c, float(inp.budget[b]),
                                      pmin)[0]
        else:
            want = alloc.kkt_residual(pg, a, alloc.vertex_term(a), c, float(inp.budget[b]), pmin)[0]
        r = got["residual"][b]
        worst = max(worst, abs(r - want) / max(want, 1e-12))
        assert abs(r - want) <= 1e-9 + 1e-6 * want, (b, r, want)
        if design != pair.DESIGN_UNIFORM:
            assert r <= 1e-5
    if design == pair.DESIGN_UNIFORM:      # one probability is not the PAIR optimum
        assert got["residual"].max() > 1e-3
    log(f"  residual vs oracle checker: worst relative difference {worst:.2e}, "
        f"largest residual {got['residual'].max():.2e}")


@pytest.mark.parametrize("design", [pair.DESIGN_PAIR, pair.DESIGN_POINTWISE])
def test_solver_failure_falls_back_to_uniform(design):
    """A sweep cap the solver cannot converge within: every prompt whose
    budget binds falls back to the uniform design of the same expected cost
    (App. C), with the status bit, negative sweep counts, and probabilities
    equal to the oracle's uniform design up to fp32 rounding."""
    w = wl.WORKLOADS["ragged"].replace(B=32)
    meta = wl.host_meta(w)
    inp = wl.alloc_inputs(w, meta.offsets)
    log(f"forced solver failure, design {design}")
    got = _run_ex(meta.offsets, inp, design, meta.gmax, max_sweeps=2)
    assert got["status"][0] & pair.ST_SOLVER
    assert np.all(got["iters"] < 0) and np.all(got["iters"] >= -2)
    want = alloc.solve_batch(meta.offsets, inp.p_hat.astype(np.float64),
                             inp.c_hat.astype(np.float64), inp.budget.astype(np.float64), PI_MIN,
                             design=alloc.UNIFORM)
    assert np.allclose(got["pi"], want["pi"], rtol=2e-7, atol=0)
    for b in range(meta.B):
        lo, hi = meta.offsets[b], meta.offsets[b + 1]
        spent = inp.c_hat[lo:hi].astype(np.float64) @ got["pi"][lo:hi].astype(np.float64)
        assert abs(spent / float(inp.budget[b]) - 1.0) <= 1e-6
    # the same inputs with the default cap converge, with no status bit
    ok = _run_ex(meta.offsets, inp, design, meta.gmax)
    assert ok["status"][0] == 0 and np.all(ok["iters"] > 2)


def test_solver_warm_start():
    """Warm starts from the previous step's probabilities (App. C): from the
    optimum itself the solver needs a fraction of the cold sweeps and returns
    the same design; from a perturbed start, from one probability for all and
    from a start with NaN and out-of-range entries it reaches the same
    optimum (the program is strictly convex)."""
    w = wl.WORKLOADS["ragged"].replace(B=64)
    meta = wl.host_meta(w)
    inp = wl.alloc_inputs(w, meta.offsets)
    cold = _run_ex(meta.offsets, inp, pair.DESIGN_PAIR, meta.gmax)
    assert cold["status"][0] == 0
    rng = np.random.default_rng(11)
    starts = {
        "optimum": cold["pi"],
        "perturbed": np.clip(cold["pi"] * rng.uniform(0.7, 1.3, meta.nv), 0.0, 1.0).astype(np.float32),
        "uniform": np.full(meta.nv, 0.5, dtype=np.float32),
        "nan": np.where(rng.random(meta.nv) < 0.2, np.nan,
                        rng.uniform(-0.5, 1.5, meta.nv)).astype(np.float32),
    }
    for name, start in starts.items():
        warm = _run_ex(meta.offsets, inp, pair.DESIGN_PAIR, meta.gmax, pi_prev=start)
        assert warm["status"][0] == 0 and np.all(warm["iters"] >= 0), name
        rel_obj = np.abs(warm["objective"] / cold["objective"] - 1.0).max()
        rel_pi = np.abs(warm["pi"].astype(np.float64) / cold["pi"] - 1.0).max()
        log(f"  warm start {name}: sweeps mean {warm['iters'].mean():.1f} "
            f"(cold {cold['iters'].mean():.1f}), max |obj rel| {rel_obj:.1e}, max pi rel {rel_pi:.1e}")
        assert rel_obj <= 1e-9 and rel_pi <= 1e-4, name
        assert warm["residual"].max() <= 1e-5
        if name == "optimum":
            assert warm["iters"].mean() <= 0.5 * cold["iters"].mean()
