"""Seeded random sweep of the HIP path against the CPU oracle.

Each case draws its own shapes: prompt counts, ragged group sizes in
[2, 64], score widths on and off the kernels' tile boundaries, padded row
strides (NaN in the padding), fp32 and bf16 scores, binary / continuous /
saturated rewards, continuation probabilities from near zero up to exactly 1,
and design seeds and replicate offsets.  The sweep covers the HT chain and
audit, every edge-weight rule (coefficients, ESS, maximum weight, gradient,
audit replay) and the exact audit of the linear rules.  The bars are those of
the parity tests: masks, logged rho and counts bit-exact; coefficients and fp32
gradients within 1e-5 relative L2, bf16 gradients within 2e-3; exact zeros
where the oracle's estimate is exactly zero; audit edge counts bit-exact,
per-replicate squared errors within 2e-3 relative L2.  Each e_r and each
prompt's MSE must be within 2e-3 relative, and the bias norm (its row applied
in fp32) within 5e-5, unless the first-order rounding bound of the
contraction allows more: with one fp16 rounding of each deviation entry
(relative error at most u = 2^-11, the same in every score column),
|Delta e_r| <= 2 u sum_i |delta_ri z_ri|, z_r = S y_r^T, which exceeds
u e_r only when the terms delta_ri z_ri cancel (a single score column, for
instance).  The bars are then 1.5 times that bound (with its fp32 terms),
computed on the host from the oracle's draws and folds; in well-conditioned
cases the bound is about u e_r, so 2e-3 relative stays the binding bar.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11368_amd as pair
from tests.gpu_util import DEV, log
from tests.gpu_util import rel_l2 as _rel_l2

pytestmark = pytest.mark.gpu


def rel_l2(got, want):
    # A random case may draw only saturated prompts (an all-zero reference);
    # exact zeros are then required, and checked again where it matters.
    return _rel_l2(got, want, zero_ok=True)


FP32_TOL = 1e-5
BF16_TOL = 2e-3
BIAS_TOL = 5e-5
WIDTHS = (1, 2, 7, 31, 255, 1000, 1023, 1025, 2047, 2049, 4095, 4097, 6000)


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pair.lib()
    yield
    torch.cuda.synchronize()


def _bf16_bits(x):
    """fp32 -> bf16 bit patterns (round to nearest even, torch on the host)."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16) \
        .view(torch.int16).numpy().view(np.uint16)


def _case(rng, max_b, widths, bf16=None):
    B = int(rng.integers(1, max_b + 1))
    sizes = rng.integers(2, 65, size=B)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    nv = int(offsets[-1])
    D = int(rng.choice(widths))
    if bf16 is None:
        bf16 = bool(rng.integers(0, 2))
    unit = 8 if bf16 else 4                          # 16-byte aligned rows
    ld = (D + unit - 1) // unit * unit + int(rng.choice([0, unit, 3 * unit]))
    rewards = np.empty(nv, dtype=np.float32)
    p = np.empty(nv, dtype=np.float32)
    for b in range(B):
        o0, o1 = offsets[b], offsets[b + 1]
        kind = rng.integers(0, 3)
        if kind == 0:
            rewards[o0:o1] = (rng.random(o1 - o0) < rng.random()).astype(np.float32)
        elif kind == 1:
            rewards[o0:o1] = rng.random(o1 - o0)
        else:
            rewards[o0:o1] = float(rng.integers(0, 2))     # saturated prompt
        pmin = float(rng.choice([1e-3, 0.05, 0.3]))
        p[o0:o1] = pmin + (1.0 - pmin) * rng.random(o1 - o0)
        p[o0:o1][rng.random(o1 - o0) < 0.1] = 1.0
    s = rng.standard_normal((nv, D)).astype(np.float32)
    if bf16:
        host = np.full((nv, ld), 0x7FC0, dtype=np.uint16)   # NaN padding
        host[:, :D] = _bf16_bits(s)
        dev = torch.from_numpy(host.view(np.int16)).to(DEV).view(torch.bfloat16)[:, :D]
    else:
        host = np.full((nv, ld), np.nan, dtype=np.float32)
        host[:, :D] = s
        dev = torch.from_numpy(host).to(DEV)[:, :D]
    seed = int(rng.integers(0, 2**63))
    rep0 = int(rng.integers(0, 1 << 20))
    return dict(B=B, offsets=offsets, nv=nv, D=D, ld=ld, bf16=bf16, rewards=rewards, p=p,
                host=host[:, :D], dev=dev, seed=seed, rep0=rep0, gmax=int(sizes.max()))


@pytest.mark.parametrize("case_id", range(96))
def test_random_gradient_chain(case_id):
    rng = np.random.default_rng(7000 + case_id)
    c = _case(rng, 24, WIDTHS)
    B, nv, gmax, D = c["B"], c["nv"], c["gmax"], c["D"]
    R = int(rng.integers(1, 4))
    log(f"random chain {case_id}: B={B} nv={nv} gmax={gmax} D={D} ld={c['ld']} "
        f"{'bf16' if c['bf16'] else 'fp32'} R={R} rep0={c['rep0']}")
    off = torch.from_numpy(c["offsets"]).to(DEV)
    rew = torch.from_numpy(c["rewards"]).to(DEV)
    p = torch.from_numpy(c["p"]).to(DEV)

    d = pair.design_inclusion(off, p, c["seed"], c["rep0"], R, gmax, nv=nv)
    od = oracle.design_inclusion(c["offsets"], c["p"], c["seed"], c["rep0"], R, gmax)
    torch.cuda.synchronize()
    assert int(d["status"].item()) == 0
    for key in ("mask", "pi", "edge_count", "completed"):
        assert np.array_equal(d[key].cpu().numpy(), od[key]), key

    r = R - 1                                        # the last replicate feeds the estimator
    co = pair.edge_coeffs(off, rew, d["mask"][r], d["pi"], gmax, nv=nv)
    want_c, ec = oracle.pair_coeffs(c["offsets"], c["rewards"], od["mask"][r], od["pi"])
    got_c = co["coeff"].cpu().numpy()
    assert int(co["status"].item()) == 0
    assert rel_l2(got_c, want_c) <= FP32_TOL
    assert np.all(got_c[want_c == 0.0] == 0.0)
    assert np.array_equal(co["edge_count"].cpu().numpy(), ec)

    # the one-launch draw + fold equals the two calls bitwise
    coeff2 = torch.empty(nv, device=DEV)
    mask2 = torch.empty(nv, dtype=torch.uint8, device=DEV)
    pi2 = torch.empty((B, gmax, gmax), device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    pair.pair_design_coeffs(B, nv, gmax, off, p, rew, c["seed"], c["rep0"] + r, coeff2, mask2, pi2,
                            None, None, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert torch.equal(mask2, d["mask"][r]) and torch.equal(pi2, d["pi"])
    assert torch.equal(coeff2, co["coeff"])

    est, _ = oracle.pair_grad(c["offsets"], c["host"], c["rewards"], od["mask"][r], od["pi"])
    tol = BF16_TOL if c["bf16"] else FP32_TOL
    g = pair.weighted_grad(off, c["dev"], co["coeff"], nv=nv)
    out = g["out"].cpu().numpy()
    assert int(g["status"].item()) == 0 and np.isfinite(out).all()
    err = rel_l2(out, est)
    log(f"  coeff rel L2 {rel_l2(got_c, want_c):.2e}, grad rel L2 {err:.2e}")
    assert err <= tol
    for b in range(B):
        if not np.any(est[b]):
            assert np.all(out[b] == 0.0), f"prompt {b} must be exactly zero"
    gm = pair.weighted_grad(off, c["dev"], co["coeff"], nv=nv, reduce=True)["out"].cpu().numpy()
    assert np.isfinite(gm).all()
    # The batch mean of a few columns can cancel far below its summands (a
    # single column at 1/680 of them in one case), and fp32 coefficients and
    # accumulation then cannot reach a bound relative to the result itself.
    # Its error is measured against the larger of the result and 1/100 of the
    # summands' magnitude sum_i |c_i| |s_i| / B (the fp32 summation bound).
    want_m = est.mean(axis=0)
    host = np.nan_to_num(np.asarray(c["host"], dtype=np.float64) if not c["bf16"] else
                         (c["host"].astype(np.uint32) << 16).view(np.float32).astype(np.float64))
    mag = np.abs(want_c) @ np.abs(np.where(want_c[:, None] != 0.0, host, 0.0)) / B
    scale = max(np.linalg.norm(want_m), np.linalg.norm(mag) / 100.0)
    if scale == 0.0:                                   # every prompt saturated: exact zeros
        assert np.all(gm == 0.0)
        return
    err_m = np.linalg.norm(gm - want_m) / scale
    log(f"  batch mean error {err_m:.2e} "
        f"(result / summands {np.linalg.norm(want_m) / np.linalg.norm(mag):.2e})")
    assert err_m <= tol


U16 = 2.0 ** -11   # fp16 rounding of a rescaled deviation entry, relative
F32 = 2.0 ** -24   # fp32 unit roundoff
BOUND_FACTOR = 1.5  # headroom over the first-order rounding bound


def _audit_rounding_bounds(c, R, rule=pair.RULE_HT, wmax=0.0):
    """First-order bounds on the audit's rounding, from the oracle's design
    draw and coefficient fold (deviations delta_r = A~^(r) - a, y_r =
    delta_r S, z_r = S y_r^T, so e_r = delta_r . z_r):
      e_r:  2 sum_i (u |delta_ri| + phi_ri) |z_ri|      fp16 deviation operand
            + 2 KP eps ||y_r|| || |delta_r| |S| ||       fp32 accumulation
            + (2 KP + 1) eps ||y_r||_1 sum_i |delta_ri| M_i   fp16 subnormals
            + || (u |delta_r| + phi_r) |S| ||^2            second order
      bias: the same terms for the mean deviation row applied in fp32 (no
            fp16 rounding), with its fp32 sums over replicates, over 2 bias.
    phi is an allowance for the fold's own fp32 rounding (2^-18 of each
    coefficient and of its target, plus 2^-17 of the row's largest, which
    covers the centring and cancelling folds: a complete design can
    reproduce the target exactly, e_r = 0, where fp32 leaves a residue), M_i
    the largest magnitude of score row i and KP the padded group size.  Returns
    (bounds on e_r [B][R], bounds on the bias norm [B])."""
    off = c["offsets"]
    B = off.size - 1
    od = oracle.design_inclusion(off, c["p"], c["seed"], c["rep0"], R, c["gmax"])
    a, _ = oracle.pair_coeffs(off, c["rewards"])
    A = np.stack([oracle.pair_coeffs_rule(off, c["rewards"], od["mask"][r], od["pi"], rule,
                                          wmax)["coeff"] for r in range(R)])
    S = (c["host"].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    kp = (c["gmax"] + 15) // 16 * 16
    nch = (R + 255) // 256
    e_bound = np.zeros((B, R))
    b_bound = np.zeros(B)
    for b in range(B):
        o0, o1 = off[b], off[b + 1]
        sb = S[o0:o1]
        asb = np.abs(sb)
        rowmax = asb.max(axis=1)
        d = A[:, o0:o1] - a[o0:o1]
        absA, absa = np.abs(A[:, o0:o1]), np.abs(a[o0:o1])
        phi = (2.0 ** -18 * (absA + absa)
               + 2.0 ** -17 * (absA.max(axis=1, keepdims=True) + absa.max()))
        y = d @ sb
        z = y @ sb.T
        ny = np.linalg.norm(y, axis=1)
        nabs = np.linalg.norm(np.abs(d) @ asb, axis=1)
        e_bound[b] = (2.0 * ((U16 * np.abs(d) + phi) * np.abs(z)).sum(axis=1)
                      + 2.0 * kp * F32 * ny * nabs
                      + (2 * kp + 1) * F32 * np.abs(y).sum(axis=1) * (np.abs(d) * rowmax).sum(axis=1)
                      + np.linalg.norm((U16 * np.abs(d) + phi) @ asb, axis=1) ** 2)
        dbar = d.mean(axis=0)
        ybar = dbar @ sb
        nb = np.linalg.norm(ybar)
        ddbar = (nch + 12) * F32 * np.abs(d).mean(axis=0) + phi.mean(axis=0)
        if nb > 0.0:
            sq = (2.0 * (ddbar * np.abs(sb @ ybar)).sum()
                  + 2.0 * (kp + 2) * F32 * nb * np.linalg.norm(np.abs(dbar) @ asb)
                  + F32 * np.abs(ybar).sum() * (np.abs(dbar) * rowmax).sum())
            b_bound[b] = sq / (2.0 * nb)
        else:
            b_bound[b] = np.linalg.norm(ddbar @ asb)
    return e_bound, b_bound


def _check_audit(got, want, c, R, rule=pair.RULE_HT, wmax=0.0):
    assert int(got["status"].item()) == 0
    assert np.array_equal(got["edge_count"].cpu().numpy(), want["edge_count"])
    reps = got["rep_sqerr"].cpu().numpy().astype(np.float64)
    mse, bias = got["mse"].cpu().numpy(), got["bias_norm"].cpu().numpy()
    e_bound, b_bound = _audit_rounding_bounds(c, R, rule, wmax)
    e_err = rel_l2(reps, want["rep_sqerr"])
    e_ok = np.abs(reps - want["rep_sqerr"]) <= np.maximum(BF16_TOL * want["rep_sqerr"], BOUND_FACTOR * e_bound)
    m_abs = np.abs(mse - want["mse"])
    m_ok = m_abs <= np.maximum(BF16_TOL * want["mse"], BOUND_FACTOR * e_bound.mean(axis=1))
    b_abs = np.abs(bias - want["bias_norm"])
    b_ok = b_abs <= np.maximum(BIAS_TOL * want["bias_norm"], BOUND_FACTOR * b_bound)
    m_rel = np.max(m_abs / np.maximum(want["mse"], 1e-300))
    b_rel = np.max(b_abs / np.maximum(want["bias_norm"], 1e-300))
    log(f"  rep_sqerr rel L2 {e_err:.2e}, max mse rel {m_rel:.2e}, max bias rel {b_rel:.2e}; "
        f"largest error / rounding bound: e_r {np.max(np.abs(reps - want['rep_sqerr']) / np.maximum(e_bound, 1e-300)):.2f}")
    assert e_err <= BF16_TOL
    assert e_ok.all(), f"e_r beyond its bar at {np.argwhere(~e_ok)[:4].tolist()}"
    assert m_ok.all(), f"MSE beyond its bar for prompts {np.flatnonzero(~m_ok).tolist()}"
    assert b_ok.all(), f"bias beyond its bar for prompts {np.flatnonzero(~b_ok).tolist()}"


@pytest.mark.parametrize("case_id", range(48))
def test_random_audit(case_id):
    rng = np.random.default_rng(9100 + case_id)
    c = _case(rng, 5, (1, 33, 500, 2047, 2049, 3000), bf16=True)
    R = int(rng.choice([1, 31, 32, 33, 63, 64, 65, 100, 129]))
    B, nv, gmax = c["B"], c["nv"], c["gmax"]
    log(f"random audit {case_id}: B={B} nv={nv} gmax={gmax} D={c['D']} ld={c['ld']} R={R} "
        f"rep0={c['rep0']}")
    off = torch.from_numpy(c["offsets"]).to(DEV)
    got = pair.audit(off, c["dev"], torch.from_numpy(c["rewards"]).to(DEV),
                     torch.from_numpy(c["p"]).to(DEV), c["seed"], c["rep0"], R, gmax, nv=nv)
    torch.cuda.synchronize()
    want = oracle.audit(c["offsets"], c["host"], c["rewards"], c["p"], c["seed"], c["rep0"], R,
                        gmax=gmax)
    _check_audit(got, want, c, R)


RULES = [pair.RULE_HT, pair.RULE_UNWEIGHTED, pair.RULE_RATIO_KE, pair.RULE_CLIPPED,
         pair.RULE_SELFNORM, pair.RULE_MARGINAL]
LINEAR_RULES = [pair.RULE_HT, pair.RULE_UNWEIGHTED, pair.RULE_CLIPPED, pair.RULE_MARGINAL]


def _rel_max(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b) / np.maximum(np.abs(b), 1e-30))) if a.size else 0.0


def _wmax(rng, rule):
    return float(rng.choice([2.0, 10.0, 50.0])) if rule == pair.RULE_CLIPPED else 0.0


@pytest.mark.parametrize("case_id", range(36))
def test_random_rule_coefficients_and_gradient(case_id):
    rng = np.random.default_rng(9500 + case_id)
    c = _case(rng, 16, WIDTHS)
    rule = RULES[case_id % len(RULES)]
    wmax = _wmax(rng, rule)
    B, nv, gmax = c["B"], c["nv"], c["gmax"]
    log(f"random rule {rule} (wmax {wmax}) case {case_id}: B={B} nv={nv} gmax={gmax} D={c['D']} "
        f"{'bf16' if c['bf16'] else 'fp32'}")
    off = torch.from_numpy(c["offsets"]).to(DEV)
    rew = torch.from_numpy(c["rewards"]).to(DEV)
    d = pair.design_inclusion(off, torch.from_numpy(c["p"]).to(DEV), c["seed"], c["rep0"], 1, gmax,
                              nv=nv)
    co = pair.edge_coeffs(off, rew, d["mask"][0], d["pi"], gmax, nv=nv, rule=rule, wmax=wmax)
    g = pair.weighted_grad(off, c["dev"], co["coeff"], nv=nv)
    torch.cuda.synchronize()
    assert int(co["status"].item()) == 0
    od = oracle.design_inclusion(c["offsets"], c["p"], c["seed"], c["rep0"], 1, gmax)
    assert np.array_equal(d["mask"].cpu().numpy(), od["mask"])
    oc = oracle.pair_coeffs_rule(c["offsets"], c["rewards"], mask=od["mask"][0], pi=od["pi"],
                                 rule=rule, wmax=wmax)
    coeff = co["coeff"].cpu().numpy()
    assert rel_l2(coeff, oc["coeff"]) <= FP32_TOL
    if rule != pair.RULE_MARGINAL:   # the marginal-only fold is not centred, so not antisymmetric
        assert np.all(coeff[oc["coeff"] == 0.0] == 0.0)
    assert np.array_equal(co["edge_count"].cpu().numpy(), oc["edge_count"])
    assert _rel_max(co["ess"].cpu().numpy(), oc["ess"]) <= 1e-5
    assert _rel_max(co["max_weight"].cpu().numpy(), oc["max_weight"]) <= 1e-6
    og = oracle.pair_grad_rule(c["offsets"], c["host"], c["rewards"], mask=od["mask"][0],
                               pi=od["pi"], rule=rule, wmax=wmax)
    err = rel_l2(g["out"].cpu().numpy(), og["out"])
    log(f"  coeff rel L2 {rel_l2(coeff, oc['coeff']):.2e}, grad rel L2 {err:.2e}")
    assert err <= (BF16_TOL if c["bf16"] else FP32_TOL)


@pytest.mark.parametrize("case_id", range(24))
def test_random_rule_audit(case_id):
    rng = np.random.default_rng(9700 + case_id)
    c = _case(rng, 4, (33, 500, 2049), bf16=True)
    rule = RULES[case_id % len(RULES)]
    wmax = _wmax(rng, rule)
    R = int(rng.choice([31, 64, 65, 129]))
    B, nv, gmax = c["B"], c["nv"], c["gmax"]
    log(f"random rule audit {rule} case {case_id}: B={B} gmax={gmax} D={c['D']} R={R}")
    off = torch.from_numpy(c["offsets"]).to(DEV)
    got = pair.audit(off, c["dev"], torch.from_numpy(c["rewards"]).to(DEV),
                     torch.from_numpy(c["p"]).to(DEV), c["seed"], c["rep0"], R, gmax, nv=nv,
                     rule=rule, wmax=wmax)
    torch.cuda.synchronize()
    want = oracle.audit(c["offsets"], c["host"], c["rewards"], c["p"], c["seed"], c["rep0"], R,
                        gmax=gmax, rule=rule, wmax=wmax)
    _check_audit(got, want, c, R, rule, wmax)
    # The update-direction column of the same replicates.
    dirn = pair.audit_direction(off, c["dev"], torch.from_numpy(c["rewards"]).to(DEV),
                                torch.from_numpy(c["p"]).to(DEV), c["seed"], c["rep0"], R, gmax,
                                rule=rule, wmax=wmax, nv=nv)
    torch.cuda.synchronize()
    assert int(dirn["status"].item()) == 0
    cos, tn = dirn["cosine"].cpu().numpy(), dirn["target_norm"].cpu().numpy()
    live = want["target_norm"] > 0
    assert np.all(cos[~live] == 0.0) and np.all(tn[~live] == 0.0)
    c_err = float(np.max(np.abs(cos - want["cosine"])))
    t_err = float(np.max(np.abs(tn[live] / want["target_norm"][live] - 1.0))) if live.any() else 0.0
    log(f"  cosine max abs {c_err:.2e}, target norm max rel {t_err:.2e}")
    assert c_err <= 1e-5 and t_err <= 1e-5


@pytest.mark.parametrize("case_id", range(24))
def test_random_exact_audit(case_id):
    rng = np.random.default_rng(9900 + case_id)
    c = _case(rng, 6, (1, 100, 513, 2049, 5000), bf16=True)
    rule = LINEAR_RULES[case_id % len(LINEAR_RULES)]
    wmax = _wmax(rng, rule)
    B, nv, gmax = c["B"], c["nv"], c["gmax"]
    log(f"random exact audit {rule} case {case_id}: B={B} gmax={gmax} D={c['D']} ld={c['ld']}")
    off = torch.from_numpy(c["offsets"]).to(DEV)
    got = pair.audit_exact(off, c["dev"], torch.from_numpy(c["rewards"]).to(DEV),
                           torch.from_numpy(c["p"]).to(DEV), gmax, rule=rule, wmax=wmax, nv=nv)
    torch.cuda.synchronize()
    want = oracle.audit_exact(c["offsets"], c["host"], c["rewards"], c["p"], gmax=gmax, rule=rule,
                              wmax=wmax)
    assert int(got["status"].item()) == 0
    mse, bias = got["mse"].cpu().numpy(), got["bias_norm"].cpu().numpy()
    zero = want["mse"] == 0.0                    # equal rewards: every edge vector is 0
    assert np.all(mse[zero] == 0.0) and np.all(bias[zero] == 0.0)
    live = ~zero
    m_err = np.max(np.abs(mse[live] - want["mse"][live]) / want["mse"][live]) if live.any() else 0.0
    b_abs = np.abs(bias - want["bias_norm"])
    b_ok = (b_abs <= 2e-3 * want["bias_norm"]) | (b_abs <= 1e-4 * np.sqrt(want["mse"]))
    log(f"  max mse rel {m_err:.2e}, max bias abs {b_abs.max():.2e}")
    assert m_err <= BF16_TOL and b_ok.all()
