"""GPU parity for the exact design audit (Prop. 1), through the C ABI:
closed-form MSE and bias against the oracle for every linear rule (reduced
sizes with ragged tails, and sampled prompts at full size), the Gram output
against an fp64 host product of the same bf16 rows, and the Monte-Carlo
audit of the full workload against the exact MSE (a z-test per prompt).
Bars: MSE within 2e-3 relative (bf16 scores); bias within 2e-3 relative, or
within 1e-4 of sqrt(MSE) where the exact bias is zero (HT).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11368_amd as pair
import workloads as wl
from tests.gpu_util import DEV, log, scores_to_device, scores_to_host, upload_meta

pytestmark = pytest.mark.gpu

LINEAR = [("ht", pair.RULE_HT, 0.0), ("unweighted", pair.RULE_UNWEIGHTED, 0.0),
          ("clipped", pair.RULE_CLIPPED, 8.0), ("marginal", pair.RULE_MARGINAL, 0.0)]


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pair.lib()
    yield
    torch.cuda.synchronize()


def _check(got, want, label):
    mse, bias = got["mse"].cpu().numpy(), got["bias_norm"].cpu().numpy()
    zero = want["mse"] == 0.0                    # equal rewards: every edge vector is 0
    assert np.all(mse[zero] == 0.0) and np.all(bias[zero] == 0.0)
    live = ~zero
    m_err = np.max(np.abs(mse[live] - want["mse"][live]) / want["mse"][live]) if live.any() else 0.0
    b_abs = np.abs(bias - want["bias_norm"])
    b_ok = (b_abs <= 2e-3 * want["bias_norm"]) | (b_abs <= 1e-4 * np.sqrt(want["mse"]))
    log(f"  {label}: max mse rel {m_err:.2e}, max bias abs {b_abs.max():.2e}")
    assert int(got["status"].item()) == 0
    assert m_err <= 2e-3 and b_ok.all()


@pytest.mark.parametrize("name,rule,wmax", LINEAR)
@pytest.mark.parametrize("wname,B,D,G", [("audit", 6, 4096 + 40, None), ("ragged", 12, 777, None),
                                         ("audit", 4, 3000, 20), ("audit", 3, 1500, 40),
                                         ("audit", 3, 100, None), ("ragged", 5, 1, None)])
def test_exact_audit_vs_oracle(name, rule, wmax, wname, B, D, G):
    w = wl.WORKLOADS[wname].replace(B=B, D=D)
    if G is not None:
        w = w.replace(G=G)
    meta = wl.host_meta(w)
    log(f"exact audit {name} {wname} B={B} D={D} gmax={meta.gmax}")
    dm = upload_meta(meta)
    ld = (w.D + 7) // 8 * 8
    s = wl.host_scores(w, meta.nv, ld=ld)
    sd = scores_to_device(s, w)[:, : w.D]
    got = pair.audit_exact(dm["offsets"], sd, dm["rewards"], dm["p"], meta.gmax, rule=rule,
                           wmax=wmax, nv=meta.nv)
    torch.cuda.synchronize()
    want = oracle.audit_exact(meta.offsets, s[:, : w.D], meta.rewards, meta.p, gmax=meta.gmax,
                              rule=rule, wmax=wmax)
    _check(got, want, name)


def test_gram_output_matches_host_product():
    w = wl.WORKLOADS["ragged"].replace(B=10, D=2049)
    meta = wl.host_meta(w)
    dm = upload_meta(meta)
    ld = (w.D + 7) // 8 * 8
    s = wl.host_scores(w, meta.nv, ld=ld)
    sd = scores_to_device(s, w)[:, : w.D]
    got = pair.audit_exact(dm["offsets"], sd, dm["rewards"], dm["p"], meta.gmax, want_gram=True,
                           nv=meta.nv)
    torch.cuda.synchronize()
    sf = sd.float().cpu().numpy().astype(np.float64)
    gram = got["gram"].cpu().numpy()
    for b in range(meta.B):
        lo, hi = meta.offsets[b], meta.offsets[b + 1]
        K = sf[lo:hi] @ sf[lo:hi].T
        g = hi - lo
        err = np.max(np.abs(gram[b, :g, :g] - K)) / np.max(np.abs(K))
        assert err <= 1e-5, (b, err)


@pytest.mark.parametrize("B,G,D", [(64, 16, 140001), (50, 40, 90001)])
def test_gram_multi_chunk_slices(B, G, D):
    """Shapes whose column slices hold several 512-column chunks, so the
    staged loads run ahead of the multiplication (two chunks ahead for
    G <= 16, one above), with a ragged last chunk; the Gram blocks against
    an fp64 host product of the same bf16 rows."""
    w = wl.WORKLOADS["audit"].replace(B=B, G=G, D=D)
    meta = wl.host_meta(w)
    log(f"gram multi-chunk B={B} G={G} D={D}")
    dm = upload_meta(meta)
    sd = wl.device_scores(w, meta.nv, DEV, ld=(D + 7) // 8 * 8)[:, :D]   # 16-byte aligned rows
    got = pair.audit_exact(dm["offsets"], sd, dm["rewards"], dm["p"], meta.gmax, want_gram=True,
                           nv=meta.nv)
    torch.cuda.synchronize()
    assert int(got["status"].item()) == 0
    gram = got["gram"].cpu().numpy()
    worst = 0.0
    for b in range(meta.B):
        lo, hi = meta.offsets[b], meta.offsets[b + 1]
        sf = sd[lo:hi].float().cpu().numpy().astype(np.float64)
        K = sf @ sf.T
        err = np.max(np.abs(gram[b, : hi - lo, : hi - lo] - K)) / np.max(np.abs(K))
        worst = max(worst, err)
    log(f"  max rel err {worst:.2e}")
    assert worst <= 1e-5


def test_exact_audit_rejects_ratio_rules():
    w = wl.WORKLOADS["audit"].replace(B=2, D=64)
    meta = wl.host_meta(w)
    dm = upload_meta(meta)
    sd = wl.device_scores(w, meta.nv, DEV)
    for rule in (pair.RULE_RATIO_KE, pair.RULE_SELFNORM):
        with pytest.raises(pair.PairError):
            pair.audit_exact(dm["offsets"], sd, dm["rewards"], dm["p"], meta.gmax, rule=rule,
                             nv=meta.nv)


@pytest.mark.timeout(400)
def test_full_size_exact_audit_and_monte_carlo_consistency():
    """The audit workload at full size: the exact audit of three prompts
    against the oracle, and the Monte-Carlo audit (R = 4096) of every prompt
    against the exact MSE (z-test with the replicates' own spread)."""
    w = wl.WORKLOADS["audit"]
    meta = wl.host_meta(w)
    log(f"full-size exact audit B={meta.B} D={w.D}")
    dm = upload_meta(meta)
    sd = wl.device_scores(w, meta.nv, DEV)
    ex = pair.audit_exact(dm["offsets"], sd, dm["rewards"], dm["p"], meta.gmax, nv=meta.nv)
    mc = pair.audit(dm["offsets"], sd, dm["rewards"], dm["p"], w.design_seed, 0, w.R, meta.gmax,
                    nv=meta.nv)
    torch.cuda.synchronize()
    assert int(ex["status"].item()) == 0 and int(mc["status"].item()) == 0
    for b in (0, 77, 255):
        lo, hi = meta.offsets[b], meta.offsets[b + 1]
        s_host = scores_to_host(sd[lo:hi])
        want = oracle.audit_exact(np.array([0, hi - lo]), s_host, meta.rewards[lo:hi],
                                  meta.p[lo:hi])
        got = {"mse": ex["mse"][b:b + 1], "bias_norm": ex["bias_norm"][b:b + 1],
               "status": ex["status"]}
        _check(got, want, f"prompt {b}")
    e_mse = ex["mse"].cpu().numpy()
    m_mse = mc["mse"].cpu().numpy()
    reps = mc["rep_sqerr"].cpu().numpy().astype(np.float64)
    sd_mc = reps.std(axis=1) / np.sqrt(w.R)
    live = e_mse > 0
    z = (m_mse[live] - e_mse[live]) / sd_mc[live]
    log(f"  z over {live.sum()} prompts: mean {z.mean():+.3f}, max |z| {np.abs(z).max():.2f}")
    assert np.all(m_mse[~live] == 0.0)
    assert abs(z.mean()) <= 4.0 / np.sqrt(live.sum()) + 0.05 and np.abs(z).max() <= 5.5
    del sd
    torch.cuda.empty_cache()


def test_audit_at_the_papers_fifty_thousand_draws():
    """The Monte-Carlo audit at the paper's draw count (R = 50,000; Sec. 6.2)
    on 64 prompts of the audit workload at full width: every prompt's MSE
    within 5 standard errors of its exact Prop. 1 value, the bias norm of the
    unbiased HT estimator at the sqrt(MSE / R) scale, and the replicate range
    split into two calls equal to one call."""
    w = wl.WORKLOADS["audit"].replace(B=64)
    meta = wl.host_meta(w)
    R = 50000
    log(f"audit at R={R}: B={meta.B} D={w.D}")
    dm = upload_meta(meta)
    sd = wl.device_scores(w, meta.nv, DEV)
    ex = pair.audit_exact(dm["offsets"], sd, dm["rewards"], dm["p"], meta.gmax, nv=meta.nv)
    mc = pair.audit(dm["offsets"], sd, dm["rewards"], dm["p"], w.design_seed, 0, R, meta.gmax,
                    nv=meta.nv)
    half = pair.audit(dm["offsets"], sd, dm["rewards"], dm["p"], w.design_seed, R // 2, R // 2,
                      meta.gmax, nv=meta.nv)
    torch.cuda.synchronize()
    assert int(ex["status"].item()) == 0 and int(mc["status"].item()) == 0
    e_mse, m_mse = ex["mse"].cpu().numpy(), mc["mse"].cpu().numpy()
    reps = mc["rep_sqerr"].cpu().numpy().astype(np.float64)
    live = e_mse > 0
    se = reps.std(axis=1) / np.sqrt(R)
    z = (m_mse[live] - e_mse[live]) / se[live]
    bias = mc["bias_norm"].cpu().numpy()
    ratio = bias[live] / np.sqrt(e_mse[live] / R)
    log(f"  z over {live.sum()} prompts: mean {z.mean():+.3f}, max |z| {np.abs(z).max():.2f}; "
        f"bias / sqrt(MSE/R): median {np.median(ratio):.2f}, max {ratio.max():.2f}")
    assert np.all(m_mse[~live] == 0.0)
    assert np.abs(z).max() <= 5.0 and abs(z.mean()) <= 4.0 / np.sqrt(live.sum()) + 0.05
    # E||mean_r g_r - t||^2 = MSE / R for HT (Theorem 2): the ratio is a
    # chi-like variable of order 1.
    assert np.median(ratio) <= 2.0 and ratio.max() <= 6.0
    assert torch.equal(half["rep_sqerr"], mc["rep_sqerr"][:, R // 2:])
    del sd
    torch.cuda.empty_cache()
