"""GPU parity for the edge-weight rules (estimator variants): coefficients,
ESS and maximum weight, the weighted gradient built from them, and the audit
replay of each rule, all through the C ABI against the CPU oracle.

Bars: coefficients and gradients within 1e-5 relative L2 for fp32 arithmetic
on fp32 inputs, 2e-3 for bf16 scores; ESS and maximum weight within 1e-5
relative; edge counts and masks bit-exact; exact zeros where the oracle is
exactly zero; audit per-replicate errors, MSE and bias norm within 2e-3.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11368_amd as pair
import workloads as wl
from tests.gpu_util import DEV, log, rel_l2, scores_to_device, scores_to_host, upload_meta

pytestmark = pytest.mark.gpu

RULES = [("ht", pair.RULE_HT, 0.0), ("unweighted", pair.RULE_UNWEIGHTED, 0.0),
         ("ratio_ke", pair.RULE_RATIO_KE, 0.0), ("clipped", pair.RULE_CLIPPED, 10.0),
         ("selfnorm", pair.RULE_SELFNORM, 0.0), ("marginal", pair.RULE_MARGINAL, 0.0)]


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pair.lib()
    yield
    torch.cuda.synchronize()


def _rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.max(np.abs(a - b) / np.maximum(np.abs(b), 1e-30))


@pytest.mark.parametrize("name,rule,wmax", RULES)
@pytest.mark.parametrize("wname,B,D", [("b128", 48, 1000 + 8), ("ragged", 64, 512)])
def test_rule_coefficients_and_gradient(name, rule, wmax, wname, B, D):
    w = wl.WORKLOADS[wname].replace(B=B, D=D)
    meta = wl.host_meta(w)
    log(f"rule {name} on {wname} B={B} D={D}")
    dm = upload_meta(meta)
    d = pair.design_inclusion(dm["offsets"], dm["p"], w.design_seed, 0, 1, meta.gmax, nv=meta.nv)
    c = pair.edge_coeffs(dm["offsets"], dm["rewards"], d["mask"][0], d["pi"], meta.gmax,
                         nv=meta.nv, rule=rule, wmax=wmax)
    s = wl.host_scores(w, meta.nv)
    g = pair.weighted_grad(dm["offsets"], scores_to_device(s, w), c["coeff"], nv=meta.nv)
    torch.cuda.synchronize()
    assert int(c["status"].item()) == 0
    od = oracle.design_inclusion(meta.offsets, meta.p, w.design_seed, 0, 1, meta.gmax)
    assert np.array_equal(d["mask"].cpu().numpy(), od["mask"])
    oc = oracle.pair_coeffs_rule(meta.offsets, meta.rewards, mask=od["mask"][0], pi=od["pi"],
                                 rule=rule, wmax=wmax)
    coeff = c["coeff"].cpu().numpy()
    err = rel_l2(coeff, oc["coeff"])
    log(f"  coeff rel L2 {err:.2e}")
    assert err <= 1e-5
    assert np.all(coeff[oc["coeff"] == 0.0] == 0.0) or rule == pair.RULE_MARGINAL
    assert np.array_equal(c["edge_count"].cpu().numpy(), oc["edge_count"])
    ess, mw = c["ess"].cpu().numpy(), c["max_weight"].cpu().numpy()
    assert _rel(ess, oc["ess"]) <= 1e-5 and _rel(mw, oc["max_weight"]) <= 1e-6
    og = oracle.pair_grad_rule(meta.offsets, s, meta.rewards, mask=od["mask"][0], pi=od["pi"],
                               rule=rule, wmax=wmax)
    gerr = rel_l2(g["out"].cpu().numpy(), og["out"])
    log(f"  grad rel L2 {gerr:.2e}")
    assert gerr <= 2e-3


def test_marginal_rule_zero_prompts_are_exact():
    """Under every rule a prompt with fewer than two completed vertices is 0."""
    w = wl.WORKLOADS["b128"].replace(B=16, D=64)
    meta = wl.host_meta(w)
    meta.p[:] = np.float32(0.05)
    dm = upload_meta(meta)
    d = pair.design_inclusion(dm["offsets"], dm["p"], 5, 0, 1, meta.gmax, nv=meta.nv)
    k = d["completed"].cpu().numpy()[0]
    assert np.any(k < 2)
    for name, rule, wmax in RULES:
        c = pair.edge_coeffs(dm["offsets"], dm["rewards"], d["mask"][0], d["pi"], meta.gmax,
                             nv=meta.nv, rule=rule, wmax=wmax)
        co = c["coeff"].cpu().numpy()
        for b in range(meta.B):
            if k[b] < 2:
                lo, hi = meta.offsets[b], meta.offsets[b + 1]
                assert np.all(co[lo:hi] == 0.0), name
                assert c["ess"][b].item() == 0.0 and c["max_weight"][b].item() == 0.0


def test_ht_rule_is_bitwise_the_default_entry_point():
    w = wl.WORKLOADS["ragged"].replace(B=40, D=64)
    meta = wl.host_meta(w)
    dm = upload_meta(meta)
    d = pair.design_inclusion(dm["offsets"], dm["p"], w.design_seed, 0, 1, meta.gmax, nv=meta.nv)
    a = pair.edge_coeffs(dm["offsets"], dm["rewards"], d["mask"][0], d["pi"], meta.gmax, nv=meta.nv)
    b = pair.edge_coeffs(dm["offsets"], dm["rewards"], d["mask"][0], d["pi"], meta.gmax, nv=meta.nv,
                         rule=pair.RULE_HT)
    torch.cuda.synchronize()
    assert torch.equal(a["coeff"], b["coeff"])


@pytest.mark.parametrize("name,rule,wmax", RULES)
def test_audit_rule_vs_oracle(name, rule, wmax):
    w = wl.WORKLOADS["audit"].replace(B=5, D=1000)
    meta = wl.host_meta(w)
    R = 256
    log(f"audit rule {name} B=5 D=1000 R={R}")
    dm = upload_meta(meta)
    ld = (w.D + 7) // 8 * 8
    s = wl.host_scores(w, meta.nv, ld=ld)
    sd = scores_to_device(s, w)[:, : w.D]
    got = pair.audit(dm["offsets"], sd, dm["rewards"], dm["p"], w.design_seed, 0, R, meta.gmax,
                     nv=meta.nv, rule=rule, wmax=wmax)
    torch.cuda.synchronize()
    want = oracle.audit(meta.offsets, s[:, : w.D], meta.rewards, meta.p, w.design_seed, 0, R,
                        gmax=meta.gmax, rule=rule, wmax=wmax)
    assert int(got["status"].item()) == 0
    assert np.array_equal(got["edge_count"].cpu().numpy(), want["edge_count"])
    e_err = rel_l2(got["rep_sqerr"].cpu().numpy(), want["rep_sqerr"])
    m_err = _rel(got["mse"].cpu().numpy(), want["mse"])
    b_err = _rel(got["bias_norm"].cpu().numpy(), want["bias_norm"])
    log(f"  rep_sqerr rel L2 {e_err:.2e}, mse {m_err:.2e}, bias {b_err:.2e}")
    assert e_err <= 2e-3 and m_err <= 2e-3 and b_err <= 2e-3


def test_audit_rule_ht_equals_default_audit():
    w = wl.WORKLOADS["audit"].replace(B=3, D=512)
    meta = wl.host_meta(w)
    dm = upload_meta(meta)
    sd = wl.device_scores(w, meta.nv, DEV)
    a = pair.audit(dm["offsets"], sd, dm["rewards"], dm["p"], 3, 0, 100, meta.gmax, nv=meta.nv)
    b = pair.audit(dm["offsets"], sd, dm["rewards"], dm["p"], 3, 0, 100, meta.gmax, nv=meta.nv,
                   rule=pair.RULE_HT)
    torch.cuda.synchronize()
    for k in ("mse", "bias_norm", "rep_sqerr", "edge_count"):
        assert torch.equal(a[k], b[k])


@pytest.fixture(scope="module")
def audit_full():
    """The audit workload at full size (B=256, G=16, D=65536, R=4096): device
    inputs, the oracle's design draw, the complete-pair target coefficients,
    and the per-prompt Gram matrices K_b = S_b S_b^T in fp64 on the host."""
    w = wl.WORKLOADS["audit"]
    meta = wl.host_meta(w)
    G = w.G
    dm = upload_meta(meta)
    sd = wl.device_scores(w, meta.nv, DEV)
    s_host = scores_to_host(sd)
    K = np.empty((meta.B, G, G), dtype=np.float64)
    for b in range(meta.B):
        sb = (s_host[b * G:(b + 1) * G].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        K[b] = sb @ sb.T
    od = oracle.design_inclusion(meta.offsets, meta.p, w.design_seed, 0, w.R, meta.gmax)
    a_full, _ = oracle.pair_coeffs(meta.offsets, meta.rewards)
    live = np.ptp(meta.rewards.reshape(meta.B, G), axis=1) > 0
    assert 0 < live.sum() < meta.B
    return {"w": w, "meta": meta, "dm": dm, "sd": sd, "s_host": s_host, "K": K, "od": od,
            "a_full": a_full, "live": live}


def _rule_gram_audit(f, rule, wmax, chunk=1024):
    """Every e_r of every prompt as delta_r K delta_r^T, with delta_r the
    oracle's coefficient fold under `rule` for replicate r minus the
    complete-pair target (the estimate is linear in the scores under every
    rule), and the bias norm as sqrt(delta_bar K delta_bar^T).  The folds of
    `chunk` replicates go to the oracle as one batch of chunk x B prompts."""
    meta, od, K, a_full = f["meta"], f["od"], f["K"], f["a_full"]
    R, nv, B, G = f["w"].R, meta.nv, meta.B, f["w"].G
    off_t = (meta.offsets[None, :-1] + nv * np.arange(chunk)[:, None]).reshape(-1)
    off_t = np.append(off_t, chunk * nv).astype(np.int64)
    rew_t = np.tile(meta.rewards, chunk)
    pi_t = np.tile(od["pi"], (chunk, 1, 1))
    e = np.empty((B, R), dtype=np.float64)
    ec = np.empty((R, B), dtype=np.int32)
    dsum = np.zeros((B, G), dtype=np.float64)
    for r0 in range(0, R, chunk):
        fold = oracle.pair_coeffs_rule(off_t, rew_t, od["mask"][r0:r0 + chunk].reshape(-1), pi_t,
                                       rule, wmax)
        d = (fold["coeff"].reshape(chunk, nv) - a_full).reshape(chunk, B, G)
        ec[r0:r0 + chunk] = fold["edge_count"].reshape(chunk, B)
        e[:, r0:r0 + chunk] = (np.einsum("rbi,bij->rbj", d, K) * d).sum(-1).T
        dsum += d.sum(axis=0)
    dbar = dsum / R
    bias = np.sqrt(np.einsum("bi,bij,bj->b", dbar, K, dbar))
    return e, ec, bias


@pytest.mark.parametrize("name,rule,wmax", RULES)
def test_audit_rule_full_size(audit_full, name, rule, wmax):
    """The audit under each edge-weight rule on the full audit workload, in
    the launch pair_audit_rule makes there:
      1. 8 prompts with unequal rewards, spread over the batch, against the
         explicit-edge oracle on replicates 0..255 (which also pins the Gram
         form below to the oracle at this size);
      2. every e_r of every prompt (256 x 4096), the MSE and the bias norm
         against the Gram form, edge counts bit-exact, exact zeros for the
         prompts with equal rewards."""
    f = audit_full
    w, meta, dm, live = f["w"], f["meta"], f["dm"], f["live"]
    G = w.G
    log(f"audit rule {name} full size B={meta.B} D={w.D} R={w.R}")
    got = pair.audit(dm["offsets"], f["sd"], dm["rewards"], dm["p"], w.design_seed, 0, w.R,
                     meta.gmax, nv=meta.nv, rule=rule, wmax=wmax)
    torch.cuda.synchronize()
    assert int(got["status"].item()) == 0
    reps = got["rep_sqerr"].cpu().numpy().astype(np.float64)
    mse = got["mse"].cpu().numpy()
    bias = got["bias_norm"].cpu().numpy()
    e, ec, bias_h = _rule_gram_audit(f, rule, wmax)

    # 1. explicit oracle on 8 live prompts, replicates 0..255
    live_ids = np.flatnonzero(live)
    pick = live_ids[np.unique(np.linspace(0, live_ids.size - 1, 8).round().astype(int))]
    assert pick.size == 8
    rows = np.concatenate([np.arange(meta.offsets[b], meta.offsets[b + 1]) for b in pick])
    sub_off = np.arange(pick.size + 1, dtype=np.int64) * G
    R1 = 256
    want = oracle.audit(sub_off, f["s_host"][rows], meta.rewards[rows], meta.p[rows], w.design_seed,
                        0, R1, prompt_id=pick, rule=rule, wmax=wmax)
    assert np.all(np.linalg.norm(want["rep_sqerr"], axis=1) > 0)
    assert np.array_equal(want["edge_count"], ec[:R1, pick].T)
    assert np.allclose(e[pick, :R1], want["rep_sqerr"], rtol=1e-10, atol=0)
    per_pick = [rel_l2(reps[b, :R1], want["rep_sqerr"][q]) for q, b in enumerate(pick)]
    log(f"  explicit oracle, prompts {pick.tolist()}: worst rep_sqerr rel L2 {max(per_pick):.2e}")
    assert max(per_pick) <= 2e-3

    # 2. every replicate of every prompt
    assert np.array_equal(got["edge_count"].cpu().numpy(), ec.T)
    assert np.all(e[~live] == 0.0) and np.all(bias_h[~live] == 0.0)
    assert np.all(reps[~live] == 0.0) and np.all(mse[~live] == 0.0) and np.all(bias[~live] == 0.0)
    per = np.array([rel_l2(reps[b], e[b]) for b in live_ids])
    m_err = np.max(np.abs(mse[live] - e[live].mean(axis=1)) / e[live].mean(axis=1))
    b_err = np.max(np.abs(bias[live] - bias_h[live]) / bias_h[live])
    log(f"  every e_r vs Gram form: worst prompt rel L2 {per.max():.2e}; "
        f"max mse rel {m_err:.2e}, max bias rel {b_err:.2e}")
    assert rel_l2(reps[live], e[live]) <= 2e-3
    assert per.max() <= 2e-3
    assert m_err <= 2e-3 and b_err <= 2e-3
