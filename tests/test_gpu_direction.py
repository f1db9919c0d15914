"""GPU parity for the audit's update-direction column (the cosine between
each replicate's estimate and the complete-pair target, averaged over
replicates, and the target norm) through the C ABI, against the CPU oracle.

Bar (derived from the arithmetic, none is stated): the GPU forms each
replicate's coefficients to one fp32 rounding and the Gram matrix from fp32
matrix-core partial sums (relative error about 1e-7 per entry), so a
replicate's cosine is off by about 1e-6 at most; the mean over replicates is
held to 1e-5 absolute, the target norm to 1e-5 relative.  Exact values where
the definition fixes them: 0 for a prompt with equal rewards, and for G = 2
the fraction of draws in which both candidates continue.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_11368_amd as pair
import workloads as wl
from tests.gpu_util import DEV, log, scores_to_host, upload_meta

pytestmark = pytest.mark.gpu

COS_TOL = 1e-5
NORM_TOL = 1e-5


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pair.lib()
    yield
    torch.cuda.synchronize()


def _check(got, want, label):
    cos, tn = got["cosine"].cpu().numpy(), got["target_norm"].cpu().numpy()
    dc = float(np.max(np.abs(cos - want["cosine"])))
    pos = want["target_norm"] > 0
    dn = float(np.max(np.abs(tn[pos] / want["target_norm"][pos] - 1.0))) if pos.any() else 0.0
    log(f"  {label}: max |d cos| {dc:.2e}, max rel d|t| {dn:.2e}, mean cos {cos.mean():.4f}")
    assert dc <= COS_TOL and dn <= NORM_TOL
    assert np.all(cos[~pos] == 0.0) and np.all(tn[~pos] == 0.0)
    assert np.all(np.abs(cos) <= 1.0 + 1e-12)


@pytest.mark.parametrize("name,rule,wmax", [("ht", pair.RULE_HT, 0.0),
                                            ("unweighted", pair.RULE_UNWEIGHTED, 0.0),
                                            ("ratio_ke", pair.RULE_RATIO_KE, 0.0),
                                            ("clipped", pair.RULE_CLIPPED, 10.0),
                                            ("selfnorm", pair.RULE_SELFNORM, 0.0),
                                            ("marginal", pair.RULE_MARGINAL, 0.0)])
@pytest.mark.parametrize("wname,B,D,R,rep0", [("audit", 12, 3000, 200, 0),
                                              ("ragged", 10, 1100, 70, 9)])
def test_direction_vs_oracle(name, rule, wmax, wname, B, D, R, rep0):
    w = wl.WORKLOADS[wname].replace(B=B, D=D)
    meta = wl.host_meta(w)
    dm = upload_meta(meta)
    s = wl.device_scores(w, meta.nv, DEV, ld=(D + 7) // 8 * 8)[:, :D]
    log(f"direction {name} on {wname} B={B} D={D} R={R} rep0={rep0} gmax={meta.gmax}")
    got = pair.audit_direction(dm["offsets"], s, dm["rewards"], dm["p"], w.design_seed, rep0, R,
                               meta.gmax, rule=rule, wmax=wmax, nv=meta.nv)
    torch.cuda.synchronize()
    assert int(got["status"].item()) == 0
    want = oracle.audit(meta.offsets, scores_to_host(s), meta.rewards, meta.p, w.design_seed,
                        rep0, R, gmax=meta.gmax, want_reps=False, rule=rule, wmax=wmax)
    _check(got, want, name)


def test_direction_weights_from_pi_w_and_special_prompts():
    """All-ones pi_w (the unweighted replay of Prop. 1), a G = 2 prompt whose
    cosine is the fraction of draws with both candidates continuing, and a
    prompt with equal rewards (zero target)."""
    rng = np.random.default_rng(7)
    sizes = [2, 2, 5, 16, 3]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    nv, B, D, R, gmax = int(off[-1]), len(sizes), 2048 + 24, 300, 16
    rew = rng.uniform(0, 1, nv).astype(np.float32)
    rew[off[4]:off[5]] = 0.25                          # equal rewards: t = 0
    p = rng.uniform(0.2, 1.0, nv).astype(np.float32)
    sc = torch.from_numpy(rng.standard_normal((nv, D)).astype(np.float32)).to(DEV)
    s = sc.to(torch.bfloat16)
    o_d, r_d, p_d = (torch.from_numpy(a).to(DEV) for a in (off, rew, p))
    log(f"direction special prompts B={B} D={D} R={R}")
    got = pair.audit_direction(o_d, s, r_d, p_d, 21, 4, R, gmax, nv=nv)
    ones = torch.ones((B, gmax, gmax), device=DEV)
    got1 = pair.audit_direction(o_d, s, r_d, p_d, 21, 4, R, gmax, pi_w=ones, nv=nv)
    d = pair.design_inclusion(o_d, p_d, 21, 4, R, gmax, nv=nv)
    torch.cuda.synchronize()
    assert int(got["status"].item()) == 0 and int(got1["status"].item()) == 0
    sh = scores_to_host(s)
    want = oracle.audit(off, sh, rew, p, 21, 4, R, gmax=gmax, want_reps=False)
    want1 = oracle.audit(off, sh, rew, p, 21, 4, R, pi_w=np.ones((B, gmax, gmax), np.float32),
                         want_reps=False)
    _check(got, want, "logged rho")
    _check(got1, want1, "all-ones pi_w")
    mask = d["mask"].cpu().numpy()
    for b in (0, 1):
        both = float(np.mean(mask[:, off[b]] & mask[:, off[b] + 1]))
        c = float(got["cosine"][b])
        assert abs(c - both) <= 1e-9, (b, c, both)


def test_direction_full_width_sampled_prompts():
    """The audit workload's full score width (D = 65536) on two prompts."""
    w = wl.WORKLOADS["audit"]
    meta = wl.host_meta(w)
    varied = [b for b in range(meta.B)
              if np.ptp(meta.rewards[meta.offsets[b]:meta.offsets[b + 1]]) > 0]
    keep = [varied[0], varied[len(varied) // 2]]       # two prompts with a nonzero target
    rows = np.concatenate([np.arange(meta.offsets[b], meta.offsets[b + 1]) for b in keep])
    full = wl.device_scores(w, meta.nv, DEV)
    s = full[torch.from_numpy(rows).to(DEV)].contiguous()
    del full
    torch.cuda.empty_cache()
    sizes = [meta.offsets[b + 1] - meta.offsets[b] for b in keep]
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    rew, p = meta.rewards[rows], meta.p[rows]
    R = 256
    log(f"direction full width D={w.D} prompts {keep} R={R}")
    o_d, r_d, p_d = (torch.from_numpy(np.ascontiguousarray(a)).to(DEV) for a in (off, rew, p))
    # Prompt ids are the positions in the subset; the oracle draws with the same ids.
    got = pair.audit_direction(o_d, s, r_d, p_d, w.design_seed, 0, R, meta.gmax, nv=len(rows))
    torch.cuda.synchronize()
    assert int(got["status"].item()) == 0
    want = oracle.audit(off, scores_to_host(s), rew, p, w.design_seed, 0, R, gmax=meta.gmax,
                        want_reps=False)
    _check(got, want, "full width")
    assert np.all(want["target_norm"] > 0)
