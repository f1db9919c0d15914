"""Pins for the CPU oracle: each test checks the oracle against something the
paper or the mathematics fixes independently of the oracle's own code --
Theorem 1 (pairwise representation), Theorem 2 (design-unbiasedness, by
exhaustive enumeration of every design outcome), Proposition 1 (unweighted
bias and exact independent-Bernoulli covariance), the Gram-matrix identity,
numpy's independent Philox implementation, and invariants of the estimator.
"""
import itertools
import math

import numpy as np
import pytest

import oracle
import workloads as wl


# ---------------------------------------------------------------- helpers --
def _prompt(rng, g, D, p_grid=None, reward="bern"):
    r = (rng.random(g) < 0.5).astype(np.float32) if reward == "bern" else rng.random(g).astype(np.float32)
    if reward == "bern" and r.min() == r.max():
        r[0] = 1.0 - r[0]
    s = rng.standard_normal((g, D)).astype(np.float32)
    if p_grid:
        # multiples of 1/64: every product p_i p_j is exact in fp32, so the
        # logged rho equals the true joint inclusion probability exactly
        p = (rng.integers(8, 65, size=g) / 64.0).astype(np.float32)
    else:
        p = rng.uniform(0.1, 1.0, g).astype(np.float32)
    return r, s, p


def _single(g):
    return np.array([0, g], dtype=np.int64)


def _pi_block(p):
    g = p.size
    blk = (p[:, None].astype(np.float64) * p[None, :].astype(np.float64)).astype(np.float32)
    np.fill_diagonal(blk, p)
    return blk.reshape(1, g, g)


def _enumerate(r, s, p, pi_for_weights):
    """Every design outcome J in {0,1}^G with its independent-Bernoulli
    probability; returns (probs[2^G], estimates[2^G][D]) from the oracle."""
    g, D = s.shape
    masks = np.array(list(itertools.product([0, 1], repeat=g)), dtype=np.uint8)
    n = masks.shape[0]
    offsets = np.arange(0, (n + 1) * g, g, dtype=np.int64)
    S = np.tile(s, (n, 1))
    R = np.tile(r, n)
    PI = np.repeat(pi_for_weights, n, axis=0)
    est, _ = oracle.pair_grad(offsets, S, R, mask=masks.reshape(-1), pi=PI)
    pd = p.astype(np.float64)
    probs = np.prod(np.where(masks == 1, pd[None, :], 1.0 - pd[None, :]), axis=1)
    return probs, est


def _h(r, s, i, j):
    # Eq. (pair-kernel)
    return 0.5 * (float(r[i]) - float(r[j])) * (s[i].astype(np.float64) - s[j].astype(np.float64))


# ------------------------------------------------------------------ Philox --
def test_philox_matches_numpy_independent_implementation():
    rng = np.random.default_rng(5)
    for _ in range(300):
        ctr = [int(x) for x in rng.integers(0, 2**63, size=4, dtype=np.int64)]
        ctr = [c * 2 + int(rng.integers(0, 2)) for c in ctr]     # full 64-bit range
        key = [int(x) * 2 + 1 for x in rng.integers(0, 2**63, size=2, dtype=np.int64)]
        v = sum(c << (64 * k) for k, c in enumerate(ctr))
        # numpy advances its 256-bit counter before producing a block
        ref = np.random.Philox(counter=(v - 1) % (1 << 256), key=np.array(key, dtype=np.uint64))
        want = ref.random_raw(4)
        got = oracle.philox4x64_10(np.array(ctr, dtype=np.uint64), np.array(key, dtype=np.uint64))
        assert np.array_equal(got, want)


def test_indicator_counter_layout_against_numpy():
    """J_i = [top32(word i&3 of Philox(key=(seed,0), ctr=(r,b,i>>2,0))) < floor(p 2^32)]."""
    rng = np.random.default_rng(6)
    for _ in range(200):
        seed = int(rng.integers(0, 2**62))
        r, b, i = (int(x) for x in rng.integers(0, 5000, size=3))
        p = np.float32(rng.uniform(0.01, 1.0))
        v = r + (b << 64) + ((i >> 2) << 128)
        ref = np.random.Philox(counter=(v - 1) % (1 << 256), key=np.array([seed, 0], dtype=np.uint64))
        u = int(ref.random_raw(4)[i & 3]) >> 32
        want = int(u < math.floor(float(p) * 2.0**32))
        assert oracle.draw_indicator(seed, r, b, i, p) == want
    assert oracle.draw_indicator(123, 0, 0, 0, np.float32(1.0)) == 1


# ----------------------------------------------------------- design draw --
def test_design_draw_logged_rho_and_edge_counts():
    w = wl.WORKLOADS["ragged"].replace(B=40)
    meta = wl.host_meta(w)
    d = oracle.design_inclusion(meta.offsets, meta.p, seed=77, rep0=3, R=25, gmax=meta.gmax)
    k = d["completed"].astype(np.int64)
    assert np.array_equal(d["edge_count"], k * (k - 1) // 2)           # K_E = C(k, 2)
    for b in range(meta.B):
        o0, o1 = meta.offsets[b], meta.offsets[b + 1]
        assert np.array_equal(d["mask"][:, o0:o1].sum(axis=1), k[:, b])
        p = meta.p[o0:o1]
        g = o1 - o0
        blk = d["pi"][b]
        prod = p[:, None] * p[None, :]                     # numpy fp32 multiply, correctly rounded
        off_diag = ~np.eye(g, dtype=bool)
        assert np.array_equal(blk[:g, :g][off_diag], prod[off_diag])
        assert np.array_equal(np.diag(blk[:g, :g]), p)
        assert not blk[g:, :].any() and not blk[:, g:].any()


def test_design_draw_inclusion_frequency_matches_p():
    """Sec. 3.3: P(J_i = 1) = pi_i.  Binomial z-test over many replicates."""
    offsets = np.array([0, 16], dtype=np.int64)
    p = np.linspace(0.05, 1.0, 16).astype(np.float32)
    R = 40000
    d = oracle.design_inclusion(offsets, p, seed=2024, rep0=0, R=R, gmax=16, want_pi=False)
    freq = d["mask"].mean(axis=0)
    pd = p.astype(np.float64)
    se = np.sqrt(np.maximum(pd * (1 - pd), 1e-12) / R)
    z = np.abs(freq - pd) / se
    assert np.all(z[pd < 1] < 5.0)
    assert np.all(freq[pd == 1] == 1.0)
    # pairwise: P(J_i J_j = 1) = pi_i pi_j (independence)
    m = d["mask"].astype(np.float64)
    joint = (m.T @ m) / R
    exp = pd[:, None] * pd[None, :]
    se2 = np.sqrt(np.maximum(exp * (1 - exp), 1e-12) / R)
    zz = np.abs(joint - exp) / se2
    off = ~np.eye(16, dtype=bool) & (exp < 1)
    assert np.all(zz[off] < 5.5)


# -------------------------------------------------- Theorem 1 (LOO form) --
@pytest.mark.parametrize("g", [2, 3, 8, 16, 64])
def test_p_one_reduces_to_leave_one_out(g):
    rng = np.random.default_rng(g)
    r, s, _ = _prompt(rng, g, 37, reward="unif")
    ones = np.ones(g, dtype=np.float32)
    d = oracle.design_inclusion(_single(g), ones, seed=1, rep0=0, R=1, gmax=g)
    assert d["mask"].all() and np.all(d["pi"][0] == 1.0)
    est, ec = oracle.pair_grad(_single(g), s, r, mask=d["mask"][0], pi=d["pi"])
    rd, sd = r.astype(np.float64), s.astype(np.float64)
    loo_baseline = (rd.sum() - rd) / (g - 1)                       # r-bar_{-i}
    loo = ((rd - loo_baseline)[:, None] * sd).sum(axis=0) / g       # Eq. (loo)
    centred = ((rd - rd.mean())[:, None] * sd).sum(axis=0) / (g - 1)
    scale = np.abs(loo).max()
    assert np.max(np.abs(est[0] - loo)) <= 1e-12 * scale
    assert np.max(np.abs(est[0] - centred)) <= 1e-12 * scale
    assert ec[0] == g * (g - 1) // 2
    # group-mean baseline is (G-1)/G times the pair average (Thm 1)
    group_mean = ((rd - rd.mean())[:, None] * sd).sum(axis=0) / g
    assert np.max(np.abs(group_mean - (g - 1) / g * est[0])) <= 1e-12 * scale


# ------------------------------------------ Theorem 2 (design-unbiasedness) --
@pytest.mark.parametrize("g", [2, 3, 5, 8, 10])
def test_enumeration_reproduces_complete_pair_target(g):
    rng = np.random.default_rng(100 + g)
    r, s, p = _prompt(rng, g, 6, p_grid=True)
    pi = _pi_block(p)
    probs, est = _enumerate(r, s, p, pi)
    assert abs(probs.sum() - 1.0) < 1e-12
    mean = probs @ est
    target, _ = oracle.pair_grad(_single(g), s, r)                # Eq. (pair-average)
    assert np.max(np.abs(mean - target[0])) <= 1e-12 * np.abs(target).max()


def test_enumeration_with_fp32_logged_rho_general_p():
    """General fp32 p: the logged rho is rounded once, so unbiasedness holds to fp32 precision."""
    g = 9
    rng = np.random.default_rng(31)
    r, s, p = _prompt(rng, g, 5, reward="unif")
    d = oracle.design_inclusion(_single(g), p, seed=5, rep0=0, R=1, gmax=g)
    probs, est = _enumerate(r, s, p, d["pi"])
    target, _ = oracle.pair_grad(_single(g), s, r)
    assert np.max(np.abs(probs @ est - target[0])) <= 3e-7 * np.abs(target).max()


def test_fewer_than_two_completed_gives_exact_zero():
    g = 6
    rng = np.random.default_rng(7)
    r, s, p = _prompt(rng, g, 11)
    pi = _pi_block(p)
    for mask in ([0] * 6, [0, 0, 1, 0, 0, 0]):
        est, ec = oracle.pair_grad(_single(g), s, r, mask=np.array(mask, np.uint8), pi=pi)
        assert ec[0] == 0 and np.all(est == 0.0)


# ----------------------------------------------------- Proposition 1 -----
@pytest.mark.parametrize("g", [3, 6, 9])
def test_unweighted_bias_closed_form(g):
    """Omitting the inverse inclusion factor (rho := 1 in the weights) biases the
    design mean by (1/M) sum_{i<j} (rho_ij - 1) h_ij."""
    rng = np.random.default_rng(200 + g)
    r, s, p = _prompt(rng, g, 7, p_grid=True)
    ones = np.ones((1, g, g), dtype=np.float32)
    probs, est = _enumerate(r, s, p, ones)
    target, _ = oracle.pair_grad(_single(g), s, r)
    M = g * (g - 1) / 2
    pd = p.astype(np.float64)
    bias = sum((pd[i] * pd[j] - 1.0) * _h(r, s, i, j) for i in range(g) for j in range(i + 1, g)) / M
    got = probs @ est - target[0]
    assert np.max(np.abs(got - bias)) <= 1e-12 * np.abs(target).max() * 10


def test_constant_inclusion_attenuates_by_rho():
    g = 7
    rng = np.random.default_rng(9)
    r, s, _ = _prompt(rng, g, 5)
    q = np.float32(0.75)
    p = np.full(g, q, dtype=np.float32)
    probs, est = _enumerate(r, s, p, np.ones((1, g, g), dtype=np.float32))
    target, _ = oracle.pair_grad(_single(g), s, r)
    assert np.allclose(probs @ est, float(q) ** 2 * target[0], rtol=0, atol=1e-13 * np.abs(target).max())


@pytest.mark.parametrize("g", [3, 5, 8])
def test_exact_design_covariance(g):
    """Prop. 1: exact covariance under independent Bernoulli vertices, with the
    shared-vertex term summed over ordered pairs (symmetric completion)."""
    rng = np.random.default_rng(300 + g)
    D = 4
    r, s, p = _prompt(rng, g, D, p_grid=True)
    probs, est = _enumerate(r, s, p, _pi_block(p))
    target, _ = oracle.pair_grad(_single(g), s, r)
    dev = est - target[0][None, :]
    cov = (dev * probs[:, None]).T @ dev
    M = g * (g - 1) / 2
    pd = p.astype(np.float64)
    H = {(i, j): _h(r, s, i, j) for i in range(g) for j in range(g) if i != j}
    closed = np.zeros((D, D))
    for i in range(g):
        for j in range(i + 1, g):
            closed += (1.0 / (pd[i] * pd[j]) - 1.0) * np.outer(H[i, j], H[i, j])
    for i in range(g):
        for j in range(g):
            for k in range(g):
                if len({i, j, k}) == 3:
                    closed += (1.0 / pd[i] - 1.0) * np.outer(H[i, j], H[i, k])
    closed /= M * M
    assert np.max(np.abs(cov - closed)) <= 1e-11 * np.abs(closed).max()


# ------------------------------------------------------- invariants -------
def test_pair_kernel_symmetry_two_vertices():
    rng = np.random.default_rng(11)
    r = np.array([1.0, 0.0], np.float32)
    s = rng.standard_normal((2, 9)).astype(np.float32)
    p = np.array([0.5, 0.25], np.float32)
    pi = _pi_block(p)
    m = np.ones(2, np.uint8)
    a, _ = oracle.pair_grad(_single(2), s, r, mask=m, pi=pi)
    b, _ = oracle.pair_grad(_single(2), s[::-1].copy(), r[::-1].copy(), mask=m, pi=pi[:, ::-1, ::-1].copy())
    h = _h(r, s, 0, 1)
    assert np.array_equal(a, b)
    assert np.allclose(a[0], h / 0.125, rtol=1e-15, atol=0)          # M = 1, rho = 1/8
    # equal rewards or equal scores: h_ij = 0
    z, _ = oracle.pair_grad(_single(2), s, np.array([1.0, 1.0], np.float32), mask=m, pi=pi)
    assert np.all(z == 0.0)
    z2, _ = oracle.pair_grad(_single(2), np.tile(s[:1], (2, 1)), r, mask=m, pi=pi)
    assert np.all(z2 == 0.0)


def test_linearity_and_permutation_invariance():
    g, D = 12, 10
    rng = np.random.default_rng(12)
    r, s, p = _prompt(rng, g, D, reward="unif")
    d = oracle.design_inclusion(_single(g), p, seed=9, rep0=0, R=1, gmax=g)
    m, pi = d["mask"][0], d["pi"]
    base, _ = oracle.pair_grad(_single(g), s, r, mask=m, pi=pi)
    twice, _ = oracle.pair_grad(_single(g), (2 * s).astype(np.float32), r, mask=m, pi=pi)
    assert np.array_equal(twice, 2 * base)
    perm = rng.permutation(g)
    pip = pi[0][np.ix_(perm, perm)]
    pip = np.triu(pip) + np.triu(pip, 1).T          # keep the i<j entries meaningful
    permuted, _ = oracle.pair_grad(_single(g), s[perm].copy(), r[perm].copy(), mask=m[perm].copy(),
                                   pi=pip.reshape(1, g, g).astype(np.float32))
    assert np.allclose(permuted, base, rtol=0, atol=1e-14 * np.abs(base).max())


def test_coefficients_reproduce_gradient_and_sum_to_zero():
    w = wl.WORKLOADS["ragged"].replace(B=30, D=64)
    meta = wl.host_meta(w)
    s = wl.host_scores(w.replace(dtype=wl.F32), meta.nv)
    d = oracle.design_inclusion(meta.offsets, meta.p, seed=3, rep0=0, R=1, gmax=meta.gmax)
    coeff, ec = oracle.pair_coeffs(meta.offsets, meta.rewards, d["mask"][0], d["pi"])
    est, ec2 = oracle.pair_grad(meta.offsets, s, meta.rewards, d["mask"][0], d["pi"])
    assert np.array_equal(ec, ec2)
    assert np.array_equal(ec, d["edge_count"][0])
    for b in range(meta.B):
        o0, o1 = meta.offsets[b], meta.offsets[b + 1]
        c = coeff[o0:o1]
        recon = c @ s[o0:o1].astype(np.float64)
        assert np.max(np.abs(recon - est[b])) <= 1e-12 * max(np.abs(est[b]).max(), 1e-300)
        assert abs(c.sum()) <= 1e-12 * max(np.abs(c).sum(), 1e-300)
        assert np.all(c[d["mask"][0][o0:o1] == 0] == 0.0)


def test_coefficients_p_one_closed_form():
    g = 16
    rng = np.random.default_rng(13)
    r = rng.random(g).astype(np.float32)
    coeff, _ = oracle.pair_coeffs(_single(g), r)
    rd = r.astype(np.float64)
    assert np.allclose(coeff, (rd - rd.mean()) / (g - 1), rtol=0, atol=1e-15)


def test_bf16_scores_are_widened_exactly():
    import torch

    rng = np.random.default_rng(14)
    x = rng.standard_normal((10, 33)).astype(np.float32)
    bits = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    as_f32 = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()
    offsets = np.array([0, 4, 10], np.int64)
    r = rng.random(10).astype(np.float32)
    a, _ = oracle.pair_grad(offsets, bits, r)
    b, _ = oracle.pair_grad(offsets, as_f32, r)
    assert np.array_equal(a, b)


def test_rows_beyond_d_and_padding_are_not_read():
    w = wl.WORKLOADS["tiny"].replace(D=50)
    meta = wl.host_meta(w)
    s_pad = wl.host_scores(w, meta.nv, ld=64)        # NaN in the padding
    s = np.ascontiguousarray(s_pad[:, :50])
    a, _ = oracle.pair_grad(meta.offsets, s_pad[:, :50], meta.rewards)   # strided view, ld = 64
    b, _ = oracle.pair_grad(meta.offsets, s, meta.rewards)
    assert np.array_equal(a, b) and np.isfinite(a).all()


def test_error_paths():
    g = 4
    rng = np.random.default_rng(15)
    r, s, p = _prompt(rng, g, 3)
    pi = _pi_block(p)
    bad = pi.copy()
    bad[0, 0, 1] = 0.0
    with pytest.raises(oracle.OracleError):
        oracle.pair_grad(_single(g), s, r, mask=np.ones(g, np.uint8), pi=bad)
    # rho = 0 on an edge that is not observed is legal and contributes nothing
    m = np.array([0, 1, 1, 1], np.uint8)
    out, ec = oracle.pair_grad(_single(g), s, r, mask=m, pi=bad)
    assert ec[0] == 3 and np.isfinite(out).all()
    with pytest.raises(oracle.OracleError):
        oracle.pair_grad(np.array([0, 1, 3], np.int64), s[:3], r[:3])
    with pytest.raises(oracle.OracleError):
        oracle.design_inclusion(_single(g), np.array([0.5, 0.0, 0.5, 0.5], np.float32), 1, 0, 1, g)


# ------------------------------------------------------------ the audit ----
def test_audit_replicates_obey_gram_identity():
    """e_r = delta_r^T (S S^T) delta_r with delta_r = A~^(r) - A~^full."""
    w = wl.WORKLOADS["audit"].replace(B=6, D=96, R=40)
    meta = wl.host_meta(w)
    s = wl.host_scores(w, meta.nv)
    res = oracle.audit(meta.offsets, s, meta.rewards, meta.p, seed=w.design_seed, rep0=0, R=w.R)
    d = oracle.design_inclusion(meta.offsets, meta.p, seed=w.design_seed, rep0=0, R=w.R, gmax=meta.gmax)
    import torch

    sf = torch.from_numpy(s.view(np.int16)).view(torch.bfloat16).double().numpy()
    full, _ = oracle.pair_coeffs(meta.offsets, meta.rewards)
    for b in range(meta.B):
        o0, o1 = meta.offsets[b], meta.offsets[b + 1]
        K = sf[o0:o1] @ sf[o0:o1].T
        for r in range(w.R):
            a, ke = oracle.pair_coeffs(np.array([0, o1 - o0], np.int64),
                                       meta.rewards[o0:o1], d["mask"][r][o0:o1], d["pi"][b:b + 1])
            delta = a - full[o0:o1]
            e = delta @ K @ delta
            assert abs(res["rep_sqerr"][b, r] - e) <= 1e-10 * max(e, 1e-30)
            assert res["edge_count"][b, r] == d["edge_count"][r, b] == ke[0]
    assert np.allclose(res["mse"], res["rep_sqerr"].mean(axis=1), rtol=1e-14, atol=0)


def test_audit_cosine_obeys_gram_identity():
    """Per-replicate cosine between estimate and target from the coefficients
    alone: cos_r = A~ K a / (sqrt(A~ K A~) sqrt(a K a)), K = S S^T, a the
    complete-pair coefficients (independent algebra); the mean over
    replicates is the oracle's cosine, |t| = sqrt(a K a)."""
    w = wl.WORKLOADS["audit"].replace(B=6, D=96, R=40)
    meta = wl.host_meta(w)
    s = wl.host_scores(w, meta.nv)
    res = oracle.audit(meta.offsets, s, meta.rewards, meta.p, seed=w.design_seed, rep0=3, R=w.R)
    d = oracle.design_inclusion(meta.offsets, meta.p, seed=w.design_seed, rep0=3, R=w.R,
                                gmax=meta.gmax)
    import torch

    sf = torch.from_numpy(s.view(np.int16)).view(torch.bfloat16).double().numpy()
    full, _ = oracle.pair_coeffs(meta.offsets, meta.rewards)
    for b in range(meta.B):
        o0, o1 = meta.offsets[b], meta.offsets[b + 1]
        K = sf[o0:o1] @ sf[o0:o1].T
        a = full[o0:o1]
        tt = a @ K @ a
        assert abs(res["target_norm"][b] - math.sqrt(tt)) <= 1e-12 * math.sqrt(tt)
        cos = []
        for r in range(w.R):
            u, _ = oracle.pair_coeffs(np.array([0, o1 - o0], np.int64), meta.rewards[o0:o1],
                                      d["mask"][r][o0:o1], d["pi"][b:b + 1])
            uu = u @ K @ u
            cos.append(u @ K @ a / math.sqrt(uu * tt) if uu > 0 and tt > 0 else 0.0)
        assert abs(res["cosine"][b] - np.mean(cos)) <= 1e-10
        assert -1.0 <= res["cosine"][b] <= 1.0


def test_audit_cosine_special_cases():
    """p = 1: every estimate is the target (cosine 1).  G = 2: a draw gives
    t / rho when both candidates continue and 0 otherwise, so the cosine is
    the fraction of such draws.  Equal rewards: zero target, cosine 0.
    Rescaling scores or rewards leaves the cosine unchanged."""
    w = wl.WORKLOADS["audit"].replace(B=4, D=40, R=30)
    meta = wl.host_meta(w)
    s = wl.host_scores(w, meta.nv)
    one = oracle.audit(meta.offsets, s, meta.rewards, np.ones_like(meta.p), seed=1, rep0=0, R=5)
    pos = one["target_norm"] > 0
    assert np.all(np.abs(one["cosine"][pos] - 1.0) <= 1e-12)
    assert np.all(one["cosine"][~pos] == 0.0)

    rng = np.random.default_rng(5)
    off = np.array([0, 2, 4, 6], np.int64)
    r2 = np.array([1, 0, 0.3, 0.9, 0.5, 0.5], np.float32)        # last prompt: equal rewards
    p2 = np.array([0.6, 0.7, 0.4, 0.9, 0.5, 0.8], np.float32)
    s2 = rng.standard_normal((6, 17)).astype(np.float32)
    R = 400
    res = oracle.audit(off, s2, r2, p2, seed=9, rep0=11, R=R)
    d = oracle.design_inclusion(off, p2, seed=9, rep0=11, R=R, gmax=2)
    for b in range(2):
        both = np.mean(d["mask"][:, 2 * b] & d["mask"][:, 2 * b + 1])
        assert abs(res["cosine"][b] - both) <= 1e-12
    assert res["target_norm"][2] == 0.0 and res["cosine"][2] == 0.0
    scaled = oracle.audit(off, (3.0 * s2).astype(np.float32), (2.0 * r2).astype(np.float32), p2,
                          seed=9, rep0=11, R=R)
    assert np.allclose(scaled["cosine"], res["cosine"], rtol=0, atol=1e-12)


def test_audit_p_one_has_zero_error():
    w = wl.WORKLOADS["audit"].replace(B=3, D=40, R=5)
    meta = wl.host_meta(w)
    s = wl.host_scores(w, meta.nv)
    res = oracle.audit(meta.offsets, s, meta.rewards, np.ones_like(meta.p), seed=1, rep0=0, R=5)
    # every replicate equals the target bitwise; only the mean of R copies rounds
    target, _ = oracle.pair_grad(meta.offsets, s, meta.rewards)
    assert np.all(res["mse"] == 0.0)
    assert np.all(res["bias_norm"] <= 1e-15 * np.linalg.norm(target, axis=1))


def test_audit_mse_matches_exact_design_variance():
    """Monte-Carlo audit MSE against the exact expectation E||g^ - g_pair||^2,
    obtained by enumerating every design outcome (Prop. 1)."""
    g, D, R = 8, 12, 20000
    rng = np.random.default_rng(41)
    r, s, p = _prompt(rng, g, D, p_grid=True)
    probs, est = _enumerate(r, s, p, _pi_block(p))
    target, _ = oracle.pair_grad(_single(g), s, r)
    exact = probs @ np.sum((est - target[0]) ** 2, axis=1)
    res = oracle.audit(_single(g), s, r, p, seed=17, rep0=0, R=R)
    e = res["rep_sqerr"][0]
    se = e.std(ddof=1) / math.sqrt(R)
    assert abs(res["mse"][0] - exact) <= 5 * se
    # HT is unbiased (Thm 2): E||mean_r g_r - t||^2 = exact / R
    assert res["bias_norm"][0] ** 2 <= 25 * exact / R


def test_audit_unweighted_bias_converges_to_prop1():
    g, D, R = 6, 5, 40000
    rng = np.random.default_rng(43)
    r, s, p = _prompt(rng, g, D, p_grid=True)
    ones = np.ones((1, g, g), dtype=np.float32)
    res = oracle.audit(_single(g), s, r, p, seed=23, rep0=0, R=R, pi_w=ones)
    M = g * (g - 1) / 2
    pd = p.astype(np.float64)
    bias = sum((pd[i] * pd[j] - 1.0) * _h(r, s, i, j) for i in range(g) for j in range(i + 1, g)) / M
    probs, est = _enumerate(r, s, p, ones)
    target, _ = oracle.pair_grad(_single(g), s, r)
    var = probs @ np.sum((est - (probs @ est)) ** 2, axis=1)
    # ||beta_hat||^2 concentrates at ||bias||^2 + var/R
    want = np.dot(bias, bias) + var / R
    got = res["bias_norm"][0] ** 2
    assert abs(got - want) <= 0.05 * want


def test_audit_subset_with_prompt_ids_matches_full_batch():
    w = wl.WORKLOADS["audit"].replace(B=5, D=33, R=7)
    meta = wl.host_meta(w)
    s = wl.host_scores(w, meta.nv)
    full = oracle.audit(meta.offsets, s, meta.rewards, meta.p, seed=8, rep0=2, R=7)
    b = 3
    o0, o1 = meta.offsets[b], meta.offsets[b + 1]
    sub = oracle.audit(np.array([0, o1 - o0]), np.ascontiguousarray(s[o0:o1]), meta.rewards[o0:o1],
                       meta.p[o0:o1], seed=8, rep0=2, R=7, prompt_id=[b])
    assert np.array_equal(sub["rep_sqerr"][0], full["rep_sqerr"][b])
    assert sub["mse"][0] == full["mse"][b]
