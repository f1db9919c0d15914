"""GPU parity: the HIP path, called through the C ABI, against the CPU oracle.

Bars:
  - masks, completed counts, edge counts, logged rho: bit-exact
  - gradients / coefficients: relative L2 <= 1e-5 for fp32 scores,
    <= 2e-3 for bf16 scores (fp32 accumulation on the GPU, fp64 in the oracle)
  - prompts whose estimate is exactly zero (saturated rewards, < 2 completed
    vertices) are exactly zero on the GPU
  - audit: per-replicate squared errors and MSE within 2e-3 relative (fp16
    matrix-core operands after power-of-two scaling), edge counts
    bit-exact; the bias norm within 5e-5 relative: its row, the mean of R
    fp32 deviation rows, is applied in fp32 without the fp16 rounding, so
    its error is the fp32 rounding of that mean (about 2^-24 sqrt(R) times
    a deviation's size over the mean's, 1e-6 at R = 4096) and of a length-D
    dot product
Full-size workloads are checked on sampled columns / prompts, plus
properties that hold at any size.
"""
import math
import itertools

import numpy as np
import pytest
import torch

import oracle
import paper_2608_11368_amd as pair
import workloads as wl
from tests.gpu_util import (DEV, log, rel_l2, scores_to_device, scores_to_host, tile_columns,
                            upload_meta)

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-5
BF16_TOL = 2e-3
BIAS_TOL = 5e-5
# Columns per workgroup tile of the bf16 weighted-gradient kernel.
WGRAD_TILE_BF16 = 4096


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pair.lib()
    yield
    torch.cuda.synchronize()


def _chain_gpu(meta, dm, scores, seed, gmax, rep=0):
    """design draw -> coefficients -> weighted gradient, all through the C ABI."""
    B, nv = meta.B, meta.nv
    d = pair.design_inclusion(dm["offsets"], dm["p"], seed, rep, 1, gmax, nv=nv)
    c = pair.edge_coeffs(dm["offsets"], dm["rewards"], d["mask"][0], d["pi"], gmax, nv=nv)
    g = pair.weighted_grad(dm["offsets"], scores, c["coeff"], nv=nv)
    torch.cuda.synchronize()
    return d, c, g


def _chain_oracle(meta, scores_host, seed, gmax, rep=0):
    d = oracle.design_inclusion(meta.offsets, meta.p, seed, rep, 1, gmax)
    est, ec = oracle.pair_grad(meta.offsets, scores_host, meta.rewards, d["mask"][0], d["pi"])
    return d, est, ec


def _assert_zero_rows(meta, coeff_gpu, out_gpu):
    c = coeff_gpu.cpu().numpy()
    for b in range(meta.B):
        o0, o1 = meta.offsets[b], meta.offsets[b + 1]
        if not np.any(c[o0:o1]):
            assert float(out_gpu[b].abs().max()) == 0.0, f"prompt {b} must be exactly zero"


# ------------------------------------------------------------ design draw --
@pytest.mark.parametrize("name,B,R,rep0", [("tiny", None, 1, 0), ("ragged", None, 3, 5),
                                           ("audit", 64, 40, 1000), ("b128", None, 2, 0)])
def test_design_draw_bit_exact(name, B, R, rep0):
    w = wl.WORKLOADS[name]
    if B:
        w = w.replace(B=B)
    meta = wl.host_meta(w)
    log(f"design draw {name} B={meta.B} R={R} rep0={rep0}")
    dm = upload_meta(meta)
    got = pair.design_inclusion(dm["offsets"], dm["p"], w.design_seed, rep0, R, meta.gmax, nv=meta.nv)
    want = oracle.design_inclusion(meta.offsets, meta.p, w.design_seed, rep0, R, meta.gmax)
    assert np.array_equal(got["mask"].cpu().numpy(), want["mask"])
    assert np.array_equal(got["pi"].cpu().numpy(), want["pi"])
    assert np.array_equal(got["edge_count"].cpu().numpy(), want["edge_count"])
    assert np.array_equal(got["completed"].cpu().numpy(), want["completed"])
    assert int(got["status"].item()) == 0


@pytest.mark.parametrize("gmax", [10, 63, 64])
def test_design_rho_block_odd_gmax(gmax):
    """The logged rho block is written in whole-wave passes over gmax^2
    entries; gmax^2 not a multiple of 64 leaves a partial last pass."""
    w = wl.WORKLOADS["ragged"].replace(B=96, gmax_ragged=gmax)
    meta = wl.host_meta(w)
    assert meta.gmax == gmax
    log(f"design rho block gmax={gmax} B={meta.B}")
    dm = upload_meta(meta)
    got = pair.design_inclusion(dm["offsets"], dm["p"], w.design_seed, 2, 2, gmax, nv=meta.nv)
    want = oracle.design_inclusion(meta.offsets, meta.p, w.design_seed, 2, 2, gmax)
    assert np.array_equal(got["pi"].cpu().numpy(), want["pi"])
    assert np.array_equal(got["mask"].cpu().numpy(), want["mask"])
    coeff = torch.empty(meta.nv, device=DEV)
    mask = torch.empty(meta.nv, dtype=torch.uint8, device=DEV)
    pi = torch.full((meta.B, gmax, gmax), float("nan"), device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    pair.pair_design_coeffs(meta.B, meta.nv, gmax, dm["offsets"], dm["p"], dm["rewards"],
                            w.design_seed, 2, coeff, mask, pi, None, None, st)
    c = pair.edge_coeffs(dm["offsets"], dm["rewards"], got["mask"][0], got["pi"], gmax, nv=meta.nv)
    torch.cuda.synchronize()
    assert int(st.item()) == 0 and int(got["status"].item()) == 0
    assert np.array_equal(pi.cpu().numpy(), want["pi"])
    assert torch.equal(mask, got["mask"][0]) and torch.equal(coeff, c["coeff"])


# ------------------------------------------------------ coefficient fold --
@pytest.mark.parametrize("name", ["tiny", "b128", "ragged"])
def test_edge_coeffs_vs_oracle(name):
    w = wl.WORKLOADS[name]
    meta = wl.host_meta(w)
    log(f"edge coeffs {name} B={meta.B}")
    dm = upload_meta(meta)
    d = oracle.design_inclusion(meta.offsets, meta.p, w.design_seed, 0, 1, meta.gmax)
    mask = torch.from_numpy(d["mask"][0]).to(DEV)
    pi = torch.from_numpy(d["pi"]).to(DEV)
    got = pair.edge_coeffs(dm["offsets"], dm["rewards"], mask, pi, meta.gmax, nv=meta.nv)
    want, ec = oracle.pair_coeffs(meta.offsets, meta.rewards, d["mask"][0], d["pi"])
    c = got["coeff"].cpu().numpy()
    err = rel_l2(c, want)
    log(f"  coeff rel L2 = {err:.3e}")
    assert err <= FP32_TOL
    assert np.all(c[want == 0.0] == 0.0)
    assert np.array_equal(got["edge_count"].cpu().numpy(), ec)
    # unweighted / complete-pair: rho := 1, every vertex completed
    full = pair.edge_coeffs(dm["offsets"], dm["rewards"], None, None, meta.gmax, nv=meta.nv)
    want_full, _ = oracle.pair_coeffs(meta.offsets, meta.rewards)
    assert rel_l2(full["coeff"].cpu().numpy(), want_full) <= FP32_TOL


# --------------------------------------------------- weighted gradient ----
def test_weighted_grad_tiny_fp32_chain():
    w = wl.WORKLOADS["tiny"]
    meta = wl.host_meta(w)
    log("chain tiny fp32")
    dm = upload_meta(meta)
    s = wl.host_scores(w, meta.nv)
    d, c, g = _chain_gpu(meta, dm, scores_to_device(s, w), w.design_seed, meta.gmax)
    od, est, ec = _chain_oracle(meta, s, w.design_seed, meta.gmax)
    assert np.array_equal(d["mask"].cpu().numpy(), od["mask"])
    assert np.array_equal(c["edge_count"].cpu().numpy(), ec)
    err = rel_l2(g["out"].cpu().numpy(), est)
    log(f"  grad rel L2 = {err:.3e}")
    assert err <= FP32_TOL
    _assert_zero_rows(meta, c["coeff"], g["out"])


@pytest.mark.parametrize("name,B,D,pad", [("b128", 32, 4096 + 37, 24), ("qwen3", 16, 8192 + 5, 0),
                                          ("ragged", 96, 2048 + 13, 8), ("audit", 24, 1000, 8)])
def test_weighted_grad_bf16_chain_reduced(name, B, D, pad):
    w = wl.WORKLOADS[name].replace(B=B, D=D)
    meta = wl.host_meta(w)
    ld = (D + 7) // 8 * 8 + pad                     # 16-byte aligned bf16 rows
    log(f"chain {name} B={B} D={D} ld={ld}")
    dm = upload_meta(meta)
    s = wl.host_scores(w, meta.nv, ld=ld)           # NaN in the row padding
    sd = scores_to_device(s, w)[:, :D]              # strided view
    d, c, g = _chain_gpu(meta, dm, sd, w.design_seed, meta.gmax)
    od, est, ec = _chain_oracle(meta, s[:, :D], w.design_seed, meta.gmax)
    assert np.array_equal(d["mask"].cpu().numpy(), od["mask"])
    out = g["out"].cpu().numpy()
    assert np.isfinite(out).all()
    err = rel_l2(out, est)
    log(f"  grad rel L2 = {err:.3e}")
    assert err <= BF16_TOL
    _assert_zero_rows(meta, c["coeff"], g["out"])


def test_weighted_grad_edge_cases():
    """G = 2 and G = 64 groups, one group above 64 rows, D = 1 and ragged
    tails, uncompleted rows holding NaN, prompts with fewer than two completed
    vertices."""
    rng = np.random.default_rng(99)
    sizes = [2, 64, 3, 130, 5, 2, 17]
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    nv = int(offsets[-1])
    for D in (1, 7, 8, 4100):
        log(f"edge cases D={D}")
        ld = (D + 7) // 8 * 8                       # 16-byte aligned rows for both dtypes
        s = rng.standard_normal((nv, D)).astype(np.float32)
        coeff = rng.standard_normal(nv).astype(np.float32)
        coeff[rng.random(nv) < 0.4] = 0.0
        coeff[offsets[2]:offsets[3]] = 0.0          # an all-zero prompt
        s_nan = np.full((nv, ld), np.nan, dtype=np.float32)
        s_nan[:, :D] = s
        s_nan[coeff == 0.0] = np.nan                # never-completed rollouts carry no score
        off_d = torch.from_numpy(offsets).to(DEV)
        c_d = torch.from_numpy(coeff).to(DEV)
        sd = torch.from_numpy(s_nan).to(DEV)[:, :D]
        out = pair.weighted_grad(off_d, sd, c_d, nv=nv)["out"].cpu().numpy()
        want = np.stack([coeff[offsets[b]:offsets[b + 1]].astype(np.float64)
                         @ s[offsets[b]:offsets[b + 1]].astype(np.float64) for b in range(len(sizes))])
        assert np.isfinite(out).all()
        assert rel_l2(out, want) <= FP32_TOL
        assert np.all(out[2] == 0.0)
        # bf16 path with the same rows
        sb = torch.from_numpy(s_nan).to(DEV).to(torch.bfloat16)[:, :D]
        outb = pair.weighted_grad(off_d, sb, c_d, nv=nv)["out"].cpu().numpy()
        sbf = sb.float().cpu().numpy()
        sbf[coeff == 0.0] = 0.0
        wantb = np.stack([coeff[offsets[b]:offsets[b + 1]].astype(np.float64)
                          @ sbf[offsets[b]:offsets[b + 1]].astype(np.float64)
                          for b in range(len(sizes))])
        assert np.isfinite(outb).all() and rel_l2(outb, wantb) <= FP32_TOL
        assert np.all(outb[2] == 0.0)


def test_fewer_than_two_completed_gives_exact_zero():
    w = wl.WORKLOADS["b128"].replace(B=16, D=512)
    meta = wl.host_meta(w)
    meta.p[:] = np.float32(0.02)          # almost every draw completes < 2 vertices ...
    meta.p[12 * 16:] = np.float32(0.9)    # ... except in the last four prompts,
    meta.rewards[12 * 16:] = np.arange(4 * 16) % 2   # which have unequal rewards
    log("k<2 zero prompts")
    dm = upload_meta(meta)
    s = wl.host_scores(w, meta.nv)
    d, c, g = _chain_gpu(meta, dm, scores_to_device(s, w), 77, meta.gmax)
    od, est, _ = _chain_oracle(meta, s, 77, meta.gmax)
    k = d["completed"].cpu().numpy()[0]
    assert np.any(k < 2) and np.any(k >= 2)
    out = g["out"].cpu().numpy()
    for b in range(meta.B):
        if k[b] < 2:
            assert np.all(out[b] == 0.0)
    assert rel_l2(out, est) <= BF16_TOL


@pytest.mark.parametrize("name", ["b128", "ragged", "qwen3"])
def test_full_size_sampled_columns(name):
    """The workload at its full size, in the launch configuration the bench
    times; the oracle recomputes sampled columns from the same
    device-resident scores: a random column inside every 4096-column tile
    the bf16 kernel writes (16,384 tiles for the 2^26-column workload), the
    first and last column of every 16th tile, and the last 16 columns."""
    w = wl.WORKLOADS[name]
    meta = wl.host_meta(w)
    log(f"full size {name} B={meta.B} nv={meta.nv} D={w.D}")
    dm = upload_meta(meta)
    sd = wl.device_scores(w, meta.nv, DEV)
    d, c, g = _chain_gpu(meta, dm, sd, w.design_seed, meta.gmax)
    cols = tile_columns(w.D, WGRAD_TILE_BF16, np.random.default_rng(3))
    log(f"  {cols.size} sampled columns")
    ci = torch.from_numpy(cols).to(DEV)
    s_host = scores_to_host(sd.index_select(1, ci))
    out = g["out"].index_select(1, ci).cpu().numpy()
    od, est, _ = _chain_oracle(meta, s_host, w.design_seed, meta.gmax)
    assert np.array_equal(d["mask"].cpu().numpy(), od["mask"])
    err = rel_l2(out, est)
    log(f"  sampled grad rel L2 = {err:.3e}")
    assert err <= BF16_TOL
    # every prompt with a nonzero estimate is compared on its own too
    live = np.linalg.norm(est, axis=1) > 0
    assert live.sum() >= meta.B // 2
    per = [rel_l2(out[b], est[b]) for b in np.flatnonzero(live)]
    log(f"  worst prompt rel L2 = {max(per):.3e} over {live.sum()} prompts")
    assert max(per) <= BF16_TOL
    _assert_zero_rows(meta, c["coeff"], g["out"])
    assert torch.isfinite(g["out"]).all()
    del sd, g
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,B", [("b128", 128), ("ragged", 512), ("tiny", 4)])
def test_fused_design_coeffs_is_bitwise_the_two_calls(name, B):
    w = wl.WORKLOADS[name].replace(B=B)
    meta = wl.host_meta(w)
    dm = upload_meta(meta)
    log(f"fused design + coefficients {name} B={B}")
    d = pair.design_inclusion(dm["offsets"], dm["p"], w.design_seed, 3, 1, meta.gmax, nv=meta.nv)
    c = pair.edge_coeffs(dm["offsets"], dm["rewards"], d["mask"][0], d["pi"], meta.gmax, nv=meta.nv)
    coeff = torch.empty(meta.nv, device=DEV)
    mask = torch.empty(meta.nv, dtype=torch.uint8, device=DEV)
    pi = torch.empty((meta.B, meta.gmax, meta.gmax), device=DEV)
    ec = torch.empty(meta.B, dtype=torch.int32, device=DEV)
    comp = torch.empty(meta.B, dtype=torch.int32, device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    pair.pair_design_coeffs(meta.B, meta.nv, meta.gmax, dm["offsets"], dm["p"], dm["rewards"],
                            w.design_seed, 3, coeff, mask, pi, ec, comp, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert torch.equal(mask, d["mask"][0]) and torch.equal(pi, d["pi"])
    assert torch.equal(coeff, c["coeff"])
    assert torch.equal(ec, d["edge_count"][0]) and torch.equal(comp, d["completed"][0])
    od = oracle.design_inclusion(meta.offsets, meta.p, w.design_seed, 3, 1, meta.gmax)
    assert np.array_equal(mask.cpu().numpy(), od["mask"][0])
    h = pair.design_coeffs(dm["offsets"], dm["p"], dm["rewards"], w.design_seed, 3, meta.gmax,
                           nv=meta.nv)
    torch.cuda.synchronize()
    assert int(h["status"].item()) == 0
    assert torch.equal(h["coeff"], coeff) and torch.equal(h["mask"], mask)
    assert torch.equal(h["pi"], pi) and torch.equal(h["edge_count"], ec)


# ------------------------------------------- weighted gradient, batch mean --
def test_weighted_grad_mean_tiny_fp32():
    w = wl.WORKLOADS["tiny"]
    meta = wl.host_meta(w)
    log("batch mean tiny fp32")
    dm = upload_meta(meta)
    s = wl.host_scores(w, meta.nv)
    d = pair.design_inclusion(dm["offsets"], dm["p"], w.design_seed, 0, 1, meta.gmax, nv=meta.nv)
    c = pair.edge_coeffs(dm["offsets"], dm["rewards"], d["mask"][0], d["pi"], meta.gmax,
                         nv=meta.nv)
    g = pair.weighted_grad(dm["offsets"], scores_to_device(s, w), c["coeff"], nv=meta.nv,
                           reduce=True)
    torch.cuda.synchronize()
    _, est, _ = _chain_oracle(meta, s, w.design_seed, meta.gmax)
    err = rel_l2(g["out"].cpu().numpy(), est.mean(axis=0))
    log(f"  mean rel L2 = {err:.3e}")
    assert g["out"].shape == (w.D,) and err <= FP32_TOL
    assert int(g["status"].item()) == 0


@pytest.mark.parametrize("name,B,D,pad", [("b128", 32, 4096 + 37, 24), ("ragged", 96, 2048 + 13, 8),
                                          ("qwen3", 16, 1024, 0)])
def test_weighted_grad_mean_bf16_reduced(name, B, D, pad):
    w = wl.WORKLOADS[name].replace(B=B, D=D)
    meta = wl.host_meta(w)
    ld = (D + 7) // 8 * 8 + pad
    log(f"batch mean {name} B={B} D={D} ld={ld}")
    dm = upload_meta(meta)
    s = wl.host_scores(w, meta.nv, ld=ld)           # NaN in the row padding
    sd = scores_to_device(s, w)[:, :D]
    d, c, _ = _chain_gpu(meta, dm, sd, w.design_seed, meta.gmax)
    gm = pair.weighted_grad(dm["offsets"], sd, c["coeff"], nv=meta.nv, reduce=True)
    torch.cuda.synchronize()
    _, est, _ = _chain_oracle(meta, s[:, :D], w.design_seed, meta.gmax)
    out = gm["out"].cpu().numpy()
    assert np.isfinite(out).all()
    err = rel_l2(out, est.mean(axis=0))
    log(f"  mean rel L2 = {err:.3e}")
    assert err <= BF16_TOL


def test_weighted_grad_mean_edge_cases():
    """Groups above 64 rows, D = 1 and ragged tails, NaN in every row with a
    zero coefficient, and an all-zero batch (exactly zero output)."""
    rng = np.random.default_rng(7)
    sizes = [2, 64, 3, 130, 5, 2, 17]
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    nv = int(offsets[-1])
    off_d = torch.from_numpy(offsets).to(DEV)
    for D in (1, 7, 8, 1029, 4100):
        log(f"batch mean edge cases D={D}")
        ld = (D + 7) // 8 * 8
        s = rng.standard_normal((nv, D)).astype(np.float32)
        coeff = rng.standard_normal(nv).astype(np.float32)
        coeff[rng.random(nv) < 0.4] = 0.0
        s_nan = np.full((nv, ld), np.nan, dtype=np.float32)
        s_nan[:, :D] = s
        s_nan[coeff == 0.0] = np.nan
        want = (coeff.astype(np.float64) @ s.astype(np.float64)) / len(sizes)
        sd = torch.from_numpy(s_nan).to(DEV)[:, :D]
        out = pair.weighted_grad(off_d, sd, torch.from_numpy(coeff).to(DEV), nv=nv,
                                 reduce=True)["out"].cpu().numpy()
        assert np.isfinite(out).all() and rel_l2(out, want) <= FP32_TOL
        sb = torch.from_numpy(s_nan).to(DEV).to(torch.bfloat16)[:, :D]
        sbf = sb.float().cpu().numpy()
        sbf[coeff == 0.0] = 0.0
        wantb = (coeff.astype(np.float64) @ sbf[:, :D].astype(np.float64)) / len(sizes)
        outb = pair.weighted_grad(off_d, sb, torch.from_numpy(coeff).to(DEV), nv=nv,
                                  reduce=True)["out"].cpu().numpy()
        assert np.isfinite(outb).all() and rel_l2(outb, wantb) <= FP32_TOL
        zero = pair.weighted_grad(off_d, sd, torch.zeros(nv, device=DEV), nv=nv,
                                  reduce=True)["out"]
        assert bool((zero == 0).all())


@pytest.mark.parametrize("name", ["b128", "ragged", "qwen3"])
def test_weighted_grad_mean_full_size_sampled(name):
    """The workload at full size in batch-mean mode (one, two or four row
    groups per workgroup, the ragged workload's 16,961 rows in several LDS
    chunks), a column in every 1024-column workgroup slice against the
    oracle, and every column against the mean of the per-prompt rows."""
    w = wl.WORKLOADS[name]
    meta = wl.host_meta(w)
    log(f"batch mean full size {name} nv={meta.nv} D={w.D}")
    dm = upload_meta(meta)
    sd = wl.device_scores(w, meta.nv, DEV)
    d, c, g = _chain_gpu(meta, dm, sd, w.design_seed, meta.gmax)
    gm = pair.weighted_grad(dm["offsets"], sd, c["coeff"], nv=meta.nv, reduce=True)
    torch.cuda.synchronize()
    cols = tile_columns(w.D, 1024, np.random.default_rng(5))
    ci = torch.from_numpy(cols).to(DEV)
    s_host = scores_to_host(sd.index_select(1, ci))
    _, est, _ = _chain_oracle(meta, s_host, w.design_seed, meta.gmax)
    err = rel_l2(gm["out"].index_select(0, ci).cpu().numpy(), est.mean(axis=0))
    log(f"  sampled mean rel L2 = {err:.3e}")
    assert err <= BF16_TOL
    # the batch mean of the per-prompt rows, on every column (fp32 rounding only)
    per_prompt_mean = torch.mean(g["out"], dim=0, dtype=torch.float64).cpu().numpy()
    assert rel_l2(gm["out"].double().cpu().numpy(), per_prompt_mean) <= 1e-6
    del sd, g, gm
    torch.cuda.empty_cache()


def test_gpu_enumeration_is_design_unbiased():
    """Theorem 2 on the GPU: all 2^G completion patterns of one population as
    a batch of prompts; probability-weighted mean of the GPU estimates equals
    the complete-pair average."""
    G, D = 8, 300
    rng = np.random.default_rng(8)
    r = (rng.random(G) < 0.5).astype(np.float32)
    r[0], r[1] = 1.0, 0.0
    p = (rng.integers(8, 65, size=G) / 64.0).astype(np.float32)
    s = rng.standard_normal((G, D)).astype(np.float32)
    masks = np.array(list(itertools.product([0, 1], repeat=G)), dtype=np.uint8)
    n = masks.shape[0]
    offsets = np.arange(0, (n + 1) * G, G, dtype=np.int64)
    od = oracle.design_inclusion(np.array([0, G]), p, 1, 0, 1, G)
    pi = np.repeat(od["pi"], n, axis=0)
    log("gpu enumeration G=8")
    off_d = torch.from_numpy(offsets).to(DEV)
    c = pair.edge_coeffs(off_d, torch.from_numpy(np.tile(r, n)).to(DEV),
                         torch.from_numpy(masks.reshape(-1)).to(DEV), torch.from_numpy(pi).to(DEV),
                         G, nv=n * G)
    g = pair.weighted_grad(off_d, torch.from_numpy(np.tile(s, (n, 1))).to(DEV), c["coeff"],
                           nv=n * G)["out"].cpu().numpy().astype(np.float64)
    pd = p.astype(np.float64)
    probs = np.prod(np.where(masks == 1, pd, 1.0 - pd), axis=1)
    target, _ = oracle.pair_grad(np.array([0, G]), s, r)
    assert rel_l2(probs @ g, target[0]) <= FP32_TOL


def test_determinism_bitwise():
    w = wl.WORKLOADS["ragged"].replace(B=64, D=4096)
    meta = wl.host_meta(w)
    log("determinism")
    dm = upload_meta(meta)
    sd = scores_to_device(wl.host_scores(w, meta.nv), w)
    a = _chain_gpu(meta, dm, sd, 5, meta.gmax)[2]["out"].clone()
    b = _chain_gpu(meta, dm, sd, 5, meta.gmax)[2]["out"]
    assert torch.equal(a, b)


def test_status_bits():
    log("status bits")
    offsets = torch.tensor([0, 4, 5, 9], dtype=torch.int64, device=DEV)   # G = 4, 1, 4
    p = torch.full((9,), 0.5, device=DEV)
    p[6] = 1.5
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    mask = torch.empty((1, 9), dtype=torch.uint8, device=DEV)
    pair.pair_design_inclusion(3, 9, 4, offsets, p, 1, 0, 1, mask, None, None, None, st)
    v = int(st.item())
    assert v & pair.ST_BAD_GROUP and v & pair.ST_P_RANGE
    # rho = 0 on an observed edge
    off2 = torch.tensor([0, 3], dtype=torch.int64, device=DEV)
    pi = torch.zeros((1, 3, 3), dtype=torch.float32, device=DEV)
    pi[0, 0, 1] = 0.5
    pi[0, 0, 2] = 0.5
    st.zero_()
    coeff = torch.empty(3, device=DEV)
    pair.pair_edge_coeffs(1, 3, 3, off2, torch.tensor([1.0, 0.0, 1.0], device=DEV),
                          torch.ones(3, dtype=torch.uint8, device=DEV), pi, coeff, None, st)
    assert int(st.item()) & pair.ST_RHO_RANGE
    # the same rho = 0 on an edge that is not observed is legal
    st.zero_()
    pair.pair_edge_coeffs(1, 3, 3, off2, torch.tensor([1.0, 0.0, 1.0], device=DEV),
                          torch.tensor([1, 1, 0], dtype=torch.uint8, device=DEV), pi, coeff, None, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0 and torch.isfinite(coeff).all()
    # batch mean: offsets not monotone, then offsets beyond nv (nothing is read)
    sc = torch.zeros((9, 8), dtype=torch.float32, device=DEV)
    c9 = torch.ones(9, device=DEV)
    gm = torch.empty(8, device=DEV)
    for bad in ([0, 5, 3, 9], [0, 4, 12]):
        st.zero_()
        ob = torch.tensor(bad, dtype=torch.int64, device=DEV)
        pair.pair_weighted_grad(len(bad) - 1, 9, ob, sc, c9, gm, 1, st)
        torch.cuda.synchronize()
        assert int(st.item()) & pair.ST_BAD_GROUP


# ------------------------------------------------------------- the audit --
def _audit_case(w, meta, R, rep0=0, pi_w=None, want_reps=True):
    dm = upload_meta(meta)
    ld = (w.D + 7) // 8 * 8                     # 16-byte aligned bf16 rows
    s = wl.host_scores(w, meta.nv, ld=ld)
    sd = scores_to_device(s, w)[:, : w.D]
    s = s[:, : w.D]
    pw = None if pi_w is None else torch.from_numpy(pi_w).to(DEV)
    got = pair.audit(dm["offsets"], sd, dm["rewards"], dm["p"], w.design_seed, rep0, R, meta.gmax,
                     pi_w=pw, want_reps=want_reps, nv=meta.nv)
    torch.cuda.synchronize()
    want = oracle.audit(meta.offsets, s, meta.rewards, meta.p, w.design_seed, rep0, R, pi_w=pi_w,
                        gmax=meta.gmax)
    return got, want


def _wide_range_scores(kind, nv, D, seed):
    """Score rows of wide dynamic range as bf16 bits: magnitudes log-uniform
    over 2^-30 .. 2^0 with random signs, or standard Cauchy entries (heavy
    tails: a row's largest entry is hundreds of times its typical one)."""
    rng = np.random.default_rng(seed)
    if kind == "loguniform":
        x = np.exp2(-30.0 * rng.random((nv, D))) * np.where(rng.random((nv, D)) < 0.5, -1.0, 1.0)
    else:
        x = np.tan(np.pi * (rng.random((nv, D)) - 0.5))
    return torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16) \
        .numpy().view(np.uint16)


def _check_audit(got, want, label):
    mse, bias = got["mse"].cpu().numpy(), got["bias_norm"].cpu().numpy()
    assert int(got["status"].item()) == 0
    assert np.array_equal(got["edge_count"].cpu().numpy(), want["edge_count"])
    e_err = rel_l2(got["rep_sqerr"].cpu().numpy(), want["rep_sqerr"])
    m_err = np.max(np.abs(mse - want["mse"]) / np.maximum(want["mse"], 1e-300))
    b_err = np.max(np.abs(bias - want["bias_norm"]) / np.maximum(want["bias_norm"], 1e-300))
    log(f"  {label}: rep_sqerr rel L2 {e_err:.2e}, max mse rel {m_err:.2e}, max bias rel {b_err:.2e}")
    assert e_err <= BF16_TOL
    assert m_err <= BF16_TOL
    assert b_err <= BIAS_TOL


@pytest.mark.parametrize("name,B,D,R,G", [("audit", 6, 4096 + 40, 300, None),
                                          ("audit", 3, 1000, 600, 40),
                                          ("ragged", 12, 777, 130, None),
                                          ("audit", 2, 512, 2000, 64)])
def test_audit_reduced_vs_oracle(name, B, D, R, G):
    w = wl.WORKLOADS[name].replace(B=B, D=D, dtype=wl.BF16)
    if G:
        w = w.replace(G=G)
    meta = wl.host_meta(w)
    log(f"audit {name} B={B} D={D} R={R} gmax={meta.gmax}")
    got, want = _audit_case(w, meta, R)
    _check_audit(got, want, name)


@pytest.mark.parametrize("kind", ["loguniform", "cauchy"])
@pytest.mark.parametrize("G", [16, 64])
def test_audit_wide_dynamic_range(kind, G):
    """Score rows whose entries span many binades: the matrix-core operands
    are the rows rescaled by their slice maximum and rounded to fp16, exact
    within 2^17 of that maximum and rounded to nearest below; the audit must
    still match the oracle within the audit's bars."""
    w = wl.WORKLOADS["audit"].replace(B=4, D=3000, G=G, dtype=wl.BF16)
    meta = wl.host_meta(w)
    s = _wide_range_scores(kind, meta.nv, w.D, 900 + G)
    log(f"audit wide range {kind} G={G} B={meta.B} D={w.D}")
    dm = upload_meta(meta)
    R = 300
    got = pair.audit(dm["offsets"], scores_to_device(s, w), dm["rewards"], dm["p"], w.design_seed,
                     0, R, meta.gmax, nv=meta.nv)
    torch.cuda.synchronize()
    want = oracle.audit(meta.offsets, s, meta.rewards, meta.p, w.design_seed, 0, R)
    _check_audit(got, want, f"{kind} G={G}")


def test_audit_unweighted_and_resumable():
    w = wl.WORKLOADS["audit"].replace(B=4, D=640)
    meta = wl.host_meta(w)
    ones = np.ones((meta.B, meta.gmax, meta.gmax), dtype=np.float32)
    log("audit unweighted (pi_w = 1)")
    got, want = _audit_case(w, meta, 200, pi_w=ones)
    _check_audit(got, want, "unweighted")
    # replicates split over two calls equal one call
    log("audit resumable")
    a, _ = _audit_case(w, meta, 100, rep0=0)
    b, _ = _audit_case(w, meta, 100, rep0=100)
    both, _ = _audit_case(w, meta, 200, rep0=0)
    joined = torch.cat([a["rep_sqerr"], b["rep_sqerr"]], dim=1)
    assert torch.equal(joined, both["rep_sqerr"])


@pytest.mark.parametrize("R,rep0", [(1, 0), (63, 37), (64, 1), (65, 64), (129, 5)])
def test_audit_replicate_counts_at_tile_pair_edges(R, rep0):
    """Replicate rows are padded to whole pairs of 32-row tiles and the
    mean-deviation row follows them: counts just below, at and above a
    pair boundary, each against the oracle."""
    w = wl.WORKLOADS["audit"].replace(B=3, D=700, dtype=wl.BF16)
    meta = wl.host_meta(w)
    log(f"audit R={R} rep0={rep0} B={meta.B} D={w.D}")
    got, want = _audit_case(w, meta, R, rep0=rep0)
    _check_audit(got, want, f"R={R}")


def test_audit_uneven_split_is_bitwise_one_call():
    """Replicates 5..133 in one call and in three calls of 1, 63 and 65
    replicates (ranges straddling tile-pair boundaries): the same e_r."""
    w = wl.WORKLOADS["ragged"].replace(B=5, D=900, dtype=wl.BF16)
    meta = wl.host_meta(w)
    log(f"audit uneven split B={meta.B} gmax={meta.gmax}")
    one, _ = _audit_case(w, meta, 129, rep0=5)
    parts = [_audit_case(w, meta, n, rep0=r0)[0] for r0, n in ((5, 1), (6, 63), (69, 65))]
    for part in parts:
        assert int(part["status"].item()) == 0
    joined = torch.cat([part["rep_sqerr"] for part in parts], dim=1)
    assert torch.equal(joined, one["rep_sqerr"])
    assert torch.equal(torch.cat([part["edge_count"] for part in parts], dim=1), one["edge_count"])


def test_audit_equal_reward_prompts():
    """Prompts whose rewards are all equal have zero deviations in every
    replicate: exact zeros for e_r, MSE and bias, their edge counts still
    drawn, and their score rows never read (NaN there raises nothing).  The
    other prompts match the oracle.  A non-finite score in a prompt that is
    swept sets PAIR_ST_NONFINITE."""
    w = wl.WORKLOADS["audit"].replace(B=9, D=3000, dtype=wl.BF16)
    meta = wl.host_meta(w)
    G = 16
    for b, v in ((1, 1.0), (4, 0.0), (8, 0.37)):
        meta.rewards[b * G:(b + 1) * G] = v
    live = np.ptp(meta.rewards.reshape(meta.B, G), axis=1) > 0
    assert live.sum() >= 3
    s = wl.host_scores(w, meta.nv)
    s_nan = s.copy()
    s_nan[4 * G:5 * G, ::7] = 0x7FC0                     # NaN in a prompt that is not swept
    dm = upload_meta(meta)
    R = 130
    log(f"audit with equal-reward prompts B={meta.B} live={int(live.sum())}")
    got = pair.audit(dm["offsets"], scores_to_device(s_nan, w), dm["rewards"], dm["p"],
                     w.design_seed, 3, R, meta.gmax, nv=meta.nv)
    torch.cuda.synchronize()
    want = oracle.audit(meta.offsets, s, meta.rewards, meta.p, w.design_seed, 3, R)
    assert int(got["status"].item()) == 0
    assert np.array_equal(got["edge_count"].cpu().numpy(), want["edge_count"])
    reps = got["rep_sqerr"].cpu().numpy()
    for name in ("mse", "bias_norm"):
        assert np.all(got[name].cpu().numpy()[~live] == 0.0) and np.all(want[name][~live] == 0.0)
    assert np.all(reps[~live] == 0.0)
    sub = {k: got[k][torch.from_numpy(live).to(DEV)] for k in ("mse", "bias_norm", "rep_sqerr",
                                                                 "edge_count")}
    sub["status"] = got["status"]
    want_live = {k: want[k][live] for k in ("mse", "bias_norm", "rep_sqerr", "edge_count")}
    _check_audit(sub, want_live, "live prompts")
    # every prompt with equal rewards: nothing is swept, everything is exactly zero
    flat = meta.rewards.copy()
    flat[:] = 0.5
    allz = pair.audit(dm["offsets"], scores_to_device(s_nan, w), torch.from_numpy(flat).to(DEV),
                      dm["p"], w.design_seed, 3, R, meta.gmax, nv=meta.nv)
    torch.cuda.synchronize()
    assert int(allz["status"].item()) == 0
    for name in ("mse", "bias_norm", "rep_sqerr"):
        assert bool((allz[name] == 0).all()), name
    assert torch.equal(allz["edge_count"], got["edge_count"])
    # a NaN score in a swept prompt is reported
    b_live = int(np.flatnonzero(live)[0])
    s_bad = s.copy()
    s_bad[b_live * G + 2, 100] = 0x7FC0
    bad = pair.audit(dm["offsets"], scores_to_device(s_bad, w), dm["rewards"], dm["p"],
                     w.design_seed, 3, R, meta.gmax, nv=meta.nv)
    torch.cuda.synchronize()
    assert int(bad["status"].item()) & pair.ST_NONFINITE


def _exact_expected_mse(K, r, p):
    """Prop. 1 trace, E||g^ - g_pair||^2 under independent Bernoulli vertices,
    from the Gram matrix K = S S^T (fp64)."""
    G = r.size
    M = G * (G - 1) / 2
    r = r.astype(np.float64)
    p = p.astype(np.float64)

    def ip(i, j, k, l):      # <h_ij, h_kl>
        return 0.25 * (r[i] - r[j]) * (r[k] - r[l]) * (K[i, k] - K[i, l] - K[j, k] + K[j, l])

    tot = 0.0
    for i in range(G):
        for j in range(i + 1, G):
            tot += (1.0 / (p[i] * p[j]) - 1.0) * ip(i, j, i, j)
    for i in range(G):
        for j in range(G):
            for k in range(G):
                if len({i, j, k}) == 3:
                    tot += (1.0 / p[i] - 1.0) * ip(i, j, i, k)
    return tot / (M * M)


@pytest.mark.timeout(600)
def test_audit_full_size():
    """The audit workload at full size (B=256, G=16, D=65536, R=4096), in the
    launch the bench times.
      1. The explicit-edge oracle on 16 prompts with unequal rewards, spread
         over the batch (and so over the XCD ranges and column slices), every
         replicate.
      2. Every e_r of every prompt (256 x 4096) against delta_r K delta_r^T,
         with the deviations delta_r = A~^(r) - a from the oracle's design
         draw and coefficient fold and K = S S^T in fp64 on the host (the
         Gram identity pinned against the explicit oracle); prompts with equal
         rewards must give exact zeros.
      3. For all prompts the Monte-Carlo MSE against its exact expectation
         (Prop. 1)."""
    w = wl.WORKLOADS["audit"]
    meta = wl.host_meta(w)
    log(f"audit full size B={meta.B} D={w.D} R={w.R}")
    dm = upload_meta(meta)
    sd = wl.device_scores(w, meta.nv, DEV)
    got = pair.audit(dm["offsets"], sd, dm["rewards"], dm["p"], w.design_seed, 0, w.R, meta.gmax,
                     nv=meta.nv)
    torch.cuda.synchronize()
    assert int(got["status"].item()) == 0
    mse = got["mse"].cpu().numpy()
    reps = got["rep_sqerr"].cpu().numpy().astype(np.float64)
    assert np.allclose(mse, reps.mean(axis=1), rtol=1e-6, atol=0)
    G = 16
    rew = meta.rewards.reshape(meta.B, G)
    live = np.ptp(rew, axis=1) > 0
    log(f"  {live.sum()} prompts with unequal rewards, {meta.B - live.sum()} with equal rewards")
    assert 0 < live.sum() < meta.B

    # 1. explicit oracle, 16 live prompts, all replicates, one call
    live_ids = np.flatnonzero(live)
    pick = live_ids[np.unique(np.linspace(0, live_ids.size - 1, 16).round().astype(int))]
    assert pick.size == 16 and pick[0] == live_ids[0] and pick[-1] == live_ids[-1]
    log(f"  oracle on prompts {pick.tolist()}, all replicates")
    rows = np.concatenate([np.arange(meta.offsets[b], meta.offsets[b + 1]) for b in pick])
    sub_off = np.arange(pick.size + 1, dtype=np.int64) * G
    want = oracle.audit(sub_off, scores_to_host(sd.index_select(0, torch.from_numpy(rows).to(DEV))),
                        meta.rewards[rows], meta.p[rows], w.design_seed, 0, w.R,
                        prompt_id=pick)
    assert np.all(np.linalg.norm(want["rep_sqerr"], axis=1) > 0)
    pk = torch.from_numpy(pick).to(DEV)
    sub = {k: got[k].index_select(0, pk) for k in ("mse", "bias_norm", "rep_sqerr", "edge_count")}
    sub["status"] = got["status"]
    _check_audit(sub, want, "16 live prompts")
    for q, b in enumerate(pick):
        e_b = rel_l2(reps[b], want["rep_sqerr"][q])
        assert e_b <= BF16_TOL, f"prompt {b}: rep_sqerr rel L2 {e_b:.2e}"

    # 2. every replicate of every prompt through the Gram identity
    log("  all prompts: oracle draws and folds, K = S S^T on the host")
    od = oracle.design_inclusion(meta.offsets, meta.p, w.design_seed, 0, w.R, meta.gmax)
    assert np.array_equal(got["edge_count"].cpu().numpy(), od["edge_count"].T)
    a_full, _ = oracle.pair_coeffs(meta.offsets, meta.rewards)
    delta = np.empty((w.R, meta.nv), dtype=np.float64)
    for r in range(w.R):
        c_r, _ = oracle.pair_coeffs(meta.offsets, meta.rewards, od["mask"][r], od["pi"])
        delta[r] = c_r - a_full
    delta = delta.reshape(w.R, meta.B, G)
    s_host = scores_to_host(sd)
    e_gram = np.empty((meta.B, w.R), dtype=np.float64)
    for b in range(meta.B):
        sb = (s_host[b * G:(b + 1) * G].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        K = sb @ sb.T
        db = delta[:, b, :]
        e_gram[b] = np.einsum("ri,ij,rj->r", db, K, db)
    del s_host
    assert np.all(e_gram[~live] == 0.0) and np.all(reps[~live] == 0.0)
    assert np.all(mse[~live] == 0.0) and np.all(got["bias_norm"].cpu().numpy()[~live] == 0.0)
    per = np.array([rel_l2(reps[b], e_gram[b]) for b in live_ids])
    tot = rel_l2(reps[live], e_gram[live])
    log(f"  every e_r vs Gram form: rel L2 {tot:.2e}, worst prompt {per.max():.2e} "
        f"(prompt {live_ids[per.argmax()]})")
    assert tot <= BF16_TOL
    assert per.max() <= BF16_TOL

    # 3. every prompt: MC MSE within 6 standard errors of the exact expectation
    S = sd.view(meta.B, 16, w.D).double()
    K = torch.bmm(S, S.transpose(1, 2).contiguous()).cpu().numpy()
    z = []
    for b in range(meta.B):
        o0, o1 = meta.offsets[b], meta.offsets[b + 1]
        ex = _exact_expected_mse(K[b], meta.rewards[o0:o1], meta.p[o0:o1])
        se = reps[b].std(ddof=1) / math.sqrt(w.R)
        if ex == 0.0:
            assert mse[b] <= 1e-12
            continue
        z.append((mse[b] - ex) / max(se, 1e-30))
    z = np.array(z)
    log(f"  MSE z-scores: max |z| = {np.abs(z).max():.2f}, mean z = {z.mean():.3f}")
    assert np.abs(z).max() < 6.0
    assert abs(z.mean()) < 6.0 / math.sqrt(len(z)) + 0.5
