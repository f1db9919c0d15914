"""CPU check of the first-order rounding bound that the random audit tests
accept results within.  The audit's matrix-core operands carry one fp16
rounding of each deviation entry, after its replicate row is rescaled by a
power of two so that the row's largest entry lies in [1, 2).  Emulating that
operand in numpy (float16, round to nearest) on the oracle's own draws and
folds, every replicate's squared error must stay within the bound, also in
single-column cases where the terms delta_ri z_ri cancel and the relative
error is far above 2^-11.
"""
import numpy as np
import pytest

import oracle
from tests import test_gpu_random as T


def _emulated_rep_sqerr(c, R):
    """e_r with each replicate row of A~^(r) - a rounded to fp16 after its
    power-of-two rescaling; the scores are exact (bf16 values)."""
    off = c["offsets"]
    od = oracle.design_inclusion(off, c["p"], c["seed"], c["rep0"], R, c["gmax"])
    a, _ = oracle.pair_coeffs(off, c["rewards"])
    S = (c["host"].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    B = off.size - 1
    exact = np.zeros((B, R))
    rounded = np.zeros((B, R))
    for r in range(R):
        A, _ = oracle.pair_coeffs(off, c["rewards"], od["mask"][r], od["pi"])
        for b in range(B):
            o0, o1 = off[b], off[b + 1]
            d = A[o0:o1] - a[o0:o1]
            m = np.abs(d).max()
            if m == 0.0:
                continue
            f = np.floor(np.log2(m))
            d16 = np.ldexp(np.ldexp(d, -int(f)).astype(np.float16).astype(np.float64), int(f))
            exact[b, r] = np.sum((d @ S[o0:o1]) ** 2)
            rounded[b, r] = np.sum((d16 @ S[o0:o1]) ** 2)
    return exact, rounded


@pytest.mark.parametrize("case_id", [5, 1062, 1064, 1171, 1192] + list(range(2000, 2012)))
def test_fp16_operand_error_within_bound(monkeypatch, case_id):
    monkeypatch.setattr(T, "DEV", "cpu")
    rng = np.random.default_rng(9100 + case_id)
    c = T._case(rng, 5, (1, 33, 500, 2047, 2049, 3000), bf16=True)
    R = int(rng.choice([1, 31, 32, 33, 63, 64, 65, 100, 129]))
    exact, rounded = _emulated_rep_sqerr(c, R)
    want = oracle.audit(c["offsets"], c["host"], c["rewards"], c["p"], c["seed"], c["rep0"], R,
                        gmax=c["gmax"])
    # The emulation's unrounded e_r is the oracle's (Gram identity, fp64).
    assert np.allclose(exact, want["rep_sqerr"], rtol=1e-9, atol=1e-300)
    e_bound, _ = T._audit_rounding_bounds(c, R)
    err = np.abs(rounded - exact)
    assert np.all(err <= e_bound), \
        f"largest error / bound {np.max(err / np.maximum(e_bound, 1e-300)):.3f}"
    # Prompts with equal rewards: zero deviations, zero error, zero bound.
    dead = exact.max(axis=1) == 0.0
    assert np.all(err[dead] == 0.0) and np.all(e_bound[dead] == 0.0)
