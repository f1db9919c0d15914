"""CPU oracle for the PAIR estimator -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never loads it and
shares no code with it; see ``pair_oracle.c`` for the paper passages each
function follows (fp64, explicit edge loops, Philox4x64-10 design draws).

Parity status of each function (what pins it, see ``tests/test_oracle_pins.py``):
  philox4x64_10     pinned: numpy's independent Philox implementation
  design_inclusion  pinned: brute-force edge count, inclusion frequencies vs p
                    (binomial z-test), bit layout of the counter reading
  pair_grad         pinned: p == 1 reduces to the leave-one-out form (Thm 1);
                    exhaustive design enumeration reproduces the complete-pair
                    average (Thm 2); unweighted-bias closed form (Prop 1);
                    linearity, permutation invariance, zero cases
  pair_coeffs       pinned: sum_i A~_i s_i equals pair_grad; A~ sums to zero;
                    p == 1 gives (r_i - mean r)/(G - 1)
  audit             pinned: exact design covariance trace (Prop 1) by
                    enumeration; Gram-matrix identity for every replicate;
                    bias^2 ~ MSE/R statistics; p == 1 gives zero MSE;
                    cosine to the target: the Gram identity over the
                    coefficients per replicate, 1 when p == 1, the fraction of
                    draws with both candidates when G == 2, 0 for equal
                    rewards, invariant to rescaled scores and rewards
  audit_exact       pinned: exhaustive design enumeration of E||g^ - t||^2 and
                    of the mean for every linear rule; zero bias for HT
                    (Thm 2); Prop. 1's unweighted bias vector; zero error
                    when p == 1
  cps_*             conditional Poisson (fixed-size) design: inclusion
                    probabilities pinned by brute force over every sample;
                    the sequential draw's sample probabilities pinned to
                    prod w / e_n by walking every path; the fit's output
                    reproduces its target and returns odds of geometric mean
                    1 (also when the start already meets the target); draw
                    frequencies vs pi and pi_ij
  *_rule variants   pinned by exhaustive design enumeration against the
                    expectations the paper states for each edge-weight rule
                    (naive bias, clipped multiplier min(1, w_max rho) - 1,
                    ratio estimator exact under a self-weighting design),
                    cross-rule identities, ESS special cases; the
                    marginal-only rule against its own enumeration closed
                    form (a reading: the paper names it without a formula)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pair_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# A separately compiled copy of the oracle to load instead of liboracle.so.
# Only the mutation test sets it, to run the pins against deliberately
# broken copies of pair_oracle.c.
_LIB_OVERRIDE = os.environ.get("PAIR_ORACLE_LIB")

F32 = 0
BF16 = 1

# Edge-weight rules (same codes as the C oracle; see pair_oracle.c).
RULE_HT = 0
RULE_UNWEIGHTED = 1
RULE_RATIO_KE = 2
RULE_CLIPPED = 3
RULE_SELFNORM = 4
RULE_MARGINAL = 5
RULES = {"ht": RULE_HT, "unweighted": RULE_UNWEIGHTED, "ratio_ke": RULE_RATIO_KE,
         "clipped": RULE_CLIPPED, "selfnorm": RULE_SELFNORM, "marginal": RULE_MARGINAL}

ERRORS = {
    0: "ok",
    -1: "invalid argument",
    -2: "unknown dtype",
    -3: "observed edge with rho outside (0, 1]",
    -4: "continuation probability outside (0, 1]",
    -5: "prompt with fewer than two candidates",
}


class OracleError(RuntimeError):
    pass


def build(force: bool = True) -> str:
    """Compile pair_oracle.c into liboracle.so with gcc (fp64, no contraction)."""
    if force or not os.path.exists(_LIB):
        cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
               "-fPIC", "-shared", "-Wall", "-Wextra", "-o", _LIB + ".tmp", _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            lib = ctypes.CDLL(_LIB_OVERRIDE)
        else:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build()
            lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i64, i32, u64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64
        lib.orc_philox4x64_10.argtypes = [P, P, P]
        lib.orc_philox4x64_10.restype = None
        lib.orc_draw_indicator.argtypes = [u64, i64, i64, i64, ctypes.c_float]
        lib.orc_draw_indicator.restype = ctypes.c_int
        lib.orc_design_inclusion.argtypes = [i64, P, i32, P, u64, i64, i64, P, P, P, P, P]
        lib.orc_design_inclusion.restype = ctypes.c_int
        lib.orc_pair_grad.argtypes = [i64, P, i32, i64, P, ctypes.c_int, i64, P, P, P, P, P]
        lib.orc_pair_grad.restype = ctypes.c_int
        lib.orc_pair_coeffs.argtypes = [i64, P, i32, P, P, P, P, P]
        lib.orc_pair_coeffs.restype = ctypes.c_int
        lib.orc_audit.argtypes = [i64, P, i32, i64, P, ctypes.c_int, i64, P, P, P, u64, i64, i64,
                                  P, P, P, P, P]
        lib.orc_audit.restype = ctypes.c_int
        dbl = ctypes.c_double
        lib.orc_pair_grad_rule.argtypes = [i64, P, i32, i64, P, ctypes.c_int, i64, P, P, P,
                                           ctypes.c_int, dbl, P, P, P, P]
        lib.orc_pair_grad_rule.restype = ctypes.c_int
        lib.orc_pair_coeffs_rule.argtypes = [i64, P, i32, P, P, P, ctypes.c_int, dbl, P, P, P, P]
        lib.orc_pair_coeffs_rule.restype = ctypes.c_int
        lib.orc_audit_rule.argtypes = [i64, P, i32, i64, P, ctypes.c_int, i64, P, P, P,
                                       ctypes.c_int, dbl, u64, i64, i64, P, P, P, P, P, P, P]
        lib.orc_audit_rule.restype = ctypes.c_int
        lib.orc_audit_exact.argtypes = [i64, P, i32, i64, P, ctypes.c_int, i64, P, P, P,
                                        ctypes.c_int, dbl, P, P]
        lib.orc_audit_exact.restype = ctypes.c_int
        lib.orc_cps_inclusion.argtypes = [P, i64, i64, P, P]
        lib.orc_cps_inclusion.restype = ctypes.c_int
        lib.orc_cps_fit.argtypes = [P, i64, i64, dbl, i64, P, P]
        lib.orc_cps_fit.restype = ctypes.c_int
        lib.orc_cps_draw.argtypes = [i64, P, P, P, u64, i64, i64, P]
        lib.orc_cps_draw.restype = ctypes.c_int
        lib.orc_num_threads.argtypes = []
        lib.orc_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc):
    if rc != 0:
        raise OracleError(f"oracle error {rc}: {ERRORS.get(rc, '?')}")


def _scores_arg(scores):
    """Return (array, dtype code, ld).  bf16 scores are passed as their uint16 bits."""
    if scores.dtype == np.float32:
        code = F32
    elif scores.dtype == np.uint16:
        code = BF16
    else:
        raise TypeError("scores must be float32 or uint16 (bf16 bit patterns)")
    if scores.ndim != 2 or scores.strides[1] != scores.itemsize:
        raise ValueError("scores must be a row-major 2-D array")
    ld = scores.strides[0] // scores.itemsize
    return scores, code, ld


def _offsets(offsets):
    return np.ascontiguousarray(offsets, dtype=np.int64)


def num_threads() -> int:
    return _load().orc_num_threads()


def philox4x64_10(ctr, key):
    lib = _load()
    c = np.ascontiguousarray(ctr, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib.orc_philox4x64_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def draw_indicator(seed, r, b, i, p):
    return _load().orc_draw_indicator(seed, r, b, i, float(np.float32(p)))


def design_inclusion(offsets, p, seed, rep0, R, gmax, prompt_id=None, want_pi=True):
    """Returns dict(mask[R][nv] u8, pi[B][gmax][gmax] f32, edge_count[R][B], completed[R][B])."""
    lib = _load()
    off = _offsets(offsets)
    B = off.size - 1
    nv = int(off[-1])
    p = np.ascontiguousarray(p, dtype=np.float32)
    mask = np.zeros((R, nv), dtype=np.uint8)
    pi = np.zeros((B, gmax, gmax), dtype=np.float32) if want_pi else None
    ec = np.zeros((R, B), dtype=np.int32)
    comp = np.zeros((R, B), dtype=np.int32)
    pid = None if prompt_id is None else np.ascontiguousarray(prompt_id, dtype=np.int64)
    _check(lib.orc_design_inclusion(B, _ptr(off), gmax, _ptr(p), seed, rep0, R, _ptr(pid),
                                    _ptr(mask), _ptr(pi), _ptr(ec), _ptr(comp)))
    return {"mask": mask, "pi": pi, "edge_count": ec, "completed": comp}


def _gmax(off, pi, gmax):
    if pi is not None:
        return pi.shape[-1]
    if gmax is None:
        return int(np.max(np.diff(off)))
    return gmax


def pair_grad_rule(offsets, scores, rewards, mask=None, pi=None, rule=RULE_HT, wmax=0.0,
                   gmax=None):
    """Per-prompt estimate under an edge-weight rule, by explicit edges in fp64.
    Returns dict(out[B][D], edge_count[B], ess[B], max_weight[B])."""
    lib = _load()
    off = _offsets(offsets)
    B = off.size - 1
    s, code, ld = _scores_arg(scores)
    D = s.shape[1]
    r = np.ascontiguousarray(rewards, dtype=np.float32)
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    if pi is not None:
        pi = np.ascontiguousarray(pi, dtype=np.float32)
    gmax = _gmax(off, pi, gmax)
    out = np.zeros((B, D), dtype=np.float64)
    ec = np.zeros(B, dtype=np.int32)
    ess = np.zeros(B, dtype=np.float64)
    mw = np.zeros(B, dtype=np.float64)
    _check(lib.orc_pair_grad_rule(B, _ptr(off), gmax, D, _ptr(s), code, ld, _ptr(r), _ptr(m),
                                  _ptr(pi), int(rule), float(wmax), _ptr(out), _ptr(ec), _ptr(ess),
                                  _ptr(mw)))
    return {"out": out, "edge_count": ec, "ess": ess, "max_weight": mw}


def pair_coeffs_rule(offsets, rewards, mask=None, pi=None, rule=RULE_HT, wmax=0.0, gmax=None):
    """Sequence advantages under an edge-weight rule (Algorithm 1's edge order).
    Returns dict(coeff[nv], edge_count[B], ess[B], max_weight[B])."""
    lib = _load()
    off = _offsets(offsets)
    B = off.size - 1
    r = np.ascontiguousarray(rewards, dtype=np.float32)
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    if pi is not None:
        pi = np.ascontiguousarray(pi, dtype=np.float32)
    gmax = _gmax(off, pi, gmax)
    coeff = np.zeros(int(off[-1]), dtype=np.float64)
    ec = np.zeros(B, dtype=np.int32)
    ess = np.zeros(B, dtype=np.float64)
    mw = np.zeros(B, dtype=np.float64)
    _check(lib.orc_pair_coeffs_rule(B, _ptr(off), gmax, _ptr(r), _ptr(m), _ptr(pi), int(rule),
                                    float(wmax), _ptr(coeff), _ptr(ec), _ptr(ess), _ptr(mw)))
    return {"coeff": coeff, "edge_count": ec, "ess": ess, "max_weight": mw}


def pair_grad(offsets, scores, rewards, mask=None, pi=None, gmax=None):
    """Eq. (pair-ht) per prompt in fp64: returns (out[B][D] float64, edge_count[B])."""
    lib = _load()
    off = _offsets(offsets)
    B = off.size - 1
    s, code, ld = _scores_arg(scores)
    D = s.shape[1]
    r = np.ascontiguousarray(rewards, dtype=np.float32)
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    if pi is not None:
        pi = np.ascontiguousarray(pi, dtype=np.float32)
        gmax = pi.shape[-1]
    if gmax is None:
        gmax = int(np.max(np.diff(off)))
    out = np.zeros((B, D), dtype=np.float64)
    ec = np.zeros(B, dtype=np.int32)
    _check(lib.orc_pair_grad(B, _ptr(off), gmax, D, _ptr(s), code, ld, _ptr(r), _ptr(m), _ptr(pi),
                             _ptr(out), _ptr(ec)))
    return out, ec


def pair_coeffs(offsets, rewards, mask=None, pi=None, gmax=None):
    """Eq. (pair-advantage) in Algorithm 1's edge order: returns (coeff[nv] f64, edge_count[B])."""
    lib = _load()
    off = _offsets(offsets)
    B = off.size - 1
    r = np.ascontiguousarray(rewards, dtype=np.float32)
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    if pi is not None:
        pi = np.ascontiguousarray(pi, dtype=np.float32)
        gmax = pi.shape[-1]
    if gmax is None:
        gmax = int(np.max(np.diff(off)))
    coeff = np.zeros(int(off[-1]), dtype=np.float64)
    ec = np.zeros(B, dtype=np.int32)
    _check(lib.orc_pair_coeffs(B, _ptr(off), gmax, _ptr(r), _ptr(m), _ptr(pi), _ptr(coeff), _ptr(ec)))
    return coeff, ec


def audit(offsets, scores, rewards, p, seed, rep0, R, pi_w=None, gmax=None, prompt_id=None,
          want_reps=True, rule=RULE_HT, wmax=0.0):
    """Frozen-population audit of the estimator under `rule`: returns
    dict(mse[B], bias_norm[B], rep_sqerr[B][R], edge_count[B][R], cosine[B],
    target_norm[B]); cosine is the mean over replicates of the cosine between
    each estimate and the target (0 for a zero estimate or target)."""
    lib = _load()
    off = _offsets(offsets)
    B = off.size - 1
    s, code, ld = _scores_arg(scores)
    D = s.shape[1]
    r = np.ascontiguousarray(rewards, dtype=np.float32)
    pp = np.ascontiguousarray(p, dtype=np.float32)
    if pi_w is not None:
        pi_w = np.ascontiguousarray(pi_w, dtype=np.float32)
        gmax = pi_w.shape[-1]
    if gmax is None:
        gmax = int(np.max(np.diff(off)))
    pid = None if prompt_id is None else np.ascontiguousarray(prompt_id, dtype=np.int64)
    mse = np.zeros(B, dtype=np.float64)
    bias = np.zeros(B, dtype=np.float64)
    cos = np.zeros(B, dtype=np.float64)
    tn = np.zeros(B, dtype=np.float64)
    reps = np.zeros((B, R), dtype=np.float64) if want_reps else None
    ec = np.zeros((B, R), dtype=np.int32) if want_reps else None
    _check(lib.orc_audit_rule(B, _ptr(off), gmax, D, _ptr(s), code, ld, _ptr(r), _ptr(pp),
                              _ptr(pi_w), int(rule), float(wmax), seed, rep0, R, _ptr(pid),
                              _ptr(mse), _ptr(bias), _ptr(reps), _ptr(ec), _ptr(cos), _ptr(tn)))
    return {"mse": mse, "bias_norm": bias, "rep_sqerr": reps, "edge_count": ec, "cosine": cos,
            "target_norm": tn}


def audit_exact(offsets, scores, rewards, p, pi_w=None, gmax=None, rule=RULE_HT, wmax=0.0):
    """Exact design MSE and bias norm per prompt (Prop. 1), no draws, for the
    linear rules (HT, unweighted, clipped, marginal-only).  Returns
    dict(mse[B], bias_norm[B])."""
    lib = _load()
    off = _offsets(offsets)
    B = off.size - 1
    s, code, ld = _scores_arg(scores)
    D = s.shape[1]
    r = np.ascontiguousarray(rewards, dtype=np.float32)
    pp = np.ascontiguousarray(p, dtype=np.float32)
    if pi_w is not None:
        pi_w = np.ascontiguousarray(pi_w, dtype=np.float32)
    gmax = _gmax(off, pi_w, gmax)
    mse = np.zeros(B, dtype=np.float64)
    bias = np.zeros(B, dtype=np.float64)
    _check(lib.orc_audit_exact(B, _ptr(off), gmax, D, _ptr(s), code, ld, _ptr(r), _ptr(pp),
                               _ptr(pi_w), int(rule), float(wmax), _ptr(mse), _ptr(bias)))
    return {"mse": mse, "bias_norm": bias}


def cps_inclusion(w, n):
    """Conditional Poisson design of one prompt with odds w and size n:
    returns (pi[g], pij[g][g]) in fp64 (pij's diagonal = pi)."""
    lib = _load()
    w = np.ascontiguousarray(w, dtype=np.float64)
    g = w.size
    pi = np.zeros(g)
    pij = np.zeros((g, g))
    _check(lib.orc_cps_inclusion(_ptr(w), g, int(n), _ptr(pi), _ptr(pij)))
    return pi, pij


def cps_fit(pi_target, n, tol=1e-12, max_iter=10000):
    """Odds whose conditional Poisson design has first-order probabilities
    pi_target (summing to n).  Returns (w, iterations; negative if not
    converged)."""
    lib = _load()
    t = np.ascontiguousarray(pi_target, dtype=np.float64)
    w = np.zeros(t.size)
    it = np.zeros(1, dtype=np.int64)
    _check(lib.orc_cps_fit(_ptr(t), t.size, int(n), float(tol), int(max_iter), _ptr(w), _ptr(it)))
    return w, int(it[0])


def cps_draw(offsets, w, n, seed, rep0, R):
    """Fixed-size draws mask[R][nv] for every prompt (prompt ids 0..B-1)."""
    lib = _load()
    off = _offsets(offsets)
    B = off.size - 1
    w = np.ascontiguousarray(w, dtype=np.float64)
    nn = np.ascontiguousarray(n, dtype=np.int32)
    mask = np.zeros((R, int(off[-1])), dtype=np.uint8)
    _check(lib.orc_cps_draw(B, _ptr(off), _ptr(w), _ptr(nn), seed, rep0, R, _ptr(mask)))
    return mask
