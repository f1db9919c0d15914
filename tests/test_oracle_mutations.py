"""Planted mistakes in the CPU oracle must fail its pins.

Each case copies ``oracle/pair_oracle.c``, replaces one fragment with a
plausible mistake, compiles the copy with the oracle's own flags, and runs the
oracle pin tests against it in a fresh process (``PAIR_ORACLE_LIB`` points the
oracle package at the copy).  The run must fail: a pin that lets the mistake
through would let the same mistake through in the oracle itself.  The
unmodified copy must pass, so the harness itself is checked too.

The same is done for the probability-design oracle, ``oracle/alloc.py``: a
mutated copy is loaded in place of ``oracle.alloc`` in a fresh process and its
pins are run.

The mistakes cover every part of the oracle: the edge term, the weights, the
normaliser, the rho entry and the edge mask of the estimator (Eq. pair-ht);
the half-edge split of the sequence advantages (Eq. pair-advantage); the
Philox reading of the design draw (word, counter layout, key schedule), the
induced-edge count and the logged rho block; bf16 widening; the audit's
target, MSE, bias and update-direction cosine (App. D, Sec. 6.2); the exact covariance trace of Prop. 1; the
conditional-Poisson inclusion probabilities; and the contrast graph's
disagreement, edge proxy and vertex term, the design objective, its gradient
and budget, and the pointwise and uniform comparison designs (Sec. 4.3-4.4).
"""
import concurrent.futures
import os
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "pair_oracle.c")
PINS = ["tests/test_oracle_pins.py", "tests/test_oracle_rules.py", "tests/test_oracle_exact.py",
        "tests/test_oracle_cps.py"]
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC",
          "-shared", "-w"]

# (label, fragment of pair_oracle.c, replacement); the first occurrence is replaced.
MUTATIONS = [
    ("edge term without the 1/2",
     "out[d] += 0.5 * (ri - rj) * (wi * si - wj * sj);",
     "out[d] += (ri - rj) * (wi * si - wj * sj);"),
    ("rho multiplied instead of divided",
     "double w = 1.0 / rho;",
     "double w = rho;"),
    ("HT normaliser K_E instead of M",
     "double N = M;\n    if (rule == ORC_RULE_RATIO_KE) N = (double)ke;\n    if (rule == ORC_RULE_SELFNORM) N = nsn;\n    for (int64_t d",
     "double N = (double)ke;\n    if (rule == ORC_RULE_RATIO_KE) N = (double)ke;\n    if (rule == ORC_RULE_SELFNORM) N = nsn;\n    for (int64_t d"),
    ("reward difference reversed",
     "double ri = (double)rewards[o + i], rj = (double)rewards[o + j];",
     "double ri = (double)rewards[o + j], rj = (double)rewards[o + i];"),
    ("rho read from the diagonal",
     "return (double)blk[lo * gmax + hi];",
     "return (double)blk[lo * gmax + lo];"),
    ("unobserved partner included",
     "if (!(Ji && Jj)) continue; /* I_ij = 0: the edge is not observed */",
     "if (!(Ji || Jj)) continue;"),
    ("advantage: wrong sign on the second endpoint",
     "coeff[o + j] -= 0.5 * dr * wj;",
     "coeff[o + j] += 0.5 * dr * wj;"),
    ("advantage: first endpoint without the 1/2",
     "coeff[o + i] += 0.5 * dr * wi;",
     "coeff[o + i] += dr * wi;"),
    ("Philox: wrong output word",
     "uint64_t u = w[i & 3] >> 32;",
     "uint64_t u = w[(i + 1) & 3] >> 32;"),
    ("Philox: replicate and prompt swapped in the counter",
     "uint64_t ctr[4] = {(uint64_t)r, (uint64_t)b, (uint64_t)(i >> 2), 0};",
     "uint64_t ctr[4] = {(uint64_t)b, (uint64_t)r, (uint64_t)(i >> 2), 0};"),
    ("Philox: wrong Weyl constant",
     "weyl1 = 0xBB67AE8584CAA73BULL",
     "weyl1 = 0xBB67AE8584CAA73DULL"),
    ("Philox: low half of the word",
     "uint64_t u = w[i & 3] >> 32;",
     "uint64_t u = w[i & 3] & 0xffffffffULL;"),
    ("induced-edge count includes self pairs",
     "/* brute-force count of induced edges */\n                for (int64_t j = i + 1; j < g; ++j)",
     "/* brute-force count of induced edges */\n                for (int64_t j = i; j < g; ++j)"),
    ("audit cosine against the estimate's own norm",
     "if (gg > 0.0 && tt > 0.0) csum += gt / (sqrt(gg) * sqrt(tt));",
     "if (gg > 0.0 && tt > 0.0) csum += gt / (sqrt(gg) * sqrt(gg));"),
    ("audit cosine: a zero estimate counted as aligned",
     "if (gg > 0.0 && tt > 0.0) csum += gt / (sqrt(gg) * sqrt(tt));",
     "csum += (gg > 0.0 && tt > 0.0) ? gt / (sqrt(gg) * sqrt(tt)) : 1.0;"),
    ("logged rho uses p_i twice",
     "val = (float)((double)p[o + i] * (double)p[o + j]);",
     "val = (float)((double)p[o + i] * (double)p[o + i]);"),
    ("bf16 widened with the wrong shift",
     "uint32_t bits = ((uint32_t)h) << 16;",
     "uint32_t bits = ((uint32_t)h) << 15;"),
    ("audit target weighted by 1/rho",
     "s = ht_estimate_one(o, g, D, scores, dtype, ld, rewards, NULL, NULL, gmax, t, NULL);",
     "s = ht_estimate_one(o, g, D, scores, dtype, ld, rewards, NULL, blk, gmax, t, NULL);"),
    ("audit MSE over R - 1",
     "if (mse) mse[b] = esum / (double)R;",
     "if (mse) mse[b] = esum / (double)(R > 1 ? R - 1 : 1);"),
    ("audit bias from the last replicate",
     "double dev = gsum[d] / (double)R - t[d];",
     "double dev = gr[d] - t[d];"),
    ("exact audit: shared-vertex covariance dropped",
     "tr += pi_ * pj * pk * (1.0 - pi_) * ip;",
     "tr += 0.0 * ip;"),
    ("exact audit: edge variance rho^2 instead of rho (1 - rho)",
     "tr += rho * (1.0 - rho) * nn;",
     "tr += rho * rho * nn;"),
    ("conditional Poisson: joint probability without w_j",
     "v = w[i] * w[j] * e[n - 2] / en;",
     "v = w[i] * e[n - 2] / en;"),
    ("conditional Poisson: first order without leaving unit i out",
     "esp_excluding(w, g, n - 1, i, -1, e);",
     "esp_excluding(w, g, n - 1, -1, -1, e);"),
]


def _build(src_text, folder, name):
    c = os.path.join(folder, name + ".c")
    so = os.path.join(folder, name + ".so")
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", *CFLAGS, "-o", so, c, "-lm"], check=True, capture_output=True)
    return so


def _run_pins(so):
    env = dict(os.environ, PAIR_ORACLE_LIB=so, OMP_NUM_THREADS="2")
    res = subprocess.run([sys.executable, "-m", "pytest", *PINS, "-x", "-q", "-p", "no:cacheprovider",
                          "-m", "not gpu", "-p", "no:xdist"],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return res.returncode, res.stdout[-2000:]


def test_every_planted_mistake_fails_a_pin():
    with open(SRC) as f:
        src = f.read()
    for label, old, new in MUTATIONS:
        assert old in src, f"mutation site not found: {label}"
    with tempfile.TemporaryDirectory() as tmp:
        libs = {"unmodified": _build(src, tmp, "unmodified")}
        for k, (label, old, new) in enumerate(MUTATIONS):
            libs[label] = _build(src.replace(old, new, 1), tmp, f"mutant{k}")
        with concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
            results = dict(zip(libs, ex.map(_run_pins, libs.values())))
    rc, out = results.pop("unmodified")
    assert rc == 0, "the unmodified copy must pass every pin:\n" + out
    survivors = [label for label, (rc, _) in results.items() if rc == 0]
    assert not survivors, f"planted mistakes no pin catches: {survivors}"
    # every mutant failed a test (exit 1), not the harness (collection or usage error)
    broken = {label: out for label, (rc, out) in results.items() if rc != 1}
    assert not broken, f"mutant runs that did not end in a failing test: {list(broken)}"


ALLOC_SRC = os.path.join(ROOT, "oracle", "alloc.py")
ALLOC_PINS = ["tests/test_oracle_alloc.py"]
ALLOC_MUTATIONS = [
    ("disagreement without the (1 - p_i) p_j term",
     "d = p[:, None] * (1.0 - p[None, :]) + (1.0 - p[:, None]) * p[None, :]",
     "d = p[:, None] * (1.0 - p[None, :]) + p[:, None] * p[None, :]"),
    ("edge proxy over 2 instead of 4",
     "a = a * (m[:, None] + m[None, :]) ** 2 / 4.0",
     "a = a * (m[:, None] + m[None, :]) ** 2 / 2.0"),
    ("vertex term without the diagonal correction",
     "return np.sum(np.sqrt(a), axis=1) ** 2 - np.sum(a, axis=1)",
     "return np.sum(np.sqrt(a), axis=1) ** 2"),
    ("objective multiplies the vertex term by pi",
     "return float(np.sum(a[iu] / (pi[iu[0]] * pi[iu[1]])) + np.sum(b / pi))",
     "return float(np.sum(a[iu] / (pi[iu[0]] * pi[iu[1]])) + np.sum(b * pi))"),
    ("solver gradient with the wrong sign",
     "return -(iu * iu) * (sym @ iu + b) / f0",
     "return (iu * iu) * (sym @ iu + b) / f0"),
    ("budget row doubled",
     'cons = {"type": "ineq", "fun": lambda u: 1.0 - float(cs @ u), "jac": lambda u: -cs}',
     'cons = {"type": "ineq", "fun": lambda u: 2.0 - float(cs @ u), "jac": lambda u: -cs}'),
    ("uniform design spends half the budget",
     "pi = np.full(p.size, np.clip(budget / np.sum(c), pi_min, 1.0))",
     "pi = np.full(p.size, np.clip(0.5 * budget / np.sum(c), pi_min, 1.0))"),
    ("pointwise design with p instead of p (1 - p)",
     "pi, ok = _solve(np.zeros_like(a), p * (1.0 - p), c, budget, pi_min)",
     "pi, ok = _solve(np.zeros_like(a), p, c, budget, pi_min)"),
]

# Runs the allocation pins with a copy of alloc.py loaded as oracle.alloc.
_ALLOC_BOOT = """
import importlib.util, sys
import pytest
import oracle
spec = importlib.util.spec_from_file_location("oracle.alloc", sys.argv[1])
mod = importlib.util.module_from_spec(spec)
spec.loader.exec_module(mod)
sys.modules["oracle.alloc"] = mod
oracle.alloc = mod
sys.exit(pytest.main(sys.argv[2:]))
"""


def _run_alloc_pins(path):
    env = dict(os.environ, OMP_NUM_THREADS="2")
    res = subprocess.run([sys.executable, "-c", _ALLOC_BOOT, path, *ALLOC_PINS, "-x", "-q",
                          "-p", "no:cacheprovider", "-m", "not gpu", "-p", "no:xdist"],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return res.returncode, res.stdout[-2000:]


def test_every_planted_allocation_mistake_fails_a_pin():
    with open(ALLOC_SRC) as f:
        src = f.read()
    for label, old, new in ALLOC_MUTATIONS:
        assert old in src, f"mutation site not found: {label}"
    with tempfile.TemporaryDirectory() as tmp:
        paths = {}
        for k, (label, old, new) in enumerate([("unmodified", "", "")] + ALLOC_MUTATIONS):
            path = os.path.join(tmp, f"alloc_{k}.py")
            with open(path, "w") as f:
                f.write(src.replace(old, new, 1) if old else src)
            paths[label] = path
        with concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
            results = dict(zip(paths, ex.map(_run_alloc_pins, paths.values())))
    rc, out = results.pop("unmodified")
    assert rc == 0, "the unmodified copy must pass every pin:\n" + out
    survivors = [label for label, (rc, _) in results.items() if rc == 0]
    assert not survivors, f"planted mistakes no pin catches: {survivors}"
    broken = {label: out for label, (rc, out) in results.items() if rc != 1}
    assert not broken, f"mutant runs that did not end in a failing test: {list(broken)}"
