#!/usr/bin/env python3
"""Benchmark of the PAIR hot path on one MI355X.

One step = one pass of every stage of the hot path over resident synthetic
inputs:
  gradient chain on workload b128 (B=128 prompts, G=16, D=2^20 bf16 scores):
      pair_design_coeffs (the design draw and the coefficient fold in one
      launch, writing the mask and the logged rho block too) ->
      pair_weighted_grad
  estimator audit on workload audit (B=256, G=16, D=65536 bf16, R=4096):
      pair_audit (replicate coefficients, matrix-core contraction with the
      squared-norm epilogue, fp64 reductions)

Prints ONE JSON line.  `value` is the gradient chain's throughput in GB/s of
algorithmic bytes (score rows with a nonzero coefficient, the coefficients,
and the fp32 output), i.e. bytes that must cross HBM, over the chain's event
time.  The audit is reported in replicate-estimates/s and TFLOP/s (2*G*D flop
per replicate estimate of the prompts it sweeps) in the "audit" object.
"roofline" is the weighted-gradient kernel on the worst of the three gradient
workloads (b128, the Qwen3-shaped slice, ragged), each timed with HIP events on
the stream it is launched on; "roofline_by_config" lists all of them, per
prompt and in batch-mean mode.

Usage: python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--no-cpu-baseline]
       python bench.py --copy-calibration     (1 GiB copy for counter scaling)
       python bench.py --audit-calls N        (N audit calls only, for counter passes)
       python bench.py --counter-pass         (the calls the traffic counter runs profile)
       python bench.py --record-traffic DIR   (counter runs -> profiles/counters.json)
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("weighted-grad score GB/s (% HBM peak); "
          "audit replicate-estimates/s (% MFMA peak)")
HBM_PEAK_GBPS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
COUNTERS = os.path.join(ROOT, "profiles", "counters.json")


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


_C_TOKENS = re.compile(r'//[^\n]*|/\*.*?\*/|"(?:\\.|[^"\\\n])*"|\'(?:\\.|[^\'\\\n])*\'', re.S)


def _code_only(text):
    """C++ source with comments removed and whitespace runs collapsed, so that
    editing a comment does not count as a change of the kernel."""
    text = _C_TOKENS.sub(lambda m: m.group(0) if m.group(0)[0] in "\"'" else " ", text)
    return " ".join(text.split())


def _source_sha(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2608_11368_amd", "csrc", n), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def _traffic(kernel, sources):
    """HBM bytes per launch from committed rocprofv3 counter runs, or None when
    the kernel's source changed since the counters were taken."""
    try:
        with open(COUNTERS) as f:
            rec = json.load(f).get(kernel)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_sha") != _source_sha(*sources):
        return None
    return rec.get("hbm_bytes_per_launch")


# Kernels whose HBM traffic is recorded from rocprofv3 counter runs of
# `bench.py --counter-pass`, which makes COUNTER_PASS_CALLS calls of each entry
# point below in this order: per-prompt and batch-mean weighted gradient on
# each workload of GRAD_WORKLOADS, then the audit.  Key -> (kernel-name prefix
# of every dispatch of one call, the dispatch counted once per call, index of
# the call group of that name in pass order, sources the record is tied to).
GRAD_WORKLOADS = ("b128", "qwen3", "ragged")
COUNTER_PASS_CALLS = 2
TRAFFIC_KERNELS = {}
for _k, _name in enumerate(GRAD_WORKLOADS):
    TRAFFIC_KERNELS[f"wgrad_{_name}"] = ("wgrad_kernel", "wgrad_kernel", _k,
                                         ["wgrad.hip", "common.hpp"])
    TRAFFIC_KERNELS[f"wgrad_mean_{_name}"] = ("wgrad_mean_kernel", "wgrad_mean_kernel", _k,
                                              ["wgrad.hip", "common.hpp"])
TRAFFIC_KERNELS["audit_b256"] = ("audit_", "audit_final_kernel", 0, ["audit.hip", "common.hpp"])


def _counter_rows(path):
    import csv
    with open(path, newline="") as f:
        return [(r["Kernel_Name"], float(r["Counter_Value"])) for r in csv.DictReader(f)]


def _kernel_kib(rows, prefix, per_call, group, calls):
    """KiB per entry-point call for call group `group` of the counter pass:
    the dispatches whose demangled name starts with `prefix` (namespaces
    dropped) from the one after the (group * calls)-th dispatch named
    `per_call` up to and including the ((group + 1) * calls)-th, over
    `calls`."""
    def base(name):
        name = name.replace("(anonymous namespace)::", "")
        name = name[5:] if name.startswith("void ") else name
        return name.split("(")[0].split("<")[0].split("::")[-1].strip()
    tot, seen = 0.0, 0
    lo, hi = group * calls, (group + 1) * calls
    for n, v in rows:
        b = base(n)
        if b.startswith(prefix) and lo <= seen < hi:
            tot += v
        if b == per_call:
            seen += 1
            if seen == hi:
                return tot / calls
    raise SystemExit(f"fewer than {hi} {per_call} dispatches in the counter file")


def record_traffic(folder):
    """Write HBM bytes per launch into the committed counter record from four
    rocprofv3 --pmc runs under `folder`: tr_FETCH_SIZE/, tr_WRITE_SIZE/ (this
    script with --counter-pass) and trc_FETCH_SIZE/, trc_WRITE_SIZE/ (this
    script with --copy-calibration).  Each counter is
    scaled by the factor that maps it to the known bytes of the calibration
    copy (1 GiB read, 1 GiB written)."""
    def rows(sub):
        return _counter_rows(os.path.join(folder, sub, "run_counter_collection.csv"))

    gib = float(1 << 30)
    factors = {}
    for ctr in ("FETCH_SIZE", "WRITE_SIZE"):
        copies = [v for n, v in rows("trc_" + ctr) if "copyBuffer" in n]
        big = sorted(v for v in copies if v > 0.5 * max(copies))
        factors[ctr] = (gib, big[len(big) // 2])
    fetch_f = factors["FETCH_SIZE"][0] / (factors["FETCH_SIZE"][1] * 1024.0)
    write_f = factors["WRITE_SIZE"][0] / (factors["WRITE_SIZE"][1] * 1024.0)
    try:
        with open(COUNTERS) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        rec = {}
    fetch_rows, write_rows = rows("tr_FETCH_SIZE"), rows("tr_WRITE_SIZE")
    cmd = "rocprofv3 --pmc {c} -f csv -d <out> -o run -- python -u <repo>/bench.py {a}"
    calls = COUNTER_PASS_CALLS
    for key, (prefix, per_call, group, sources) in TRAFFIC_KERNELS.items():
        fk = _kernel_kib(fetch_rows, prefix, per_call, group, calls)
        wk = _kernel_kib(write_rows, prefix, per_call, group, calls)
        rd, wr = fk * 1024.0 * fetch_f, wk * 1024.0 * write_f
        rec[key] = {
            "kernels": prefix + "*",
            "source_sha": _source_sha(*sources),
            "fetch_size_kib_per_launch": round(fk, 1),
            "write_size_kib_per_launch": round(wk, 1),
            "calibration": {
                "fetch_factor": round(fetch_f, 4), "write_factor": round(write_f, 4),
                "basis": "plain 1 GiB device copy: FETCH_SIZE %.0f KiB, WRITE_SIZE %.0f KiB"
                         % (factors["FETCH_SIZE"][1], factors["WRITE_SIZE"][1])},
            "hbm_read_bytes_per_launch": int(rd),
            "hbm_write_bytes_per_launch": int(wr),
            "hbm_bytes_per_launch": int(rd + wr),
            "calls_counted": calls,
            "commands": [cmd.format(c=c, a=a) for a in ("--counter-pass", "--copy-calibration")
                         for c in ("FETCH_SIZE", "WRITE_SIZE")],
        }
    with open(COUNTERS, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps({k: rec[k]["hbm_bytes_per_launch"] for k in TRAFFIC_KERNELS}))


def cpu_baseline(meta, w, scores_dev, meta_a, wa, scores_a_dev, budget_s=24.0):
    """The CPU oracle as it stands, timed on the host cores on bounded samples:
    the gradient chain on a column slice of the b128 scores (all prompts;
    the whole workload when that is shorter than half the budget), and the
    audit on the first prompts of the audit workload, growing the replicate
    window to all R replicates and then the number of prompts until about
    half the budget is spent.  Returns a dict."""
    import numpy as np

    import oracle
    from tests.gpu_util import scores_to_host

    cores = oracle.num_threads()
    # gradient: grow the column slice until the run is long enough
    cols = 2048
    while True:
        s_host = scores_to_host(scores_dev[:, :cols])
        t0 = time.perf_counter()
        d = oracle.design_inclusion(meta.offsets, meta.p, w.design_seed, 0, 1, meta.gmax)
        est, _ = oracle.pair_grad(meta.offsets, s_host, meta.rewards, d["mask"][0], d["pi"])
        dt = time.perf_counter() - t0
        coeff, _ = oracle.pair_coeffs(meta.offsets, meta.rewards, d["mask"][0], d["pi"])
        if dt >= budget_s / 2 or cols >= w.D:
            break
        cols = min(w.D, cols * max(2, int(budget_s / 2 / max(dt, 1e-3))))
    nz_rows = int(np.count_nonzero(coeff))
    grad_bytes = nz_rows * cols * 2 + meta.nv * 4 + meta.B * cols * 4
    # audit: the first `nprom` prompts, `reps` replicates each
    reps, nprom = 8, 1
    while True:
        o0, o1 = meta_a.offsets[0], meta_a.offsets[nprom]
        sa = scores_to_host(scores_a_dev[o0:o1])
        t0 = time.perf_counter()
        oracle.audit(meta_a.offsets[:nprom + 1] - o0, sa, meta_a.rewards[o0:o1], meta_a.p[o0:o1],
                     wa.design_seed, 0, reps, prompt_id=list(range(nprom)), want_reps=False)
        da = time.perf_counter() - t0
        if da >= budget_s / 2 or (reps >= wa.R and nprom >= meta_a.B):
            break
        grow = max(2, int(budget_s / 2 / max(da, 1e-3)))
        if reps < wa.R:
            reps = min(wa.R, reps * grow)
        else:
            nprom = min(meta_a.B, nprom * grow)
    return {
        "value": grad_bytes / dt / 1e9,
        "unit": "GB/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"gradient chain (design draw + explicit-edge fp64 estimator) on all "
                   f"{meta.B} prompts x first {cols} of {w.D} columns: {dt:.2f} s; "
                   f"audit on prompts 0..{nprom - 1}, {reps} replicates each x D={wa.D}: "
                   f"{da:.2f} s"),
        "audit_value": nprom * reps / da,
        "audit_unit": "replicate-estimates/s",
        "seconds": dt + da,
        "cpu_model": _cpu_model(),
    }


def _grow(fn, target_s, n0, n_max):
    """Run fn(n) with n doubling (or more) until it takes target_s or n reaches
    n_max; returns (n, seconds) of the last run."""
    n = n0
    while True:
        t0 = time.perf_counter()
        fn(n)
        dt = time.perf_counter() - t0
        if dt >= target_s or n >= n_max:
            return n, dt
        n = min(n_max, n * max(2, int(target_s / max(dt, 1e-3))))


def cpu_next_rows(wl, meta_a, wa, scores_a_dev, target_s=2.0):
    """The CPU oracle on bounded samples of the widened rows' workloads: the
    estimator variants (audit replay per edge-weight rule), the exact audit,
    the probability design and the fixed-size design fit.  Returns one dict
    per row, to sit beside that row's GPU timing."""
    import numpy as np

    import oracle
    from oracle import alloc as oalloc
    from tests.gpu_util import scores_to_host

    cores = oracle.num_threads()
    o0, o1 = meta_a.offsets[0], meta_a.offsets[1]
    sa0 = scores_to_host(scores_a_dev[o0:o1])
    out = {}

    def variants(reps):
        for rule in range(len(RULE_NAMES)):
            oracle.audit(np.array([0, o1 - o0]), sa0, meta_a.rewards[o0:o1], meta_a.p[o0:o1],
                         wa.design_seed, 0, reps, prompt_id=[0], want_reps=False, rule=rule,
                         wmax=10.0 if RULE_NAMES[rule] == "clipped" else 0.0)
    n, dt = _grow(variants, target_s, 4, wa.R)
    out["variants"] = {"value": round(n * len(RULE_NAMES) / dt, 1), "unit": "replicate-estimates/s",
                       "cores": cores, "kind": "oracle",
                       "sample": f"audit workload prompt 0, {n} replicates under each of the "
                                 f"{len(RULE_NAMES)} rules: {dt:.2f} s"}

    def exact(k):
        lo, hi = meta_a.offsets[0], meta_a.offsets[k]
        oracle.audit_exact(meta_a.offsets[:k + 1] - lo, scores_to_host(scores_a_dev[lo:hi]),
                           meta_a.rewards[lo:hi], meta_a.p[lo:hi], gmax=meta_a.gmax)
    n, dt = _grow(exact, target_s, 1, meta_a.B)
    out["exact_audit"] = {"value": round(n / dt, 1), "unit": "prompts/s", "cores": cores,
                          "kind": "oracle",
                          "sample": f"first {n} prompts of the audit workload: {dt:.2f} s"}

    wr = wl.WORKLOADS["ragged"]
    mr = wl.host_meta(wr)
    inp = wl.alloc_inputs(wr, mr.offsets)

    def design(k):
        oalloc.solve_batch(mr.offsets[:k + 1], inp.p_hat, inp.c_hat, inp.budget[:k], 0.08,
                           oalloc.PAIR)
    n, dt = _grow(design, target_s, 1, mr.B)
    out["design_alloc"] = {"value": round(n / dt, 1), "unit": "prompts/s", "cores": 1,
                           "kind": "oracle",
                           "sample": f"first {n} prompts of the ragged structure, graph-coupled "
                                     f"design (SLSQP, one thread): {dt:.2f} s"}

    tg = wl.cps_targets(mr.offsets)

    def cps(k):
        for b in range(k):
            lo, hi = mr.offsets[b], mr.offsets[b + 1]
            t = tg[lo:hi].astype(np.float64)
            oracle.cps_fit(t, int(round(float(t.sum()))))
    n, dt = _grow(cps, target_s, 1, mr.B)
    out["fixed_size_design"] = {"value": round(n / dt, 1), "unit": "prompts/s", "cores": 1,
                                "kind": "oracle",
                                "sample": f"fit of the first {n} prompts of the ragged structure "
                                          f"(one thread): {dt:.2f} s"}
    return out


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


RULE_NAMES = ("ht", "unweighted", "ratio_ke", "clipped", "selfnorm", "marginal")


class TimingEvent:
    """A HIP event used only to measure time on a stream.  It is created with
    hipEventDisableSystemFence: recording it then does not write back and
    invalidate the caches, which with default events adds several
    microseconds to the work around each event and perturbs the kernel that
    follows.  Elapsed times are read only after a device synchronisation."""

    _hip = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    @classmethod
    def _lib(cls):
        if cls._hip is None:
            # The HIP runtime torch has already loaded (the one libpair uses too).
            hip = ctypes.CDLL("libamdhip64.so.7", mode=os.RTLD_NOLOAD | os.RTLD_GLOBAL)
            hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
            hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                ctypes.c_void_p]
            hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
            cls._hip = hip
        return cls._hip

    def __init__(self):
        self.h = ctypes.c_void_p()
        rc = self._lib().hipEventCreateWithFlags(ctypes.byref(self.h), self.DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")

    def record(self, stream):
        rc = self._lib().hipEventRecord(self.h, ctypes.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def synchronize(self):
        rc = self._lib().hipEventSynchronize(self.h)
        if rc != 0:
            raise RuntimeError(f"hipEventSynchronize failed ({rc})")

    def elapsed_time(self, end) -> float:
        ms = ctypes.c_float()
        rc = self._lib().hipEventElapsedTime(ctypes.byref(ms), self.h, end.h)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(ms.value)

    def __del__(self):
        # At interpreter exit the HIP runtime may already be torn down; the
        # process ends anyway, so the event is left to it.
        if sys.is_finalizing() or self._hip is None or not self.h:
            return
        try:
            self._hip.hipEventDestroy(self.h)
        except Exception:
            pass


def _event_ms(stream, fn, reps):
    import torch

    fn()
    e0 = TimingEvent()
    e1 = TimingEvent()
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    e1.synchronize()
    return e0.elapsed_time(e1) / reps


def time_wgrad_configs(pair, stream, wl, dev, coeff, out, scores, off, rew, p, mask, pi, ec, comp,
                       status, B, nv, G, D, w):
    """The weighted-gradient stream beyond the headline workload: the b128
    batch-mean reduce mode (score bytes are nearly all its traffic), and the
    per-prompt and batch-mean modes on the Qwen3-shaped slice (B=64, G=8,
    D=2^26, 68.7 GB of bf16 scores) and on the ragged workload (B=512,
    G_b ~ U{2..64}, D=2^18).
    GB/s of algorithmic bytes (nonzero score rows, coefficients, offsets,
    output), kernel timed alone with events on the launch stream."""
    import torch

    res = {}
    with torch.cuda.stream(stream):
        mean = torch.empty(D, dtype=torch.float32, device=dev)
        nz = int(torch.count_nonzero(coeff).item())
        ms = _event_ms(stream, lambda: pair.pair_weighted_grad(B, nv, off, scores, coeff, mean, 1,
                                                                status, stream), 10)
        alg = nz * D * 2 + nv * 4 + (B + 1) * 8 + D * 4
        res["b128_batch_mean"] = {"ms": round(ms, 4), "GBps": round(alg / ms / 1e6, 1),
                                  "frac": round(alg / ms / 1e6 / HBM_PEAK_GBPS, 4),
                                  "algorithmic_bytes": alg}
    del mean
    for name in ("qwen3", "ragged"):
        wk = wl.WORKLOADS[name]
        meta = wl.host_meta(wk)
        _log(f"[bench] generating {name} scores {meta.nv}x{wk.D} bf16")
        s_k = wl.device_scores(wk, meta.nv, dev)
        o_k = torch.from_numpy(meta.offsets).to(dev)
        r_k = torch.from_numpy(meta.rewards).to(dev)
        p_k = torch.from_numpy(meta.p).to(dev)
        c_k = torch.empty(meta.nv, dtype=torch.float32, device=dev)
        out_k = torch.empty((meta.B, wk.D), dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            pair.pair_design_coeffs(meta.B, meta.nv, meta.gmax, o_k, p_k, r_k, wk.design_seed, 0,
                                    c_k, None, None, None, None, status, stream)
            reps = 3 if wk.D > (1 << 24) else 10
            ms = _event_ms(stream, lambda: pair.pair_weighted_grad(
                meta.B, meta.nv, o_k, s_k, c_k, out_k, 0, status, stream), reps)
            del out_k
            mean_k = torch.empty(wk.D, dtype=torch.float32, device=dev)
            ms_mean = _event_ms(stream, lambda: pair.pair_weighted_grad(
                meta.B, meta.nv, o_k, s_k, c_k, mean_k, 1, status, stream), reps)
        nz = int(torch.count_nonzero(c_k).item())
        alg = nz * wk.D * 2 + meta.nv * 4 + (meta.B + 1) * 8 + meta.B * wk.D * 4
        res[name] = {"B": meta.B, "nv": meta.nv, "D": wk.D, "rows_nonzero": nz,
                     "ms": round(ms, 4), "GBps": round(alg / ms / 1e6, 1),
                     "score_only_GBps": round(nz * wk.D * 2 / ms / 1e6, 1),
                     "frac": round(alg / ms / 1e6 / HBM_PEAK_GBPS, 4), "algorithmic_bytes": alg}
        alg_mean = nz * wk.D * 2 + meta.nv * 4 + (meta.B + 1) * 8 + wk.D * 4
        res[name + "_batch_mean"] = {"ms": round(ms_mean, 4),
                                     "GBps": round(alg_mean / ms_mean / 1e6, 1),
                                     "frac": round(alg_mean / ms_mean / 1e6 / HBM_PEAK_GBPS, 4),
                                     "algorithmic_bytes": alg_mean}
        del s_k, mean_k
        torch.cuda.empty_cache()
    if int(status.item()) != 0:
        raise RuntimeError(f"device status {int(status.item())} in the gradient configurations")
    return res


def time_alloc(pair, stream, wl, dev, reps=5):
    """Probability design (Sec. 4.4) on the ragged workload's prompt structure
    (B = 512, G_b ~ U{2..64}) with synthetic prefix statistics; each design
    timed with events on the launch stream."""
    import torch

    w = wl.WORKLOADS["ragged"]
    meta = wl.host_meta(w)
    inp = wl.alloc_inputs(w, meta.offsets)
    t = lambda a: torch.from_numpy(a).to(dev)
    off, ph, ch, bu = t(meta.offsets), t(inp.p_hat), t(inp.c_hat), t(inp.budget)
    B, nv = meta.B, meta.nv
    pi = torch.empty(nv, dtype=torch.float32, device=dev)
    obj = torch.empty(B, dtype=torch.float64, device=dev)
    its = torch.empty(B, dtype=torch.int32, device=dev)
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    out = {"workload": f"B={B}, G_b~U{{2..64}}, nv={nv}, budget 0.5 sum c, pi_min 0.08"}
    with torch.cuda.stream(stream):
        for name, design in (("pair", 0), ("pointwise", 1), ("uniform", 2)):
            def run():
                pair.pair_design_alloc(B, nv, meta.gmax, off, ph, ch, None, bu, 0.08, design, pi,
                                       obj, its, st, stream)
            run()
            e0 = TimingEvent()
            e1 = TimingEvent()
            e0.record(stream)
            for _ in range(reps):
                run()
            e1.record(stream)
            e1.synchronize()
            ms = e0.elapsed_time(e1) / reps
            out[name] = {"ms": round(ms, 4), "prompts_per_s": round(B / (ms * 1e-3), 1),
                         "mean_objective": float(obj.mean().item()),
                         "sweeps_mean": round(float(its.float().mean().item()), 1),
                         "sweeps_max": int(its.max().item())}
    if int(st.item()) != 0:
        raise RuntimeError(f"device status {int(st.item())} in the probability design")
    return out


def time_cps(pair, stream, wl, dev, reps=5, R=1):
    """Fixed-size conditional Poisson design on the ragged workload's prompt
    structure (B = 512, G_b ~ U{2..64}): the odds fit with the exact joint
    block, and one draw of every prompt, timed with events."""
    import torch

    w = wl.WORKLOADS["ragged"]
    meta = wl.host_meta(w)
    tgt = torch.from_numpy(wl.cps_targets(meta.offsets)).to(dev)
    off = torch.from_numpy(meta.offsets).to(dev)
    B, nv, G = meta.B, meta.nv, meta.gmax
    wv = torch.empty(nv, dtype=torch.float64, device=dev)
    n = torch.empty(B, dtype=torch.int32, device=dev)
    pj = torch.empty((B, G, G), dtype=torch.float32, device=dev)
    its = torch.empty(B, dtype=torch.int32, device=dev)
    mask = torch.empty((R, nv), dtype=torch.uint8, device=dev)
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    res = {"workload": f"B={B}, G_b~U{{2..64}}, nv={nv}, targets U[0.08, 0.92] scaled to an "
                       "integer sum"}
    with torch.cuda.stream(stream):
        for name, fn in (("fit_ms", lambda: pair.pair_cps_fit(B, nv, G, off, tgt, wv, n, pj, its,
                                                              st, stream)),
                         ("draw_ms", lambda: pair.pair_cps_draw(B, nv, G, off, wv, n, 7, 0, R,
                                                                mask, None, st, stream))):
            fn()
            e0 = TimingEvent()
            e1 = TimingEvent()
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            e1.synchronize()
            res[name] = round(e0.elapsed_time(e1) / reps, 4)
    res["fit_iters_mean"] = round(float(its.float().mean().item()), 1)
    res["fit_iters_max"] = int(its.max().item())
    if int(st.item()) != 0:
        raise RuntimeError(f"device status {int(st.item())} in the fixed-size design")
    return res


def time_exact_audit(pair, stream, B, nv, G, off, scores, rew, p, D, reps=10):
    """Exact design audit (Gram on the matrix cores + closed form) on the
    audit workload, timed with events on the launch stream.  HBM-bound: the
    algorithmic bytes are the score block read once."""
    import torch

    dev = scores.device
    ws = torch.empty(pair.pair_audit_exact_workspace_bytes(B, G, D), dtype=torch.uint8, device=dev)
    mse = torch.empty(B, dtype=torch.float64, device=dev)
    bias = torch.empty(B, dtype=torch.float64, device=dev)
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    with torch.cuda.stream(stream):
        def run():
            pair.pair_audit_exact(B, nv, G, off, scores, rew, p, None, 0, 0.0, mse, bias, None, ws,
                                  st, stream)
        run()
        e0 = TimingEvent()
        e1 = TimingEvent()
        e0.record(stream)
        for _ in range(reps):
            run()
        e1.record(stream)
        e1.synchronize()
    if int(st.item()) != 0:
        raise RuntimeError(f"device status {int(st.item())} in the exact audit")
    ms = e0.elapsed_time(e1) / reps
    nbytes = nv * D * 2
    gbps = nbytes / (ms * 1e-3) / 1e9
    return {"ms": round(ms, 4), "prompts_per_s": round(B / (ms * 1e-3), 1),
            "mean_mse": float(mse.mean().item()),
            "roofline": {"kernel": "gram_kernel + exact_final_kernel (pair_audit_exact)",
                         "bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS,
                         "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
                         "algorithmic_bytes": nbytes}}


def audit_matrix(pair, stream, wl, dev, R=1000, D=4096):
    """The frozen-policy audit matrix (App. E; the procedure behind the audit
    tables of Sec. 6.2) on a synthetic population: the ragged workload's
    prompt structure (B = 512, G_b ~ U{2..64}), rewards, prefix statistics and
    suffix lengths, with bf16 N(0, 1/D) scores of width D.  Each row's design
    is replayed over R draws against the complete-pair target: bias norm and
    MSE (pair_audit_rule), the mean cosine to the target
    (pair_audit_direction), and from the same draws (pair_design_inclusion)
    the completed vertices, observed edges and the suffix tokens spent as a
    fraction of the full group's.  Bias, MSE and cosine are averaged over the
    prompts whose target is nonzero, the rest over all prompts."""
    import numpy as np
    import torch

    w = wl.WORKLOADS["ragged"].replace(D=D)
    meta = wl.host_meta(w)
    inp = wl.alloc_inputs(w, meta.offsets)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    off, rew, ph, ch, bu = (t(a) for a in (meta.offsets, meta.rewards, inp.p_hat, inp.c_hat,
                                           inp.budget))
    B, nv, G = meta.B, meta.nv, meta.gmax
    scores = wl.device_scores(w, nv, dev)
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    designs = {"full": torch.ones(nv, dtype=torch.float32, device=dev)}
    with torch.cuda.stream(stream):
        for name, code in (("pair", pair.DESIGN_PAIR), ("pointwise", pair.DESIGN_POINTWISE),
                           ("uniform", pair.DESIGN_UNIFORM)):
            designs[name] = torch.empty(nv, dtype=torch.float32, device=dev)
            pair.pair_design_alloc(B, nv, G, off, ph, ch, None, bu, 0.08, code, designs[name],
                                   None, None, st, stream)
    rows = [("full candidate graph", "full", pair.RULE_HT),
            ("uniform vertex HT", "uniform", pair.RULE_HT),
            ("pointwise p(1-p) HT", "pointwise", pair.RULE_HT),
            ("adaptive unweighted", "pair", pair.RULE_UNWEIGHTED),
            ("marginal-only weighting", "pair", pair.RULE_MARGINAL),
            ("PAIR", "pair", pair.RULE_HT)]
    ws = torch.empty(pair.pair_audit_workspace_bytes(B, G, D, R), dtype=torch.uint8, device=dev)
    wsd = torch.empty(pair.pair_audit_direction_workspace_bytes(B, G, D, R), dtype=torch.uint8,
                      device=dev)
    mse = torch.empty(B, dtype=torch.float64, device=dev)
    bias = torch.empty(B, dtype=torch.float64, device=dev)
    cos = torch.empty(B, dtype=torch.float64, device=dev)
    tnorm = torch.empty(B, dtype=torch.float64, device=dev)
    mask = torch.empty((R, nv), dtype=torch.uint8, device=dev)
    ec = torch.empty((R, B), dtype=torch.int32, device=dev)
    comp = torch.empty((R, B), dtype=torch.int32, device=dev)
    sizes = torch.from_numpy(np.diff(meta.offsets)).to(dev)
    owner = torch.repeat_interleave(torch.arange(B, device=dev), sizes)
    c_tot = torch.zeros(B, dtype=torch.float64, device=dev).index_add_(0, owner, ch.double())
    seed = w.design_seed
    out = {"workload": f"ragged structure B={B}, nv={nv}, G_b~U{{2..64}}, D={D} bf16 N(0,1/D), "
                       f"R={R} draws per design; designs from pair_design_alloc (budget 0.5 sum c, "
                       f"pi_min 0.08)"}
    e0, e1 = TimingEvent(), TimingEvent()
    res = {}
    with torch.cuda.stream(stream):
        e0.record(stream)
        for label, dname, rule in rows:
            p = designs[dname]
            pair.pair_audit_rule(B, nv, G, off, scores, rew, p, None, rule, 0.0, seed, 0, R, mse,
                                 bias, None, None, ws, st, stream)
            pair.pair_audit_direction(B, nv, G, off, scores, rew, p, None, rule, 0.0, seed, 0, R,
                                      cos, tnorm, wsd, st, stream)
            pair.pair_design_inclusion(B, nv, G, off, p, seed, 0, R, mask, None, ec, comp, st,
                                       stream)
            cost = torch.zeros((R, B), dtype=torch.float64, device=dev).index_add_(
                1, owner, mask.double() * ch.double()[None, :]) / c_tot[None, :]
            live = tnorm > 0
            res[label] = {"bias": bias[live].mean(), "mse": mse[live].mean(), "cosine": cos[live].mean(),
                          "vertices": comp.double().mean(), "edges": ec.double().mean(),
                          "suffix_tokens": cost.mean()}
        e1.record(stream)
    torch.cuda.synchronize()
    if int(st.item()) != 0:
        raise RuntimeError(f"device status {int(st.item())} in the audit matrix")
    out["ms"] = round(e0.elapsed_time(e1), 3)
    out["rows"] = {k: {m: round(float(v.item()), 6) for m, v in r.items()} for k, r in res.items()}
    return out


def time_variants(pair, stream, B, nv, G, off, rew, mask, pi, coeff, audit_args, status, reps=5):
    """Estimator variants (edge-weight rules): the coefficient fold on the
    b128 draw and the audit replay on the audit workload, per rule, timed
    with events on the launch stream (outside the main timed steps)."""
    import torch

    Ba, nva, Ga, off_a, scores_a, rew_a, p_a, wa, R, mse, bias, rps, ec_a, ws = audit_args
    dev = coeff.device
    ess = torch.empty(B, dtype=torch.float32, device=dev)
    mw = torch.empty(B, dtype=torch.float32, device=dev)
    cos = torch.empty(Ba, dtype=torch.float64, device=dev)
    tnorm = torch.empty(Ba, dtype=torch.float64, device=dev)
    wsd = torch.empty(pair.pair_audit_direction_workspace_bytes(Ba, Ga, scores_a.shape[1], R),
                      dtype=torch.uint8, device=dev)
    out = {}
    with torch.cuda.stream(stream):
        for rule, name in enumerate(RULE_NAMES):
            wmax = 10.0 if name == "clipped" else 0.0

            def coeffs():
                pair.pair_edge_coeffs_rule(B, nv, G, off, rew, mask[0], pi, rule, wmax, coeff, None,
                                           ess, mw, status, stream)

            def audit():
                pair.pair_audit_rule(Ba, nva, Ga, off_a, scores_a, rew_a, p_a, None, rule, wmax,
                                     wa.design_seed, 0, R, mse, bias, rps, ec_a, ws, status, stream)

            def direction():
                pair.pair_audit_direction(Ba, nva, Ga, off_a, scores_a, rew_a, p_a, None, rule,
                                          wmax, wa.design_seed, 0, R, cos, tnorm, wsd, status,
                                          stream)

            res = {}
            for key, fn in (("coeffs_us", coeffs), ("audit_ms", audit),
                            ("direction_ms", direction)):
                fn()
                e0 = TimingEvent()
                e1 = TimingEvent()
                e0.record(stream)
                for _ in range(reps):
                    fn()
                e1.record(stream)
                e1.synchronize()
                t = e0.elapsed_time(e1) / reps
                res[key] = round(t * 1e3 if key == "coeffs_us" else t, 4)
            res["audit_mean_mse"] = float(mse.mean().item())
            res["audit_mean_bias"] = float(bias.mean().item())
            live = tnorm > 0
            res["audit_mean_cosine"] = round(float(cos[live].mean().item()), 6)
            res["b128_mean_ess"] = round(float(ess.mean().item()), 3)
            out[name] = res
    if int(status.item()) != 0:
        raise RuntimeError(f"device status {int(status.item())} in the variant timings")
    return out


def copy_calibration(gib=1.0, reps=5):
    """Plain device copy of known size, for scaling rocprofv3 FETCH/WRITE
    counters, timed with events; also a read-only reduction over a 4x larger
    buffer as a measured read ceiling."""
    import torch

    n = int(gib * (1 << 30)) // 2
    src = torch.empty(n, dtype=torch.bfloat16, device="cuda:0").normal_()
    dst = torch.empty_like(src)
    big = torch.empty(4 * n, dtype=torch.bfloat16, device="cuda:0").normal_()
    for _ in range(2):
        dst.copy_(src)
        big.sum()
    torch.cuda.synchronize()
    e = [TimingEvent() for _ in range(3)]
    cur = torch.cuda.current_stream()
    e[0].record(cur)
    for _ in range(reps):
        dst.copy_(src)
    e[1].record(cur)
    for _ in range(reps):
        big.sum()
    e[2].record(cur)
    torch.cuda.synchronize()
    copy_ms = e[0].elapsed_time(e[1]) / reps
    read_ms = e[1].elapsed_time(e[2]) / reps
    print(json.dumps({"copy_calibration_bytes": n * 2, "reps": reps,
                      "copy_GBps": round(2 * n * 2 / (copy_ms * 1e-3) / 1e9, 1),
                      "read_GBps": round(4 * n * 2 / (read_ms * 1e-3) / 1e9, 1)}), flush=True)


def counter_pass():
    """The program the traffic counter runs profile: COUNTER_PASS_CALLS calls
    each of the per-prompt and the batch-mean weighted gradient on every
    workload of GRAD_WORKLOADS, then of the audit on the audit workload, each
    call followed by a synchronisation, in that order."""
    import torch

    import paper_2608_11368_amd as pair
    import workloads as wl

    dev = torch.device("cuda:0")
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    for name in GRAD_WORKLOADS:
        w = wl.WORKLOADS[name]
        m = wl.host_meta(w)
        off, rew, p = (torch.from_numpy(a).to(dev) for a in (m.offsets, m.rewards, m.p))
        s = wl.device_scores(w, m.nv, dev)
        coeff = torch.empty(m.nv, dtype=torch.float32, device=dev)
        pair.pair_design_coeffs(m.B, m.nv, m.gmax, off, p, rew, w.design_seed, 0, coeff, None,
                                None, None, None, st)
        out = torch.empty((m.B, w.D), dtype=torch.float32, device=dev)
        mean = torch.empty(w.D, dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        for reduce, o in ((0, out), (1, mean)):
            for _ in range(COUNTER_PASS_CALLS):
                pair.pair_weighted_grad(m.B, m.nv, off, s, coeff, o, reduce, st)
                torch.cuda.synchronize()
        print(json.dumps({"counter_pass": name, "nonzero_rows": int(torch.count_nonzero(coeff))}),
              flush=True)
        del s, out, mean
        torch.cuda.empty_cache()
    audit_calls(COUNTER_PASS_CALLS)
    if int(st.item()) != 0:
        raise RuntimeError(f"device status {int(st.item())} in the counter pass")


def audit_calls(n):
    """`n` plain pair_audit calls on the audit workload (B=256, G=16,
    D=65536, R=4096), each followed by a synchronisation, and nothing else:
    the program a matrix-core counter pass profiles."""
    import torch

    import paper_2608_11368_amd as pair
    import workloads as wl

    dev = torch.device("cuda:0")
    wa = wl.WORKLOADS["audit"]
    m = wl.host_meta(wa)
    off, rew, p = (torch.from_numpy(a).to(dev) for a in (m.offsets, m.rewards, m.p))
    s = wl.device_scores(wa, m.nv, dev)
    ws = torch.empty(pair.pair_audit_workspace_bytes(m.B, m.gmax, wa.D, wa.R), dtype=torch.uint8,
                     device=dev)
    mse = torch.empty(m.B, dtype=torch.float64, device=dev)
    bias = torch.empty_like(mse)
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    for k in range(n):
        pair.pair_audit(m.B, m.nv, m.gmax, off, s, rew, p, None, wa.design_seed, 0, wa.R, mse, bias,
                        None, None, ws, st)
        torch.cuda.synchronize()
        if int(st.item()) != 0:
            raise RuntimeError(f"device status {int(st.item())} in audit call {k}")
        print(json.dumps({"audit_call": k, "mean_mse": float(mse.mean())}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--audit-calls", type=int, default=0, metavar="N")
    ap.add_argument("--counter-pass", action="store_true",
                    help="the fixed sequence of calls the traffic counter runs profile")
    ap.add_argument("--record-traffic", metavar="DIR",
                    help="write profiles/counters.json from rocprofv3 --pmc runs under DIR")
    args = ap.parse_args()

    if args.record_traffic:
        record_traffic(args.record_traffic)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one MI355X: the library runs on a single GPU "
              "(no collectives); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2608_11368_amd as pair
    import workloads as wl

    if args.copy_calibration:
        copy_calibration()
        return
    if args.audit_calls > 0:
        audit_calls(args.audit_calls)
        return
    if args.counter_pass:
        counter_pass()
        return

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.Stream(device=dev)

    # ---- gradient-chain inputs (b128) ----
    w = wl.WORKLOADS["b128"]
    meta = wl.host_meta(w)
    B, nv, G, D = meta.B, meta.nv, meta.gmax, w.D
    off = torch.from_numpy(meta.offsets).to(dev)
    rew = torch.from_numpy(meta.rewards).to(dev)
    p = torch.from_numpy(meta.p).to(dev)
    _log(f"[bench] generating b128 scores {nv}x{D} bf16")
    scores = wl.device_scores(w, nv, dev)
    mask = torch.empty((1, nv), dtype=torch.uint8, device=dev)
    pi = torch.empty((B, G, G), dtype=torch.float32, device=dev)
    ec = torch.empty((1, B), dtype=torch.int32, device=dev)
    comp = torch.empty((1, B), dtype=torch.int32, device=dev)
    coeff = torch.empty(nv, dtype=torch.float32, device=dev)
    out = torch.empty((B, D), dtype=torch.float32, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)

    # ---- audit inputs ----
    wa = wl.WORKLOADS["audit"]
    meta_a = wl.host_meta(wa)
    Ba, nva, Ga, Da, R = meta_a.B, meta_a.nv, meta_a.gmax, wa.D, wa.R
    off_a = torch.from_numpy(meta_a.offsets).to(dev)
    rew_a = torch.from_numpy(meta_a.rewards).to(dev)
    p_a = torch.from_numpy(meta_a.p).to(dev)
    _log(f"[bench] generating audit scores {nva}x{Da} bf16")
    scores_a = wl.device_scores(wa, nva, dev)
    ws = torch.empty(pair.pair_audit_workspace_bytes(Ba, Ga, Da, R), dtype=torch.uint8, device=dev)
    mse = torch.empty(Ba, dtype=torch.float64, device=dev)
    bias = torch.empty(Ba, dtype=torch.float64, device=dev)
    reps = torch.empty((Ba, R), dtype=torch.float32, device=dev)
    ec_a = torch.empty((Ba, R), dtype=torch.int32, device=dev)
    torch.cuda.synchronize()

    def step(ev):
        # design draw + coefficient fold in one launch (the mask and the
        # logged rho block are still written), then the weighted gradient,
        # then the audit; one event between consecutive stages
        ev[0].record(stream)
        pair.pair_design_coeffs(B, nv, G, off, p, rew, w.design_seed, 0, coeff, mask[0], pi, ec[0],
                                comp[0], status, stream)
        ev[1].record(stream)
        pair.pair_weighted_grad(B, nv, off, scores, coeff, out, 0, status, stream)
        ev[2].record(stream)
        pair.pair_audit(Ba, nva, Ga, off_a, scores_a, rew_a, p_a, None, wa.design_seed, 0, R, mse,
                        bias, reps, ec_a, ws, status, stream)
        ev[3].record(stream)

    def events():
        return [TimingEvent() for _ in range(4)]

    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            step(events())
        torch.cuda.synchronize()
        if int(status.item()) != 0:
            raise RuntimeError(f"device status {int(status.item())}")
        evs = [events() for _ in range(args.steps)]
        _log(f"[bench] timing {args.steps} steps")
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(args.steps):
            step(evs[k])
        torch.cuda.synchronize()
        t1 = time.perf_counter()

    def part(a, b):
        return float(np.mean([e[a].elapsed_time(e[b]) for e in evs]))   # ms

    ms_design, ms_wgrad, ms_audit = part(0, 1), part(1, 2), part(2, 3)
    ms_chain = part(0, 2)
    ms_step = (t1 - t0) * 1e3 / args.steps

    nz_rows = int(torch.count_nonzero(coeff).item())
    bytes_wgrad = nz_rows * D * 2 + nv * 4 + (B + 1) * 8 + B * D * 4
    bytes_dense = nv * D * 2 + nv * 4 + (B + 1) * 8 + B * D * 4
    gbps_chain = bytes_wgrad / (ms_chain * 1e-3) / 1e9
    gbps_wgrad = bytes_wgrad / (ms_wgrad * 1e-3) / 1e9
    # The audit sweeps only prompts whose rewards are not all equal: a prompt
    # with equal rewards has zero deviations in every replicate, and its
    # e_r, MSE and bias are exact zeros without any matrix work.
    live_a = int(sum(np.ptp(meta_a.rewards[meta_a.offsets[b]:meta_a.offsets[b + 1]]) > 0
                     for b in range(Ba)))
    flops_audit = 2.0 * live_a * R * Ga * Da
    tflops_audit = flops_audit / (ms_audit * 1e-3) / 1e12

    def roof_wgrad(key, kernel, ms, alg):
        gbps = alg / (ms * 1e-3) / 1e9
        return {"kernel": kernel, "workload": key.split("_")[-1], "bound": "hbm",
                "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(gbps / HBM_PEAK_GBPS, 4),
                "traffic": _traffic(key, ["wgrad.hip", "common.hpp"]),
                "ms": round(ms, 4), "algorithmic_bytes": alg}

    roof_w = roof_wgrad("wgrad_b128", "wgrad_kernel<bf16> (pair_weighted_grad)", ms_wgrad,
                        bytes_wgrad)
    roof_a = {"kernel": "pair_audit (coeffs + mean + mfma + finalize)", "bound": "mfma",
              "achieved": round(tflops_audit, 1), "peak": BF16_MFMA_PEAK_TFLOPS,
              "unit": "TFLOP/s", "frac": round(tflops_audit / BF16_MFMA_PEAK_TFLOPS, 4),
              "traffic": _traffic("audit_b256", ["audit.hip", "common.hpp"]),
              "ms": round(ms_audit, 4), "flops": flops_audit,
              "flops_note": "2*G*D per replicate estimate of the swept prompts",
              "swept_prompts": live_a, "swept_fraction": round(live_a / Ba, 4),
              "frac_if_all_prompts_counted": round(
                  2.0 * Ba * R * Ga * Da / (ms_audit * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4)}

    result = {
        "metric": METRIC,
        "value": round(gbps_chain, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "score_dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "b128 gradient chain + audit (timed step); per-prompt and batch-mean "
                        "gradient on b128, qwen3 and ragged",
            "grad": {"B": B, "G": G, "D": D, "scores": "bf16 N(0,1/D)", "nv": nv,
                     "rows_nonzero": nz_rows},
            "audit": {"B": Ba, "G": Ga, "D": Da, "R": R, "scores": "bf16 N(0,1/D)"},
        },
        "parts_ms": {"design_coeffs": round(ms_design, 4), "wgrad": round(ms_wgrad, 4),
                     "audit": round(ms_audit, 4)},
        "dense_equiv_GBps": round(bytes_dense / (ms_chain * 1e-3) / 1e9, 1),
        "score_only_GBps": round(nz_rows * D * 2 / (ms_wgrad * 1e-3) / 1e9, 1),
        "roofline": roof_w,
        "audit": {"value": round(Ba * R / (ms_audit * 1e-3), 1),
                  "unit": "replicate-estimates/s", "roofline": roof_a},
    }
    cfgs = time_wgrad_configs(pair, stream, wl, dev, coeff, out, scores, off, rew, p, mask, pi,
                              ec, comp, status, B, nv, G, D, w)
    result["wgrad_configs"] = cfgs
    # The headline roofline is the worst per-prompt weighted gradient of the
    # three gradient workloads in this run; every one, and the batch-mean
    # mode of each, is listed beside it.
    by_cfg = {"b128": roof_w}
    for name in ("qwen3", "ragged"):
        by_cfg[name] = roof_wgrad(f"wgrad_{name}", "wgrad_kernel<bf16> (pair_weighted_grad)",
                                  cfgs[name]["ms"], cfgs[name]["algorithmic_bytes"])
    for name in GRAD_WORKLOADS:
        rec = cfgs[name + "_batch_mean"]
        by_cfg[name + "_batch_mean"] = roof_wgrad(
            f"wgrad_mean_{name}", "wgrad_mean_kernel<bf16> (pair_weighted_grad, reduce=1)",
            rec["ms"], rec["algorithmic_bytes"])
    worst = min(GRAD_WORKLOADS, key=lambda k: by_cfg[k]["frac"])
    result["roofline"] = dict(by_cfg[worst], selection="worst per-prompt weighted gradient of "
                              "the b128, qwen3 and ragged workloads in this run")
    result["roofline_by_config"] = by_cfg
    result["config"]["grad_configs"] = {
        name: {k: cfgs[name][k] for k in ("B", "nv", "D", "rows_nonzero")}
        for name in ("qwen3", "ragged")}
    result["exact_audit"] = time_exact_audit(pair, stream, Ba, nva, Ga, off_a, scores_a, rew_a,
                                             p_a, Da)
    result["design_alloc"] = time_alloc(pair, stream, wl, dev)
    result["fixed_size_design"] = time_cps(pair, stream, wl, dev)
    result["variants"] = time_variants(pair, stream, B, nv, G, off, rew, mask, pi, coeff,
                                       (Ba, nva, Ga, off_a, scores_a, rew_a, p_a, wa, R, mse, bias,
                                        reps, ec_a, ws), status)
    result["audit_matrix"] = audit_matrix(pair, stream, wl, dev)
    if not args.no_cpu_baseline:
        _log("[bench] timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(meta, w, scores, meta_a, wa, scores_a)
        _log("[bench] timing the CPU oracle of the widened rows")
        for key, rec in cpu_next_rows(wl, meta_a, wa, scores_a).items():
            result[key]["cpu_oracle"] = rec
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
