"""Seeded synthetic inputs for the PAIR estimator workloads.

This module only *draws inputs*: prompt offsets, rewards, continuation
probabilities and score matrices.  It contains none of the estimator's
arithmetic (no design draw, no joint inclusion probability, no edge term), so
both the HIP path and the CPU oracle may use it.

Workloads (shapes and value distributions of the paper's setting: groups of
G = 8..64 candidate rollouts per prompt, binary or partial-credit rewards,
positive continuation probabilities with a floor, per-rollout score vectors on
one parameter block):

  tiny     B=4,   G=8,  D=4096,  fp32 scores ~ N(0,1), rewards ~ Bernoulli(0.5),
           p ~ U[0.2, 1], one design draw
  b128     B=128, G=16, D=2^20,  bf16 scores ~ N(0, 1/D), rewards ~ Bernoulli(q_b),
           q_b ~ Beta(1/2, 1/2), p ~ U[0.1, 1]
  qwen3    B=64,  G=8,  D=2^26,  bf16 scores ~ N(0, 1/D) (a 1.7B-parameter-model
           layer-scale chunk), rewards ~ Bernoulli(q_b), q_b ~ U[0, 1],
           p = clip(sigmoid(z), 0.05, 1), z ~ N(0, 1)
  audit    B=256, G=16, D=65536, bf16 scores ~ N(0, 1/D), rewards and p as b128,
           R=4096 design replicates per prompt
  ragged   B=512, G_b ~ U{2..64}, D=2^18, bf16 scores ~ N(0, 1/D),
           rewards ~ U[0, 1], predicted suffix length c_i ~ LogNormal with mean
           4000 tokens and sigma 1, p_i = clip(kappa / c_i, 0.05, 1) with kappa
           chosen per prompt (bisection) so that sum_i p_i c_i = 0.5 sum_i c_i

Every D above is a power of 4, so the 1/sqrt(D) score scale is a power of two
and scaling a bf16 sample by it is exact.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    G: int | None           # None => ragged group sizes
    D: int
    dtype: str
    R: int
    reward: str             # "bern_half" | "bern_beta" | "bern_unif" | "unif"
    prob: str               # "u0.2" | "u0.1" | "logit" | "budget"
    score_std: str          # "unit" | "inv_sqrt_d"
    gmin: int = 2
    gmax_ragged: int = 64
    data_seed: int = 0
    design_seed: int = 0

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    @property
    def gmax(self) -> int:
        return self.G if self.G is not None else self.gmax_ragged


WORKLOADS = {
    "tiny": Workload("tiny", B=4, G=8, D=4096, dtype=F32, R=1, reward="bern_half", prob="u0.2",
                     score_std="unit", data_seed=1001, design_seed=2001),
    "b128": Workload("b128", B=128, G=16, D=1 << 20, dtype=BF16, R=1, reward="bern_beta",
                     prob="u0.1", score_std="inv_sqrt_d", data_seed=1002, design_seed=2002),
    "qwen3": Workload("qwen3", B=64, G=8, D=1 << 26, dtype=BF16, R=1, reward="bern_unif",
                      prob="logit", score_std="inv_sqrt_d", data_seed=1003, design_seed=2003),
    "audit": Workload("audit", B=256, G=16, D=65536, dtype=BF16, R=4096, reward="bern_beta",
                      prob="u0.1", score_std="inv_sqrt_d", data_seed=1004, design_seed=2004),
    "ragged": Workload("ragged", B=512, G=None, D=1 << 18, dtype=BF16, R=1, reward="unif",
                       prob="budget", score_std="inv_sqrt_d", data_seed=1005, design_seed=2005),
}


@dataclasses.dataclass
class HostMeta:
    offsets: np.ndarray     # int64 [B+1]
    rewards: np.ndarray     # float32 [nv]
    p: np.ndarray           # float32 [nv], continuation probabilities in (0, 1]
    gmax: int

    @property
    def B(self) -> int:
        return self.offsets.size - 1

    @property
    def nv(self) -> int:
        return int(self.offsets[-1])


def _budget_probs(rng: np.random.Generator, g: int) -> np.ndarray:
    """Suffix-length-driven probabilities at half the expected full-group cost."""
    sigma = 1.0
    mu = math.log(4000.0) - 0.5 * sigma * sigma           # LogNormal mean 4000
    c = rng.lognormal(mu, sigma, size=g)
    target = 0.5 * c.sum()

    def spent(kappa):
        return float(np.sum(np.clip(kappa / c, 0.05, 1.0) * c))

    lo, hi = 0.0, float(c.max())
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if spent(mid) < target:
            lo = mid
        else:
            hi = mid
    return np.clip(hi / c, 0.05, 1.0)


def host_meta(w: Workload, seed: int | None = None) -> HostMeta:
    """Offsets, rewards and continuation probabilities for workload ``w``."""
    rng = np.random.default_rng(w.data_seed if seed is None else seed)
    if w.G is not None:
        sizes = np.full(w.B, w.G, dtype=np.int64)
    else:
        sizes = rng.integers(w.gmin, w.gmax_ragged + 1, size=w.B).astype(np.int64)
    offsets = np.zeros(w.B + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(sizes)
    rewards, probs = [], []
    for g in sizes:
        g = int(g)
        if w.reward == "bern_half":
            r = rng.random(g) < 0.5
        elif w.reward == "bern_beta":
            q = rng.beta(0.5, 0.5)
            r = rng.random(g) < q
        elif w.reward == "bern_unif":
            q = rng.random()
            r = rng.random(g) < q
        elif w.reward == "unif":
            r = rng.random(g)
        else:
            raise ValueError(w.reward)
        if w.prob == "u0.2":
            p = rng.uniform(0.2, 1.0, g)
        elif w.prob == "u0.1":
            p = rng.uniform(0.1, 1.0, g)
        elif w.prob == "logit":
            z = rng.standard_normal(g)
            p = np.clip(1.0 / (1.0 + np.exp(-z)), 0.05, 1.0)
        elif w.prob == "budget":
            p = _budget_probs(rng, g)
        else:
            raise ValueError(w.prob)
        rewards.append(np.asarray(r, dtype=np.float32))
        probs.append(np.asarray(p, dtype=np.float32))
    rew = np.concatenate(rewards).astype(np.float32)
    pr = np.concatenate(probs).astype(np.float32)
    pr = np.minimum(pr, np.float32(1.0))
    return HostMeta(offsets=offsets, rewards=rew, p=pr, gmax=int(w.gmax))


@dataclasses.dataclass
class AllocInputs:
    p_hat: np.ndarray      # float32 [nv] predicted success probabilities
    c_hat: np.ndarray      # float32 [nv] predicted remaining suffix tokens
    budget: np.ndarray     # float32 [B] expected-cost budget per prompt


def alloc_inputs(w: Workload, offsets: np.ndarray, ratio: float = 0.5,
                 seed: int | None = None) -> AllocInputs:
    """Prefix statistics for the probability design: predicted success
    uniform on [0.02, 0.98], predicted suffix lengths LogNormal with mean 4000
    tokens (sigma 1), and a budget of `ratio` times each prompt's total
    predicted cost (the configuration's default budget ratio is 0.5)."""
    rng = np.random.default_rng((w.data_seed if seed is None else seed) + 104729)
    nv = int(offsets[-1])
    p_hat = rng.uniform(0.02, 0.98, nv).astype(np.float32)
    sigma = 1.0
    c_hat = rng.lognormal(math.log(4000.0) - 0.5 * sigma * sigma, sigma, nv).astype(np.float32)
    budget = np.array([ratio * float(np.sum(c_hat[offsets[b]:offsets[b + 1]], dtype=np.float64))
                       for b in range(offsets.size - 1)], dtype=np.float32)
    return AllocInputs(p_hat=p_hat, c_hat=c_hat, budget=budget)


def cps_targets(offsets: np.ndarray, seed: int = 4242, lo: float = 0.08, hi: float = 0.92
                ) -> np.ndarray:
    """Target first-order probabilities for the fixed-size design: uniform on
    [lo, hi] per candidate, then scaled within each prompt so that the sum is
    the nearest admissible integer n (1 <= n < G), all values staying below 1.
    float32 [nv]."""
    rng = np.random.default_rng(seed)
    out = np.zeros(int(offsets[-1]), dtype=np.float32)
    for b in range(offsets.size - 1):
        lo_i, hi_i = int(offsets[b]), int(offsets[b + 1])
        g = hi_i - lo_i
        while True:
            t = rng.uniform(lo, hi, g)
            n = int(min(max(round(t.sum()), 1), g - 1))
            t = t * (n / t.sum())
            if t.max() < 0.97:
                break
        out[lo_i:hi_i] = t.astype(np.float32)
    return out


def cps_odds(offsets: np.ndarray, seed: int = 777) -> tuple[np.ndarray, np.ndarray]:
    """Synthetic odds (float64 [nv], LogNormal(0, 1)) and sample sizes
    (int32 [B], uniform on 1..G-1) for the fixed-size draw."""
    rng = np.random.default_rng(seed)
    nv = int(offsets[-1])
    w = rng.lognormal(0.0, 1.0, nv)
    n = np.array([rng.integers(1, int(offsets[b + 1] - offsets[b]))
                  for b in range(offsets.size - 1)], dtype=np.int32)
    return w, n


def score_scale(w: Workload) -> float:
    return 1.0 if w.score_std == "unit" else 1.0 / math.sqrt(w.D)


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (torch's round-to-nearest-even) and return the bits."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def host_scores(w: Workload, nv: int, seed: int | None = None, ld: int | None = None) -> np.ndarray:
    """Score matrix [nv][ld] on the host: float32, or uint16 bf16 bit patterns.

    Columns D..ld-1 (row padding) are filled with NaN so that any kernel that
    reads past D corrupts its result visibly.
    """
    rng = np.random.default_rng((w.data_seed if seed is None else seed) + 7919)
    ld = w.D if ld is None else ld
    x = rng.standard_normal((nv, w.D), dtype=np.float32) * np.float32(score_scale(w))
    if ld != w.D:
        full = np.full((nv, ld), np.nan, dtype=np.float32)
        full[:, : w.D] = x
        x = full
    return x if w.dtype == F32 else _bf16_bits(x)


def device_scores(w: Workload, nv: int, device, seed: int | None = None, ld: int | None = None):
    """Score matrix [nv][ld] drawn directly in device memory with torch's seeded
    generator (row by row, so no full-size fp32 temporary).  bf16 samples are
    scaled by a power of two, which is exact."""
    import torch

    ld = w.D if ld is None else ld
    dt = torch.float32 if w.dtype == F32 else torch.bfloat16
    gen = torch.Generator(device=device)
    gen.manual_seed((w.data_seed if seed is None else seed) + 7919)
    out = torch.empty((nv, ld), dtype=dt, device=device)
    if ld != w.D:
        out[:, w.D:] = float("nan")
    scale = score_scale(w)
    rows_per_call = max(1, (1 << 28) // max(w.D, 1))
    for r0 in range(0, nv, rows_per_call):
        r1 = min(nv, r0 + rows_per_call)
        blk = out[r0:r1, : w.D]
        blk.normal_(generator=gen)
        if scale != 1.0:
            blk.mul_(scale)
    return out
