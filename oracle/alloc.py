"""Graph-coupled probability design -- TEST INFRASTRUCTURE ONLY (the oracle of
the allocation solver; only tests/, the smoke check and the bench's CPU
baseline may use it).

Follows the paper's Sec. 4.3 (contrast graph) and Sec. 4.4 (graph-coupled
probability design) in fp64:

  disagreement      d_ij = p_i (1 - p_j) + (1 - p_i) p_j          Eq. (disagreement)
  edge proxy        a_ij = d_ij, or d_ij (m_i + m_j)^2 / 4 with a
                    score-norm predictor m                          Eq. (edge-proxy)
  vertex term       b_i  = (sum_{j != i} sqrt(a_ij))^2 - sum_{j != i} a_ij
  design            min_x  Phi(x) = sum_{i<j} a_ij e^{x_i + x_j} + sum_i b_i e^{x_i}
                    s.t.   sum_i c_i e^{-x_i} <= budget,  0 <= x_i <= -log(pi_min)
                                                                    Eqs. (convex-objective), (budget)
  probabilities     pi_i = e^{-x_i}

solved as the paper's implementation does (App. C "Probability
optimization"): SLSQP in double precision, here with tight tolerances so the
result is the optimum itself, and with pi = e^{-x} as the variables (the same
program and optimum; the budget is then linear).  Two comparison designs of the audit tables:
uniform (one probability, the same expected cost) and pointwise (the same
program with a = 0 and b_i = p_i (1 - p_i): each vertex's own Bernoulli
variance over its probability -- a reading, the paper names the design
without its formula).

Parity: the solver's output is pinned in tests/test_oracle_alloc.py by the
KKT conditions (checked independently of SLSQP), closed forms (two vertices,
symmetric graphs, slack and tight budgets), objective comparisons against
feasible alternatives, and the paper's bound b_i >= 2 sum |<h_ij, h_ik>| and
trace bound of App. A "Variance upper bound and convexity".
"""
from __future__ import annotations

import numpy as np
from scipy.optimize import minimize

PAIR = 0
POINTWISE = 1
UNIFORM = 2


def disagreement(p_hat):
    p = np.asarray(p_hat, dtype=np.float64)
    d = p[:, None] * (1.0 - p[None, :]) + (1.0 - p[:, None]) * p[None, :]
    np.fill_diagonal(d, 0.0)
    return d


def edge_proxy(p_hat, m_hat=None):
    a = disagreement(p_hat)
    if m_hat is not None:
        m = np.asarray(m_hat, dtype=np.float64)
        a = a * (m[:, None] + m[None, :]) ** 2 / 4.0
        np.fill_diagonal(a, 0.0)
    return a


def vertex_term(a):
    a = np.asarray(a, dtype=np.float64).copy()
    np.fill_diagonal(a, 0.0)
    return np.sum(np.sqrt(a), axis=1) ** 2 - np.sum(a, axis=1)


def objective_pi(pi, a, b):
    """Phi written in the probabilities: sum_{i<j} a_ij / (pi_i pi_j) + sum_i b_i / pi_i."""
    pi = np.asarray(pi, dtype=np.float64)
    iu = np.triu_indices(pi.size, 1)
    return float(np.sum(a[iu] / (pi[iu[0]] * pi[iu[1]])) + np.sum(b / pi))


def _solve(a, b, c, budget, pi_min):
    g = c.size
    if np.sum(c) <= budget:
        return np.ones(g), True
    if budget < pi_min * np.sum(c) * (1.0 - 1e-12):
        raise ValueError("budget below pi_min * sum(c): no feasible design")
    if budget <= pi_min * np.sum(c):
        return np.full(g, pi_min), True
    # The same program in pi = e^{-x}: Phi(pi) = sum_{i<j} a_ij / (pi_i pi_j)
    # + sum_i b_i / pi_i is convex in pi as well (so is x -> pi a bijection of
    # the box), and the budget becomes linear, which SLSQP handles far more
    # accurately than the exponential form.  The objective is scaled by its
    # value at the uniform start; the budget row by 1 / budget.
    sym = np.triu(a, 1) + np.triu(a, 1).T
    u0 = np.full(g, np.clip(budget / np.sum(c), pi_min, 1.0))
    f0 = max(objective_pi(u0, a, b), 1e-300)
    cs = c / budget

    def phi(u):
        iu = 1.0 / u
        return (0.5 * iu @ sym @ iu + b @ iu) / f0

    def grad(u):
        iu = 1.0 / u
        return -(iu * iu) * (sym @ iu + b) / f0

    cons = {"type": "ineq", "fun": lambda u: 1.0 - float(cs @ u), "jac": lambda u: -cs}
    res = minimize(phi, u0, jac=grad, bounds=[(pi_min, 1.0)] * g, constraints=[cons],
                   method="SLSQP", options={"ftol": 1e-16, "maxiter": 5000})
    pi = np.clip(res.x, pi_min, 1.0)
    # SLSQP may end on a line-search flag at the optimum; success is judged by
    # the KKT conditions instead.
    ok = kkt_residual(pi, a, b, c, budget, pi_min)[0] <= 1e-5
    return pi, ok


def solve(p_hat, c_hat, budget, pi_min, design=PAIR, m_hat=None):
    """Continuation probabilities of one prompt under a design (PAIR, POINTWISE,
    UNIFORM).  Returns dict(pi, objective, a, b, success); the objective is
    the PAIR proxy Phi evaluated at pi."""
    p = np.asarray(p_hat, dtype=np.float64)
    c = np.asarray(c_hat, dtype=np.float64)
    a = edge_proxy(p, m_hat)
    b = vertex_term(a)
    if design == UNIFORM:
        pi = np.full(p.size, np.clip(budget / np.sum(c), pi_min, 1.0))
        ok = True
    elif design == POINTWISE:
        pi, ok = _solve(np.zeros_like(a), p * (1.0 - p), c, budget, pi_min)
    else:
        pi, ok = _solve(a, b, c, budget, pi_min)
    return {"pi": pi, "objective": objective_pi(pi, a, b), "a": a, "b": b, "success": ok}


def kkt_residual(pi, a, b, c, budget, pi_min):
    """Largest violation of the KKT conditions of the design in the variables
    pi (the program is convex in pi as well): with A_i = sum_j a_ij / pi_j + b_i,
    d Phi / d pi_i = -A_i / pi_i^2, and one multiplier lam >= 0 for the budget:
      interior i:    A_i / pi_i^2 = lam c_i
      pi_i = 1:      A_i / pi_i^2 >= lam c_i
      pi_i = pi_min: A_i / pi_i^2 <= lam c_i
    lam is fitted from the interior coordinates.  Returns (residual, lam)."""
    pi = np.asarray(pi, dtype=np.float64)
    A = (a / pi[None, :]).sum(axis=1) - np.diag(a) / pi + b
    gneg = A / pi ** 2
    tol = 1e-7
    interior = (pi > pi_min * (1 + tol)) & (pi < 1 - tol)
    spent = float(c @ pi)
    if interior.any():
        lam = float(np.median(gneg[interior] / c[interior]))
    elif spent < budget * (1 - 1e-9):
        lam = 0.0
    else:
        lo = np.max(np.where(pi <= pi_min * (1 + tol), gneg / c, 0.0))
        lam = lo
    scale = max(float(np.max(gneg / c)), 1e-300)
    r = 0.0
    if interior.any():
        r = max(r, float(np.max(np.abs(gneg[interior] / c[interior] - lam))) / scale)
    top = pi >= 1 - tol
    if top.any():
        r = max(r, float(np.max(np.maximum(lam - gneg[top] / c[top], 0.0))) / scale)
    bot = pi <= pi_min * (1 + tol)
    if bot.any():
        r = max(r, float(np.max(np.maximum(gneg[bot] / c[bot] - lam, 0.0))) / scale)
    if lam > 0:
        r = max(r, abs(spent - budget) / budget)
    r = max(r, max(spent - budget, 0.0) / budget)
    return r, lam


def solve_batch(offsets, p_hat, c_hat, budget, pi_min, design=PAIR, m_hat=None):
    """Every prompt of a packed batch; budget is per prompt [B].  Returns
    dict(pi[nv], objective[B], success[B])."""
    off = np.asarray(offsets, dtype=np.int64)
    B = off.size - 1
    pi = np.zeros(int(off[-1]), dtype=np.float64)
    obj = np.zeros(B)
    ok = np.zeros(B, dtype=bool)
    for b in range(B):
        lo, hi = off[b], off[b + 1]
        r = solve(p_hat[lo:hi], c_hat[lo:hi], float(budget[b]), pi_min, design,
                  None if m_hat is None else m_hat[lo:hi])
        pi[lo:hi] = r["pi"]
        obj[b] = r["objective"]
        ok[b] = r["success"]
    return {"pi": pi, "objective": obj, "success": ok}
