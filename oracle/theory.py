"""Closed forms and exact laws from the paper's analysis.

TEST INFRASTRUCTURE: part of the CPU oracle.  Only tests/, the smoke check and
the benchmark's CPU-baseline leg may import it.

  * Theorem 2 (proposal depth selection) and its bound
        E[C] <= f(d1, d2) = d1 + beta d1^-alpha d2 + 2 beta d2^-alpha R
    (Eq. upper-C), the closed-form stationary point (Eq. optimal_depths), the
    Hessian of f and the validity condition on R;
  * the power-law envelope phi(r) = beta r^-alpha fitted so that phi >= TV and
    max_r phi(r)/TV_r is minimal (Sec. 4.1, Observation);
  * the branch-growth recurrence s_k = s_{k-1} + s_{k - d2/d1}, s_k = 1 for
    k < d2/d1, B = sum_{k < R/d1} s_k (Sec. 4.3, Gating mechanism);
  * the exact law of the token that the cascade verification commits, and of a
    full restart, for given p_R, q1 = p_{d1} and q2~ = p_{d2} (Theorem 1 and its
    proof; speculative sampling's acceptance probability, Proofs).
  * the mean accepted length gamma (Implementation and Metrics).
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, List, Tuple

import numpy as np

from . import dist as D


# ----------------------------------------------------------------------------
# Theorem 2
# ----------------------------------------------------------------------------
def f_bound(d1: float, d2: float, alpha: float, beta: float, R: float) -> float:
    return d1 + beta * d1 ** (-alpha) * d2 + 2.0 * beta * d2 ** (-alpha) * R


def f_grad(d1, d2, alpha, beta, R) -> Tuple[float, float]:
    g1 = 1.0 - alpha * beta * d1 ** (-alpha - 1.0) * d2
    g2 = beta * d1 ** (-alpha) - 2.0 * alpha * beta * R * d2 ** (-alpha - 1.0)
    return g1, g2


def f_hessian(d1, d2, alpha, beta, R) -> np.ndarray:
    return np.array([
        [alpha * (alpha + 1) * beta * d1 ** (-alpha - 2) * d2, -alpha * beta * d1 ** (-alpha - 1)],
        [-alpha * beta * d1 ** (-alpha - 1), 2 * alpha * (alpha + 1) * beta * R * d2 ** (-alpha - 2)],
    ])


def optimal_depths(alpha: float, beta: float, R: float) -> Tuple[float, float]:
    """(d1*, d2*) of Eq. optimal_depths."""
    den = alpha * alpha + alpha + 1.0
    ab, aR = alpha * beta, 2.0 * alpha * R
    d1 = ab ** ((alpha + 1.0) / den) * aR ** (1.0 / den)
    d2 = ab ** (alpha / den) * aR ** ((alpha + 1.0) / den)
    return d1, d2


def validity_threshold(alpha: float, beta: float) -> float:
    """Theorem 2 holds for R strictly above this value."""
    ab = alpha * beta
    return max(ab ** (1 / alpha), ab ** (-alpha - 1),
               ab ** (1 / alpha) * (2 * alpha) ** ((alpha ** 2 + alpha + 1) / alpha ** 2)) \
        / (2 * alpha)


def integer_argmin(alpha: float, beta: float, R: int, d2_max: int = 0):
    """Integer (d1, d2), 1 <= d1 < d2 < R, minimising f; returns (d1, d2, f)."""
    best = None
    for d1 in range(1, R - 1):
        for d2 in range(d1 + 1, (d2_max or R - 1) + 1):
            v = f_bound(d1, d2, alpha, beta, R)
            if best is None or v < best[2]:
                best = (d1, d2, v)
    return best


# ----------------------------------------------------------------------------
# power-law envelope
# ----------------------------------------------------------------------------
def envelope_fit(tv: Dict[int, float], alpha_max: float = 8.0) -> Tuple[float, float, float]:
    """Fit phi(r) = beta r^-alpha >= TV_r minimising max_r phi(r)/TV_r.

    For a fixed alpha the smallest admissible beta is max_r TV_r r^alpha, and the
    objective becomes max_r(TV_r r^alpha) / min_r(TV_r r^alpha): the exponential
    of the range of log TV_r + alpha log r, a convex function of alpha.
    Returns (alpha, beta, objective).
    """
    rs = np.array(sorted(r for r in tv if tv[r] > 0), float)
    lt = np.log(np.array([tv[int(r)] for r in rs]))
    lr = np.log(rs)

    def obj(a):
        y = lt + a * lr
        return y.max() - y.min()

    lo, hi = 1e-9, alpha_max
    g = (math.sqrt(5) - 1) / 2
    x1, x2 = hi - g * (hi - lo), lo + g * (hi - lo)
    f1, f2 = obj(x1), obj(x2)
    for _ in range(200):
        if f1 <= f2:
            hi, x2, f2 = x2, x1, f1
            x1 = hi - g * (hi - lo)
            f1 = obj(x1)
        else:
            lo, x1, f1 = x1, x2, f2
            x2 = lo + g * (hi - lo)
            f2 = obj(x2)
    a = (lo + hi) / 2
    beta = float(np.exp((lt + a * lr).max()))
    return float(a), beta, float(np.exp(obj(a)))


# ----------------------------------------------------------------------------
# branch growth
# ----------------------------------------------------------------------------
def branch_growth(R: int, d1: int, d2: int) -> Tuple[List[int], int]:
    """s_k and B = sum_{k=0}^{R/d1-1} s_k for aligned depths (d1 | d2, d1 | R)."""
    if d2 % d1 or R % d1:
        raise ValueError("the recurrence assumes d1 | d2 and d1 | R")
    m = d2 // d1
    s: List[int] = []
    for k in range(R // d1):
        s.append(1 if k < m else s[k - 1] + s[k - m])
    return s, sum(s)


# ----------------------------------------------------------------------------
# exact laws of the cascade
# ----------------------------------------------------------------------------
def cascade_law(p, q1, q2t, gate: str = "gated") -> Tuple[np.ndarray, float, float, float]:
    """Exact distribution of the committed token under the cascade.

    gate = "gated": second proposal iff q2~(x1) < q1(x1); "open": always;
    "closed": never.  Returns (law, Pr[accept1], Pr[accept2], Pr[restart]).
    """
    p, q1, q2t = (np.asarray(a, np.float64) for a in (p, q1, q2t))
    V = p.size
    law = np.zeros(V)
    acc1 = acc2 = restart = 0.0
    rho1, _ = D.residual(p, q1)
    q2, _ = D.residual(q2t, q1)
    rho2, _ = D.residual(rho1, q2)
    for x1 in range(V):
        if q1[x1] == 0:
            continue
        a1 = min(1.0, p[x1] / q1[x1])
        law[x1] += q1[x1] * a1
        acc1 += q1[x1] * a1
        rej = q1[x1] * (1.0 - a1)
        if rej == 0:
            continue
        opened = gate == "open" or (gate == "gated" and q2t[x1] < q1[x1])
        if not opened:
            law += rej * rho1
            restart += rej
            continue
        for x2 in range(V):
            if q2[x2] == 0:
                continue
            a2 = min(1.0, rho1[x2] / q2[x2])
            law[x2] += rej * q2[x2] * a2
            acc2 += rej * q2[x2] * a2
            law += rej * q2[x2] * (1.0 - a2) * rho2
            restart += rej * q2[x2] * (1.0 - a2)
    return law, acc1, acc2, restart


def cascade_law_variant(p, q1, q2t, variant: int) -> Tuple[np.ndarray, float, float, float]:
    """cascade_law for a second-proposal variant of the ablation (Table 3), whose
    second proposal may depend on the first (masking): for every x1 the
    second proposal is drawn from second_proposal(q1, q2~, x1, variant) and
    verified against rho1 = p (-) q1 like any proposal of the cascade."""
    from .loopspec import second_proposal
    p, q1, q2t = (np.asarray(a, np.float64) for a in (p, q1, q2t))
    V = p.size
    law = np.zeros(V)
    acc1 = acc2 = restart = 0.0
    rho1, _ = D.residual(p, q1)
    for x1 in range(V):
        if q1[x1] == 0:
            continue
        a1 = min(1.0, p[x1] / q1[x1])
        law[x1] += q1[x1] * a1
        acc1 += q1[x1] * a1
        rej = q1[x1] * (1.0 - a1)
        if rej == 0:
            continue
        q2, _ = second_proposal(q1, q2t, x1, variant)
        if q2 is None:
            law += rej * rho1
            restart += rej
            continue
        rho2, _ = D.residual(rho1, q2)
        for x2 in range(V):
            if q2[x2] == 0:
                continue
            a2 = min(1.0, rho1[x2] / q2[x2])
            law[x2] += rej * q2[x2] * a2
            acc2 += rej * q2[x2] * a2
            law += rej * q2[x2] * (1.0 - a2) * rho2
            restart += rej * q2[x2] * (1.0 - a2)
    return law, acc1, acc2, restart


def gamma(n_decode: int, n_acc1: int, n_acc2: int, R: int, d1: int, d2: int) -> float:
    den = n_acc1 * d1 + n_acc2 * d2 + (n_decode - n_acc1 - n_acc2) * R
    return n_decode * R / den


def worst_case_branches(R: int, d1: int, d2: int, steps: int = 0, accept: int = 1) -> int:
    """Largest active set (effective batch) Alg. 1 reaches when every gate opens
    and every verification accepts proposal `accept`.  Brute-force tree
    simulation; for aligned depths it equals B of the branch-growth recurrence.
    Children spawned inside a subtree pruned in the same step never count."""
    nodes = {0: {"r": 0, "kids": []}}
    nid, root, peak = 1, 0, 1
    for _ in range(steps or 16 * R):
        peak = max(peak, len(nodes))
        for b in list(nodes):
            nb = nodes[b]
            nb["r"] += 1
            if nb["r"] == d1 or (d2 and nb["r"] == d2):
                nodes[nid] = {"r": 0, "kids": []}
                nb["kids"].append(nid)
                nid += 1
        if nodes[root]["r"] == R:
            kids = nodes[root]["kids"]
            keep = kids[min(accept, len(kids)) - 1]
            alive, stack = set(), [keep]
            while stack:
                x = stack.pop()
                alive.add(x)
                stack.extend(nodes[x]["kids"])
            nodes = {k: v for k, v in nodes.items() if k in alive}
            root = keep
        peak = max(peak, len(nodes))
    return peak
