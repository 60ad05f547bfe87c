"""Readout distributions and the speculative-sampling operators, in fp64.

TEST INFRASTRUCTURE: part of the CPU oracle.  Only tests/, the smoke check and
the benchmark's CPU-baseline leg may import it.

Sources (LoopSpec paper):
  * post-layers C: temperature scaling, optional top-k/top-p, softmax
    (Preliminaries, Looped Transformers);
  * residual operator  (mu (-) nu)(v) = [mu - nu]_+(v) / sum_u [mu - nu]_+(u)
    (Eq. residual-op);
  * acceptance min{1, p(x)/q(x)} and residual resampling (Eqs. acceptance,
    residual);
  * total variation  TV(p,q) = sum_x [p - q]_+(x)  (Proofs, Definition).

Readings where the paper is silent:
  * greedy (T = 0) is a one-hot distribution at the arg-max, ties to the lowest id;
  * top-p keeps token v iff the mass of the tokens ranked strictly before v
    (descending probability, ties by lower id) is < top_p, then renormalises;
    top-k is not used;
  * (mu (-) nu) with zero positive mass is undefined in the paper; the oracle
    returns mu and reports the event (it is unreachable in exact arithmetic);
  * a categorical draw x ~ w is an exponential race: x = argmax_v w_v / E_v with
    E_v = -log U_v and independent uniforms U_v in (0,1); ids with w_v = 0 never
    win; exact ties go to the lowest id.
"""
from __future__ import annotations

import numpy as np


def argmax_lowest(x: np.ndarray) -> int:
    """Index of the maximum; the lowest index among exact ties (np.argmax's rule)."""
    return int(np.argmax(x))


def top2_margin(x: np.ndarray) -> float:
    """Gap between the largest and second largest entries."""
    if x.size < 2:
        return float("inf")
    a = np.partition(np.asarray(x, np.float64), -2)[-2:]
    return float(a[1] - a[0])


def readout_dist(logits: np.ndarray, temperature: float, top_p: float = 1.0) -> np.ndarray:
    """Next-token distribution from readout logits: T, then softmax, then top-p."""
    z = np.asarray(logits, dtype=np.float64)
    if temperature == 0.0:
        p = np.zeros_like(z)
        p[argmax_lowest(z)] = 1.0
        return p
    z = z / temperature
    e = np.exp(z - z.max())
    p = e / e.sum()
    if top_p < 1.0:
        order = np.lexsort((np.arange(p.size), -p))        # descending p, ties by id
        before = np.cumsum(p[order]) - p[order]            # mass ranked strictly before
        keep = np.zeros(p.size, bool)
        keep[order] = before < top_p
        p = np.where(keep, p, 0.0)
        p = p / p.sum()
    return p


def positive_part(mu: np.ndarray, nu: np.ndarray) -> np.ndarray:
    return np.maximum(np.asarray(mu, np.float64) - np.asarray(nu, np.float64), 0.0)


def residual(mu: np.ndarray, nu: np.ndarray):
    """(mu (-) nu); returns (distribution, zero_mass) where zero_mass flags sum [mu-nu]_+ <= 0."""
    d = positive_part(mu, nu)
    s = d.sum()
    if not s > 0.0:
        return np.asarray(mu, np.float64).copy(), True
    return d / s, False


def tv(p: np.ndarray, q: np.ndarray) -> float:
    return float(positive_part(p, q).sum())


def race_sample(w: np.ndarray, u: np.ndarray):
    """Exponential race: argmax_v w_v / (-log u_v) over w_v > 0.

    Returns (token, relative gap between the two best race values); the gap lets
    a caller recognise draws that a lower-precision implementation could flip.
    """
    w = np.asarray(w, np.float64)
    e = -np.log(np.asarray(u, np.float64))
    score = np.where(w > 0.0, w / e, -np.inf)
    x = argmax_lowest(score)
    if not np.isfinite(score[x]):
        raise ValueError("race over an all-zero weight vector")
    s = np.sort(score[np.isfinite(score)])
    gap = float("inf") if s.size < 2 else float((s[-1] - s[-2]) / s[-1])
    return x, gap
