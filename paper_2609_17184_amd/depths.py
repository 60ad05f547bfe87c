"""Choosing the proposal depths (d1, d2) from the model's own readouts.

Host-side planning around the decode path (no step of a decode runs here):

  * Sec. 4.1, Observation: the total-variation distance TV(p_r, p_R) between
    the readout distribution at an intermediate depth r and the final one
    shrinks with depth, under a power-law envelope phi(r) = beta r^-alpha with
    phi >= TV at every depth, (alpha, beta) chosen to minimise the largest
    ratio phi(r) / TV_r;
  * Sec. 5, Theorem 2: with that envelope the expected number of decode steps
    per committed token is at most
        f(d1, d2) = d1 + beta d1^-alpha d2 + 2 beta d2^-alpha R,
    minimised over the reals at
        d1* = (alpha beta)^((alpha+1)/D) (2 alpha R)^(1/D),
        d2* = (alpha beta)^(alpha/D) (2 alpha R)^((alpha+1)/D),  D = alpha^2 + alpha + 1,
    valid when 1 <= d1* < d2* < R.

The readouts come from the library (teacher-forced readout logits at every
depth along a token sequence); this module turns them into distributions
(temperature, then top-p), averages TV per depth, fits the envelope and
returns the integer pair that minimises f (the closed form is reported with
its validity, since at small R it often falls outside 1 <= d1 < d2 < R).

The envelope fit is exact: in log space the objective max_r phi(r)/TV_r is
the range of y_r + alpha x_r (y = log TV_r, x = log r) over the depths, a
convex piecewise-linear function of alpha whose minimum sits where two of
the lines cross (or at alpha -> 0); every crossing is evaluated.
"""
from __future__ import annotations

import itertools
import math
from typing import Dict, Optional, Sequence, Tuple

import numpy as np


def readout_probs(logits: np.ndarray, temperature: float, top_p: float) -> np.ndarray:
    """Rows of logits -> readout distributions: softmax(z / T), then top-p keeps
    a token when the mass ranked strictly before it (descending probability,
    ties by lower id) is below top_p, renormalised.  T = 0: one-hot argmax."""
    z = np.asarray(logits, np.float64)
    if temperature == 0.0:
        out = np.zeros_like(z)
        out[np.arange(z.shape[0]), np.argmax(z, axis=1)] = 1.0
        return out
    z = z / temperature
    z -= z.max(axis=1, keepdims=True)
    e = np.exp(z)
    p = e / e.sum(axis=1, keepdims=True)
    if top_p < 1.0:
        ids = np.arange(p.shape[1])
        for i in range(p.shape[0]):
            order = np.lexsort((ids, -p[i]))
            ranked = p[i][order]
            before = np.cumsum(ranked) - ranked
            drop = order[before >= top_p]
            p[i, drop] = 0.0
            p[i] /= p[i].sum()
    return p


def depth_tv(logits: np.ndarray, temperature: float = 1.0, top_p: float = 0.7) -> Dict[int, float]:
    """Mean over positions of TV(p_r, p_R) for r = 1 .. R-1.

    logits: [positions][R][V], the readout at depth r in column r - 1."""
    lg = np.asarray(logits)
    n, R, _ = lg.shape
    final = readout_probs(lg[:, R - 1], temperature, top_p)
    out = {}
    for r in range(1, R):
        q = readout_probs(lg[:, r - 1], temperature, top_p)
        out[r] = float(np.maximum(q - final, 0.0).sum(axis=1).mean())
    return out


def fit_envelope(tv: Dict[int, float]) -> Tuple[float, float, float]:
    """(alpha, beta, ratio): the power law beta r^-alpha >= TV_r with the
    smallest largest ratio to TV over the depths (alpha >= 0)."""
    pts = [(math.log(r), math.log(t)) for r, t in sorted(tv.items()) if t > 0.0]
    if not pts:
        raise ValueError("no depth with a positive TV")
    xs = np.array([p[0] for p in pts])
    ys = np.array([p[1] for p in pts])

    def spread(a: float) -> float:
        v = ys + a * xs
        return float(v.max() - v.min())

    cands = {0.0}
    for (x1, y1), (x2, y2) in itertools.combinations(pts, 2):
        if x1 != x2:
            a = (y2 - y1) / (x1 - x2)
            if a > 0.0:
                cands.add(a)
    alpha = min(sorted(cands), key=spread)
    beta = math.exp(float((ys + alpha * xs).max()))
    return alpha, beta, math.exp(spread(alpha))


def steps_bound(d1: float, d2: float, alpha: float, beta: float, R: float) -> float:
    """Theorem 2's bound f(d1, d2) on the expected decode steps per token."""
    return d1 + beta * d2 / d1 ** alpha + 2.0 * beta * R / d2 ** alpha


def closed_form(alpha: float, beta: float, R: float) -> Tuple[float, float, bool]:
    """(d1*, d2*, valid): Theorem 2's minimiser and whether 1 <= d1* < d2* < R."""
    D = alpha * alpha + alpha + 1.0
    ab, tar = alpha * beta, 2.0 * alpha * R
    d1 = math.exp(((alpha + 1.0) * math.log(ab) + math.log(tar)) / D)
    d2 = math.exp((alpha * math.log(ab) + (alpha + 1.0) * math.log(tar)) / D)
    return d1, d2, 1.0 <= d1 < d2 < R


def best_integer_pair(alpha: float, beta: float, R: int) -> Tuple[int, int, float]:
    """Integer 1 <= d1 < d2 < R minimising f (ties to the smaller d1, then d2)."""
    best: Optional[Tuple[int, int, float]] = None
    for d1 in range(1, R - 1):
        for d2 in range(d1 + 1, R):
            v = steps_bound(d1, d2, alpha, beta, R)
            if best is None or v < best[2]:
                best = (d1, d2, v)
    if best is None:
        raise ValueError("R >= 3 is needed for two proposal depths")
    return best


def select_depths(dec, seq: int, ids: Sequence[int], temperature: float = 1.0, top_p: float = 0.7) -> dict:
    """Measure TV per depth from the handle's teacher-forced readouts along
    `ids` (after sequence `seq`'s prefill) and plan (d1, d2).

    The handle's decoding configuration does not matter (readouts are taken
    at every depth); rewind the sequence afterwards to decode it."""
    lg, _ = dec.forced_readout(seq, ids)
    tv = depth_tv(lg, temperature, top_p)
    alpha, beta, ratio = fit_envelope(tv)
    R = lg.shape[1]
    d1s, d2s, valid = closed_form(alpha, beta, R)
    d1, d2, f = best_integer_pair(alpha, beta, R)
    return {"tv": tv, "alpha": alpha, "beta": beta, "envelope_ratio": ratio,
            "closed_form": (d1s, d2s), "closed_form_valid": valid,
            "d1": d1, "d2": d2, "steps_bound": f, "positions": len(ids)}
