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

Online (OnlinePlanner, decode_adaptive): the decode itself sums
TV(p_R, p_d1) and TV(p_R, p_d2) over its verifications; between decode calls
the planner folds them into per-depth means, re-fits the envelope and moves
the handle to the pair that minimises f (loopspec_set_depths), so the
depths follow the text being generated without a calibration pass.

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


# ---------------------------------------------------------------------------
# online re-planning while decoding
# ---------------------------------------------------------------------------
class OnlinePlanner:
    """Per-depth TV estimates from the decode's own verifications, and the
    proposal pair they imply.

    Every verification in Alg. 1 holds the root's final readout p_R next to
    its readouts at d1 and d2; the library sums TV(p_R, p_d1) and
    TV(p_R, p_d2) over verifications (loopspec_stats tv_d1, tv_d2, tv_count,
    in units of 2^-32).  TV at a depth is a property of the model along the
    decoded sequence, not of the pair that measured it, so the sums are kept
    per depth across pairs and the envelope is fitted over every depth seen
    (the minimax rule of fit_envelope; through two points it is the power law
    through both).  A depth whose measured TV is zero is floored at
    0.5 / count (a finite sample cannot resolve a smaller distance).  The
    pair minimising Theorem 2's f among those `fits` allows is
    adopted when it lowers f by more than `margin` (a switch drops the
    speculative tree, so small gains are not worth it)."""

    def __init__(self, R: int, fits=None, margin: float = 0.05, min_count: int = 16):
        self.R = int(R)
        self.fits = fits if fits is not None else (lambda d1, d2: True)
        self.margin = float(margin)
        self.min_count = int(min_count)
        self.sums: Dict[int, list] = {}

    def add(self, d1: int, d2: int, tv1: float, tv2: float, count: int) -> None:
        """Fold in `count` verifications at pair (d1, d2) whose TV sums are
        tv1 (depth d1) and tv2 (depth d2; ignored when d2 = 0)."""
        if count <= 0:
            return
        for d, v in ((d1, tv1), (d2, tv2)):
            if d > 0:
                acc = self.sums.setdefault(int(d), [0.0, 0])
                acc[0] += float(v)
                acc[1] += int(count)

    def tv(self) -> Dict[int, float]:
        """Mean TV per depth with at least min_count verifications."""
        out = {}
        for d, (s, n) in sorted(self.sums.items()):
            if n >= self.min_count:
                out[d] = max(s / n, 0.5 / n)
        return out

    def plan(self, d1: int, d2: int) -> Optional[dict]:
        """The envelope over the measured depths and the pair to decode with
        next (None until two depths are measured): the best pair that `fits`
        allows now, and under "unrestricted" the best of all pairs (for the
        next sequence, when the handle only allows some pairs mid-sequence)."""
        tv = self.tv()
        if len(tv) < 2:
            return None
        alpha, beta, ratio = fit_envelope(tv)
        best = anywhere = None
        for a in range(1, self.R - 1):
            for b in range(a + 1, self.R):
                v = steps_bound(a, b, alpha, beta, self.R)
                if anywhere is None or v < anywhere[2]:
                    anywhere = (a, b, v)
                if self.fits(a, b) and (best is None or v < best[2]):
                    best = (a, b, v)
        cur = steps_bound(d1, d2, alpha, beta, self.R) if d2 > 0 else math.inf
        out = {"tv": tv, "alpha": alpha, "beta": beta, "envelope_ratio": ratio, "current_bound": cur,
               "unrestricted": anywhere, "d1": d1, "d2": d2, "steps_bound": cur, "switch": False}
        if best is not None:
            out.update(d1=best[0], d2=best[1], steps_bound=best[2],
                       switch=(best[0], best[1]) != (d1, d2) and best[2] < (1.0 - self.margin) * cur)
        return out


def decode_adaptive(dec, n_tokens: int, every: int = 32, margin: float = 0.05, min_count: int = 16):
    """Decode n_tokens for every prefilled sequence in segments of `every`
    tokens, re-planning (d1, d2) after each segment from the TV statistics
    gathered so far (OnlinePlanner) and switching the handle's pair when the
    plan says so.  Only pairs the handle accepts now are planned (slot pool;
    on models with coda blocks, readout depths whose coda caches cover the
    generated positions).  Returns (tokens [max_seqs][n_tokens], one plan
    record per segment)."""
    planner = OnlinePlanner(dec.R, lambda a, b: dec.can_set_depths(a, b) == 0, margin, min_count)
    out = np.full((dec.max_seqs, n_tokens), -1, np.int32)
    log = []
    s0 = dec.stats()
    done = 0
    while done < n_tokens:
        k = min(every, n_tokens - done)
        out[:, done:done + k] = dec.decode(k)
        done += k
        s1 = dec.stats()
        scale = 2.0 ** -32
        planner.add(dec.d1, dec.d2, (s1["tv_d1"] - s0["tv_d1"]) * scale, (s1["tv_d2"] - s0["tv_d2"]) * scale,
                    s1["tv_count"] - s0["tv_count"])
        s0 = s1
        plan = planner.plan(dec.d1, dec.d2)
        rec = {"tokens": done, "d1": dec.d1, "d2": dec.d2, "plan": plan}
        if plan is not None and plan["switch"] and done < n_tokens:
            dec.set_depths(plan["d1"], plan["d2"])
            rec["switched_to"] = (plan["d1"], plan["d2"])
        log.append(rec)
    return out, log
