"""Proposal-depth analysis: teacher-forced TV between readout depths, the
power-law envelope over it, and Theorem 2's prediction of (d1, d2).

TEST INFRASTRUCTURE: part of the CPU oracle.  Only tests/, the smoke check and
the benchmark's CPU-baseline leg may import it.  Run as a script it prints one
JSON object per model (the prediction that the measured depth sweeps are set
against):

    python -m oracle.depths --model ouro14 --alpha 0.3 --positions 64

Sources (LoopSpec paper):
  * Sec. 4.1, Observation: the distance TV(p_r, p_R) between an intermediate
    readout and the final one shrinks with depth and is bounded by a power law
    phi(r) = beta r^-alpha fitted over the depths;
  * Theorem 2: with that envelope the expected number of decode steps per
    committed token is at most f(d1, d2) (theory.f_bound), minimised in closed
    form (theory.optimal_depths) when R exceeds theory.validity_threshold.

Readings where the paper is silent or specific to its own setting:
  * TV_r is averaged over teacher-forced positions: the sequence is the
    synthetic prompt, and position t compares the depth-r and depth-R
    readouts of the prefix x_{<=t} (the distributions for x_{t+1});
  * the distributions use temperature 1 and top-p 0.7, as the paper's
    envelope measurement does; every depth r = 1..R-1 enters the fit
    (TV_R = 0 carries no information);
  * when R is not above the validity threshold the closed form is reported but
    flagged, and the integer argmin of f over 1 <= d1 < d2 < R is the
    prediction that is compared with a measured sweep.
"""
from __future__ import annotations

import argparse
import json
from typing import Dict, Sequence

import numpy as np

import synth
from . import dist as D
from . import theory as TH
from .model import LoopedLM


def teacher_forced_tv(lm: LoopedLM, tokens: Sequence[int], temperature: float = 1.0,
                      top_p: float = 0.7, first: int = 0) -> Dict[int, float]:
    """TV_r = mean over positions t >= first of TV(p_r(.|x_<=t), p_R(.|x_<=t)),
    for r = 1..R (so TV_R = 0), from one cache-free forward over `tokens`."""
    R = lm.spec.R
    logits = lm.forward_full(list(tokens))
    T = len(tokens)
    out: Dict[int, float] = {}
    final = [D.readout_dist(logits[R][t], temperature, top_p) for t in range(first, T)]
    for r in range(1, R + 1):
        tv = [D.tv(D.readout_dist(logits[r][t], temperature, top_p), final[t - first])
              for t in range(first, T)]
        out[r] = float(np.mean(tv))
    return out


def predict(tv: Dict[int, float], R: int) -> dict:
    """Envelope fit over TV_1..TV_{R-1}, Theorem 2's closed form and validity,
    and the integer argmin of f with f at every grid point."""
    fit_tv = {r: v for r, v in tv.items() if 1 <= r < R and v > 0}
    res: dict = {"tv": {str(r): tv[r] for r in sorted(tv)}}
    if len(fit_tv) < 2:
        res["envelope"] = None
        return res
    a, beta, ratio = TH.envelope_fit(fit_tv)
    d1c, d2c = TH.optimal_depths(a, beta, R)
    thr = TH.validity_threshold(a, beta)
    i1, i2, fv = TH.integer_argmin(a, beta, R)
    res["envelope"] = {"alpha": a, "beta": beta, "max_ratio": ratio}
    res["closed_form"] = {"d1": d1c, "d2": d2c, "valid": R > thr, "R_threshold": thr}
    res["integer_argmin"] = {"d1": i1, "d2": i2, "f": fv}
    res["f"] = {f"{d1},{d2}": TH.f_bound(d1, d2, a, beta, R)
                for d1 in range(1, R - 1) for d2 in range(d1 + 1, R)}
    return res


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--model", default="ouro14", choices=sorted(synth.PRESETS))
    ap.add_argument("--alpha", type=float, nargs="+", default=[0.3],
                    help="residual-branch scale(s) of the synthetic model")
    ap.add_argument("--positions", type=int, default=64, help="teacher-forced prompt length")
    ap.add_argument("--temperature", type=float, default=1.0)
    ap.add_argument("--top-p", type=float, default=0.7)
    a = ap.parse_args(argv)
    for alpha in a.alpha:
        spec = synth.preset(a.model, alpha=alpha)
        # keep fp64 copies of the weights only when they fit comfortably in memory
        lm = LoopedLM(spec, synth.make_weights(spec), cache64=spec.n_params() * 8 < (16 << 30))
        prompt = synth.make_prompt(spec.vocab, a.positions)
        tv = teacher_forced_tv(lm, prompt, a.temperature, a.top_p)
        res = {"model": a.model, "alpha": alpha, "R": spec.R, "positions": a.positions,
               "temperature": a.temperature, "top_p": a.top_p}
        res.update(predict(tv, spec.R))
        print(json.dumps(res), flush=True)
        del lm
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
