"""Pins for the oracle's proposal-depth analysis (teacher-forced TV, envelope,
Theorem 2 prediction)."""
import numpy as np
import pytest

import synth
from oracle import depths as DP
from oracle.model import LoopedLM


def _lm(name="micro", **kw):
    spec = synth.preset(name, **kw)
    return LoopedLM(spec, synth.make_weights(spec))


def test_alpha_zero_gives_zero_tv():
    # with no residual branches every depth holds the embedding: p_r = p_R
    lm = _lm(alpha=0.0)
    tv = DP.teacher_forced_tv(lm, synth.make_prompt(lm.spec.vocab, 12), 1.0, 0.7)
    assert all(v == 0.0 for v in tv.values())


@pytest.mark.parametrize("name,top_p", [("micro", 0.7), ("micro", 1.0), ("small_raven", 0.9)])
def test_tv_matches_incremental_decoding(name, top_p):
    # the analysis uses one cache-free forward; recompute every position with
    # the cached incremental path and TV as half the L1 distance
    lm = _lm(name)
    R = lm.spec.R
    toks = [int(t) for t in synth.make_prompt(lm.spec.vocab, 9)]
    got = DP.teacher_forced_tv(lm, toks, 1.0, top_p)
    ref = {r: [] for r in range(1, R + 1)}
    node = lm.prefill(toks[:1])
    for t in range(len(toks)):
        if t:
            node = lm.extend(node, toks[t])
        z = {r: lm.logits(node, r) for r in range(1, R + 1)}
        pR = _dist(z[R], top_p)
        for r in range(1, R + 1):
            ref[r].append(0.5 * np.abs(_dist(z[r], top_p) - pR).sum())
    for r in range(1, R + 1):
        assert got[r] == pytest.approx(np.mean(ref[r]), abs=1e-9)
    assert got[R] == 0.0


def _dist(z, top_p):
    # softmax + nucleus by sorting, written independently of oracle.dist
    p = np.exp(z - z.max())
    p /= p.sum()
    idx = sorted(range(p.size), key=lambda i: (-p[i], i))
    keep, acc = np.zeros(p.size, bool), 0.0
    for i in idx:
        if acc >= top_p:
            break
        keep[i] = True
        acc += p[i]
    q = np.where(keep, p, 0.0)
    return q / q.sum()


def test_tiny_nucleus_is_argmax_mismatch_rate():
    # a nucleus that keeps only the top token makes TV the rate of argmax mismatches
    lm = _lm()
    R = lm.spec.R
    toks = synth.make_prompt(lm.spec.vocab, 16)
    got = DP.teacher_forced_tv(lm, toks, 1.0, 1e-12)
    logits = lm.forward_full(list(toks))
    for r in range(1, R):
        miss = np.mean(np.argmax(logits[r], 1) != np.argmax(logits[R], 1))
        assert got[r] == pytest.approx(miss, abs=1e-12)


@pytest.mark.parametrize("a,b,R", [(1.03, 0.175, 32), (0.5, 0.3, 4), (2.0, 0.9, 8)])
def test_exact_power_law_is_recovered(a, b, R):
    tv = {r: b * r ** -a for r in range(1, R)}
    tv[R] = 0.0
    res = DP.predict(tv, R)
    assert res["envelope"]["alpha"] == pytest.approx(a, rel=1e-6)
    assert res["envelope"]["beta"] == pytest.approx(b, rel=1e-5)
    assert res["envelope"]["max_ratio"] == pytest.approx(1.0, abs=1e-6)
    # the integer argmin is the smallest bound f(d1, d2) = d1 + b d1^-a d2 + 2 b d2^-a R
    best = min(((d1 + b * d1 ** -a * d2 + 2 * b * d2 ** -a * R, d1, d2)
                for d1 in range(1, R - 1) for d2 in range(d1 + 1, R)))
    assert (res["integer_argmin"]["d1"], res["integer_argmin"]["d2"]) == best[1:]


def test_paper_calibration_point():
    # with the paper's envelope (1.03, 0.175) at R = 32 the closed form is
    # (1.26, 8.85) and R = 32 lies above the validity threshold
    tv = {r: 0.175 * r ** -1.03 for r in range(1, 32)}
    res = DP.predict(tv, 32)
    assert round(res["closed_form"]["d1"], 2) == 1.26 and round(res["closed_form"]["d2"], 2) == 8.85
    assert res["closed_form"]["valid"]
