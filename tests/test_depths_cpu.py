"""The library's proposal-depth planner (host side) against the paper's
printed Theorem 2 values, exact power laws and the oracle's own analysis."""
import json
import os

import numpy as np
import pytest

from oracle import dist as OD
from oracle import theory as OT
from paper_2609_17184_amd import depths as PD

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


@pytest.mark.parametrize("case", GOLD["theorem2"])
def test_closed_form_matches_paper(case):
    d1, d2, valid = PD.closed_form(case["alpha"], case["beta"], case["R"])
    assert valid
    assert round(d1, 2) == case["d1"] and round(d2, 2) == case["d2"]


def test_closed_form_is_the_stationary_point():
    rng = np.random.default_rng(0)
    for _ in range(100):
        a, b, R = rng.uniform(0.3, 2.0), rng.uniform(0.05, 0.9), rng.uniform(20, 80)
        d1, d2, _ = PD.closed_form(a, b, R)
        g1, g2 = OT.f_grad(d1, d2, a, b, R)
        assert abs(g1) < 1e-9 and abs(g2) < 1e-9


def test_envelope_recovers_an_exact_power_law():
    for a, b in ((1.03, 0.175), (0.4, 0.9), (2.5, 0.05)):
        tv = {r: b * r ** -a for r in range(1, 17)}
        fa, fb, ratio = PD.fit_envelope(tv)
        assert abs(fa - a) < 1e-9 and abs(fb - b) < 1e-12 and abs(ratio - 1.0) < 1e-12


def test_envelope_dominates_and_matches_oracle_objective():
    rng = np.random.default_rng(1)
    for _ in range(300):
        tv = {r: float(rng.uniform(0.005, 1.0)) for r in range(1, int(rng.integers(3, 33)))}
        a, b, ratio = PD.fit_envelope(tv)
        phi = {r: b * r ** -a for r in tv}
        assert all(phi[r] >= tv[r] * (1 - 1e-12) for r in tv)
        assert np.isclose(ratio, max(phi[r] / tv[r] for r in tv))
        # the oracle's golden-section fit reaches the same optimum (up to its tolerance)
        assert ratio <= OT.envelope_fit(tv)[2] * (1 + 1e-7)


def test_best_integer_pair_is_the_grid_argmin():
    rng = np.random.default_rng(2)
    for _ in range(200):
        a, b, R = rng.uniform(0.2, 2.5), rng.uniform(0.02, 1.0), int(rng.integers(3, 40))
        d1, d2, f = PD.best_integer_pair(a, b, R)
        o1, o2, of = OT.integer_argmin(a, b, R)
        assert (d1, d2) == (o1, o2) and np.isclose(f, of)


@pytest.mark.parametrize("T,top_p", [(1.0, 1.0), (1.0, 0.7), (0.7, 0.95), (0.0, 1.0)])
def test_readout_probs_and_tv_match_the_oracle(T, top_p):
    rng = np.random.default_rng(3)
    lg = rng.normal(size=(6, 4, 40)) * 2.0
    lg[2, 1, 7] = lg[2, 1, 8]                     # an exact tie inside one row
    got = PD.depth_tv(lg, T, top_p)
    for r in range(1, 4):
        ref = np.mean([OD.tv(OD.readout_dist(lg[t, r - 1], T, top_p), OD.readout_dist(lg[t, 3], T, top_p))
                       for t in range(6)])
        assert abs(got[r] - ref) < 1e-12
