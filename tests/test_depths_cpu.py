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


# ---------------------------------------------------------------------------
# online re-planning (OnlinePlanner): TV sums as the decode reports them
# ---------------------------------------------------------------------------
def _sums(a, b, d, n):
    """TV sum over n verifications at depth d under the exact law b d^-a."""
    return b * d ** -a * n


@pytest.mark.parametrize("a,b,R", [(1.08, 0.207, 32), (1.03, 0.175, 16), (0.5, 0.6, 24)])
def test_online_two_depths_recover_the_power_law_and_its_argmin(a, b, R):
    """Two measured depths fix the envelope exactly; the planned pair is the
    oracle's integer argmin of Theorem 2's f."""
    pl = PD.OnlinePlanner(R, min_count=1)
    d1, d2, n = 3, 9, 200
    pl.add(d1, d2, _sums(a, b, d1, n), _sums(a, b, d2, n), n)
    p = pl.plan(d1, d2)
    assert abs(p["alpha"] - a) < 1e-9 and abs(p["beta"] - b) < 1e-9
    i1, i2, fv = OT.integer_argmin(a, b, R)
    assert (p["d1"], p["d2"]) == (i1, i2)
    assert abs(p["steps_bound"] - fv) < 1e-9
    assert p["switch"] == ((i1, i2) != (d1, d2) and fv < 0.95 * OT.f_bound(d1, d2, a, b, R))


def test_online_pools_depths_across_pairs_like_the_oracle_fit():
    """Measurements at several pairs enter one per-depth table; the fit over
    it has the oracle's minimax objective."""
    rng = np.random.default_rng(3)
    pl = PD.OnlinePlanner(32, min_count=1)
    truth = {}
    for d1, d2, n in ((2, 8, 100), (4, 12, 60), (2, 16, 50)):
        t1, t2 = rng.uniform(0.05, 0.6), rng.uniform(0.01, 0.2)
        pl.add(d1, d2, t1 * n, t2 * n, n)
        for d, t in ((d1, t1), (d2, t2)):
            s, m = truth.get(d, (0.0, 0))
            truth[d] = (s + t * n, m + n)
    tv = pl.tv()
    assert sorted(tv) == [2, 4, 8, 12, 16]
    for d, (s, m) in truth.items():
        assert abs(tv[d] - s / m) < 1e-12
    a, b, ratio = PD.fit_envelope(tv)
    oa, ob, oratio = OT.envelope_fit(tv)
    assert abs(ratio - oratio) < 1e-6 * oratio
    for r, t in tv.items():
        assert b * r ** -a >= t * (1 - 1e-12)


def test_online_respects_the_slot_pool_and_the_floor():
    """Pairs whose worst-case tree does not fit are never planned (brute force
    over the oracle's tree simulation); a depth that never disagreed is
    floored at 0.5 / count instead of dropping out of the fit; nothing is
    planned before two depths have min_count verifications; d2 = 0 measures
    one depth."""
    R, a, b = 16, 0.9, 0.5
    limit = 12
    fits = lambda x, y: OT.worst_case_branches(R, x, y) <= limit
    pl = PD.OnlinePlanner(R, fits=fits, min_count=10)
    pl.add(2, 6, _sums(a, b, 2, 9), _sums(a, b, 6, 9), 9)
    assert pl.plan(2, 6) is None
    pl.add(2, 6, _sums(a, b, 2, 1), _sums(a, b, 6, 1), 1)
    p = pl.plan(2, 6)
    best = min(((x, y) for x in range(1, R - 1) for y in range(x + 1, R) if fits(x, y)),
               key=lambda xy: OT.f_bound(xy[0], xy[1], a, b, R))
    assert (p["d1"], p["d2"]) == best
    assert OT.worst_case_branches(R, p["d1"], p["d2"]) <= limit
    z = PD.OnlinePlanner(R, min_count=1)
    z.add(3, 7, 20.0, 0.0, 40)
    assert z.tv() == {3: 0.5, 7: 0.5 / 40}
    one = PD.OnlinePlanner(R, min_count=1)
    one.add(3, 0, 5.0, 0.0, 40)
    assert one.tv() == {3: 5.0 / 40} and one.plan(3, 0) is None


def test_online_keeps_the_pair_within_the_margin():
    R, a, b = 32, 1.08, 0.207
    i1, i2, fv = OT.integer_argmin(a, b, R)
    pl = PD.OnlinePlanner(R, min_count=1, margin=0.05)
    pl.add(i1, i2, _sums(a, b, i1, 100), _sums(a, b, i2, 100), 100)
    assert pl.plan(i1, i2)["switch"] is False
    # a neighbour within 5 % of the optimum is kept as well
    nb = min(((x, y) for x in range(1, R - 1) for y in range(x + 1, R) if (x, y) != (i1, i2)),
             key=lambda xy: OT.f_bound(xy[0], xy[1], a, b, R))
    assert OT.f_bound(*nb, a, b, R) < fv / 0.95
    assert pl.plan(*nb)["switch"] is False
