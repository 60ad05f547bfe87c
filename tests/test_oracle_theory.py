"""Pins for the oracle's theory tools (Theorem 2, envelope, branch growth)."""
import json
import os

import numpy as np
import pytest

from oracle import loopspec as L
from oracle import theory as T

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


@pytest.mark.parametrize("case", GOLD["theorem2"])
def test_theorem2_matches_paper(case):
    d1, d2 = T.optimal_depths(case["alpha"], case["beta"], case["R"])
    assert round(d1, 2) == case["d1"] and round(d2, 2) == case["d2"]


@pytest.mark.parametrize("a,b,R", [(1.03, 0.175, 32), (1.08, 0.207, 32), (0.7, 0.4, 64), (2.0, 0.3, 100)])
def test_theorem2_is_stationary_minimum(a, b, R):
    d1, d2 = T.optimal_depths(a, b, R)
    # gradient by central differences of f itself (independent of f_grad)
    h = 1e-6
    g1 = (T.f_bound(d1 + h, d2, a, b, R) - T.f_bound(d1 - h, d2, a, b, R)) / (2 * h)
    g2 = (T.f_bound(d1, d2 + h, a, b, R) - T.f_bound(d1, d2 - h, a, b, R)) / (2 * h)
    assert abs(g1) < 1e-6 and abs(g2) < 1e-6
    # Hessian: finite differences vs the analytic matrix, and the determinant form of the proof
    H = T.f_hessian(d1, d2, a, b, R)
    e = 1e-4
    fd = np.zeros((2, 2))
    for i in range(2):
        for j in range(2):
            def f(di, dj):
                x = [d1, d2]
                x[i] += di
                x[j] += dj
                return T.f_bound(x[0], x[1], a, b, R)
            fd[i, j] = (f(e, e) - f(e, -e) - f(-e, e) + f(-e, -e)) / (4 * e * e)
    assert np.allclose(H, fd, rtol=1e-4)
    det_proof = a * b * b * d1 ** (-2 * a - 2) * (a * a + a + 1)
    assert np.isclose(np.linalg.det(H), det_proof, rtol=1e-9) and det_proof > 0
    # local minimum against a grid around it
    for dd1 in (-0.05, 0.05):
        for dd2 in (-0.2, 0.2):
            assert T.f_bound(d1 + dd1, d2 + dd2, a, b, R) > T.f_bound(d1, d2, a, b, R)


def _closed_form_valid(a, b, R):
    d1, d2 = T.optimal_depths(a, b, R)
    return 1 <= d1 < d2 < R


@pytest.mark.parametrize("a,b,binding", [
    (1.03, 0.175, "d1 >= 1"),     # the paper's Raven-Llama envelope: d1* reaches 1 last
    (2.0, 0.4, "d2 < R"),         # steep envelope: d2* < R is the last constraint to hold
    (0.4, 10.0, "d1 < d2"),       # shallow, high envelope: d1* < d2* is the last
])
def test_theorem2_validity_condition(a, b, binding):
    """Theorem 2's stationary point is feasible (1 <= d1* < d2* < R) exactly for R
    above the threshold: each of its three terms is the R at which one of the
    constraints becomes tight, so just above it every constraint holds and just
    below it the binding one fails, and at the threshold that one is an equality.
    The three (alpha, beta) pairs make each constraint the binding one in turn."""
    thr = T.validity_threshold(a, b)
    assert _closed_form_valid(a, b, thr * (1 + 1e-6))
    assert not _closed_form_valid(a, b, thr * (1 - 1e-6))
    d1, d2 = T.optimal_depths(a, b, thr)
    slack = {"d1 >= 1": d1 - 1.0, "d1 < d2": d2 / d1 - 1.0, "d2 < R": thr / d2 - 1.0}
    assert abs(slack[binding]) < 1e-9, slack
    assert all(v > 1e-3 for k, v in slack.items() if k != binding), slack


def test_theorem2_valid_at_the_papers_depth():
    a, b = 1.03, 0.175
    assert T.validity_threshold(a, b) < 32 and _closed_form_valid(a, b, 32)


def test_integer_argmin_bruteforce():
    a, b, R = 1.03, 0.175, 32
    best = min(((T.f_bound(i, j, a, b, R), i, j) for i in range(1, R) for j in range(i + 1, R)))
    d1, d2, f = T.integer_argmin(a, b, R)
    assert (d1, d2) == (best[1], best[2]) and np.isclose(f, best[0])


def test_branch_growth_matches_paper():
    g = GOLD["branch_count"]
    s, B = T.branch_growth(g["R"], g["d1"], g["d2"])
    assert B == g["B"]
    assert s[:4] == [1, 1, 1, 1]


@pytest.mark.parametrize("R,d1,d2", [(32, 2, 8), (4, 1, 2), (32, 4, 8), (32, 4, 12), (32, 8, 16),
                                     (16, 2, 4), (12, 3, 6)])
def test_worst_case_tree_equals_recurrence(R, d1, d2):
    assert T.worst_case_branches(R, d1, d2) == T.branch_growth(R, d1, d2)[1]


class _Scripted:
    """Readouts that make every gate open and every first proposal correct:
    argmax p_{d1} = 0, argmax p_{d2} = 1, argmax p_R = 0 for every prefix."""

    def __init__(self, R, d1, d2, V=4):
        self.R, self.d1, self.d2, self.V = R, d1, d2, V

    def root(self):
        return (0,)

    def child(self, node, t):
        return node + (t,)

    def position(self, node):
        return len(node) - 1

    def logits(self, node, r):
        z = np.zeros(self.V)
        z[1 if r == self.d2 else 0] = 1.0
        return z


def test_simulator_tree_reaches_paper_branch_count():
    # Alg. 1 simulator with all gates open and first proposals always accepted:
    # its effective batch peaks at the paper's B = 249 for (R, d1, d2) = (32, 2, 8).
    g = GOLD["branch_count"]
    R, d1, d2 = g["R"], g["d1"], g["d2"]
    res = L.decode_loopspec(_Scripted(R, d1, d2), R, d1, d2, 40, L.Sampler(0.0))
    assert max(res.M) == g["B"]
    assert res.n_acc1 == res.n_decode
    assert res.gate_open == res.gate_eval > 0


def test_envelope_fit_recovers_power_law():
    a0, b0 = 1.03, 0.175
    tv = {r: b0 * r ** -a0 for r in range(1, 32)}
    a, b, obj = T.envelope_fit(tv)
    assert abs(a - a0) < 1e-6 and abs(b - b0) < 1e-6 and abs(obj - 1) < 1e-9


def test_envelope_fit_is_upper_envelope_and_optimal():
    rng = np.random.default_rng(0)
    tv = {r: 0.3 * r ** -0.9 * np.exp(0.2 * rng.standard_normal()) for r in range(1, 11)}
    a, b, obj = T.envelope_fit(tv)
    assert all(b * r ** -a >= tv[r] * (1 - 1e-12) for r in tv)
    # brute force over alpha: no alpha gives a smaller max ratio
    for aa in np.linspace(0.01, 4, 2000):
        bb = max(tv[r] * r ** aa for r in tv)
        assert max(bb * r ** -aa / tv[r] for r in tv) >= obj * (1 - 1e-6)


def test_gamma_bound():
    # gamma <= R/d1 with equality when every token is a first-proposal accept
    assert T.gamma(10, 10, 0, 32, 2, 8) == 16
    assert T.gamma(10, 3, 4, 32, 2, 8) < 16
