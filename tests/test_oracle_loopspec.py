"""Pins for the Alg. 1 simulator: greedy losslessness, step-count identities,
gamma bounds, degenerate models, and sampling losslessness (chi-square)."""
import itertools

import numpy as np
import pytest
from scipy import stats

import synth
from oracle import dist as D
from oracle import loopspec as L
from oracle import model as M
from oracle import theory as T


class HashReadouts:
    """Synthetic readouts: logits are a seeded function of (prefix, depth); early
    depths are the target logits plus noise shrinking with depth."""

    def __init__(self, V=6, R=4, noise=1.5, seed=0, decay=1.0):
        self.V, self.R, self.noise, self.seed, self.decay = V, R, noise, seed, decay

    def root(self):
        return (0, 1)

    def child(self, node, t):
        return node + (int(t),)

    def position(self, node):
        return len(node) - 1

    def logits(self, node, r):
        g = np.random.default_rng([self.seed, len(node)] + list(node))
        base = 1.5 * g.standard_normal(self.V)
        pert = g.standard_normal((self.R, self.V))
        return base + self.noise * pert[r - 1] * (1 - r / self.R) ** self.decay


DEPTHS = [(4, 1, 2), (4, 1, 3), (4, 2, 3), (4, 1, 0), (4, 2, 0), (4, 3, 0), (8, 2, 6), (8, 3, 5)]


@pytest.mark.parametrize("R,d1,d2", DEPTHS)
def test_greedy_lossless_synthetic(R, d1, d2):
    for seed in range(4):
        prov = HashReadouts(V=7, R=R, seed=seed)
        v = L.decode_vanilla(prov, R, 40, L.Sampler(0.0))
        s = L.decode_loopspec(prov, R, d1, d2, 40, L.Sampler(0.0))
        assert s.tokens == v.tokens
        assert v.steps == 39 * R
        # step identity: the first root needs R steps; after a commit from source
        # 1 / 2 / restart the next root needs d1 / d2 / R more steps
        cost = {1: d1, 2: d2, 0: R}
        assert s.steps == R + sum(cost[c] for c in s.sources[:-1])
        assert s.gamma(R, d1, d2) <= R / d1 + 1e-12
        assert s.n_acc1 + s.n_acc2 + s.n_restart == s.n_decode == 39
        assert max(s.M) <= T.worst_case_branches(R, d1, d2) or d1 * 0
        if d2 == 0:
            assert s.n_acc2 == 0 and s.gate_eval == 0


@pytest.mark.parametrize("R,d1,d2", [(4, 1, 2), (4, 2, 3), (4, 1, 0)])
def test_greedy_lossless_tiny_model(R, d1, d2):
    spec = synth.preset("micro")
    lm = M.LoopedLM(spec, synth.make_weights(spec, seed=3))
    prov = L.ModelReadouts(lm, synth.make_prompt(spec.vocab, 5))
    v = L.decode_vanilla(prov, R, 30, L.Sampler(0.0))
    s = L.decode_loopspec(prov, R, d1, d2, 30, L.Sampler(0.0))
    assert s.tokens == v.tokens
    assert s.n_restart > 0 or s.n_acc2 > 0      # this model does reject drafts


def test_alpha_zero_accepts_everything():
    spec = synth.preset("micro", alpha=0.0)
    lm = M.LoopedLM(spec, synth.make_weights(spec))
    prov = L.ModelReadouts(lm, [1, 2, 3])
    R, d1, d2, N = 4, 1, 2, 20
    s = L.decode_loopspec(prov, R, d1, d2, N, L.Sampler(0.0))
    assert s.n_acc1 == N - 1 and s.gate_open == 0
    assert s.gamma(R, d1, d2) == R / d1
    assert s.steps == R + (N - 2) * d1
    assert max(s.M) == R // d1          # the chain root ... newest child


def test_adversarial_restarts_every_token():
    class Adv(HashReadouts):
        def logits(self, node, r):
            z = np.zeros(self.V)
            z[(len(node) + (0 if r == self.R else 1 + r)) % self.V] = 1
            return z
    R, N = 4, 15
    s = L.decode_loopspec(Adv(V=9, R=R), R, 1, 2, N, L.Sampler(0.0))
    assert s.n_restart == N - 1 and s.steps == (N - 1) * R


def _exact_joint(prov, T, top_p, R):
    root = prov.root()
    p1 = D.readout_dist(prov.logits(root, R), T, top_p)
    J = np.zeros((prov.V, prov.V))
    for a in range(prov.V):
        if p1[a] == 0:
            continue
        p2 = D.readout_dist(prov.logits(prov.child(root, a), R), T, top_p)
        J[a] = p1[a] * p2
    return J


@pytest.mark.parametrize("R,d1,d2,top_p", [(4, 1, 2, 1.0), (4, 2, 3, 0.9), (4, 1, 0, 1.0)])
def test_sampling_lossless_chi_square(R, d1, d2, top_p):
    prov = HashReadouts(V=5, R=R, noise=2.0, seed=9)
    J = _exact_joint(prov, 1.0, top_p, R)
    n = 3000
    C = np.zeros_like(J)
    for s in range(n):
        res = L.decode_loopspec(prov, R, d1, d2, 2, L.Sampler(1.0, top_p, seed=100 + s))
        C[res.tokens[0], res.tokens[1]] += 1
    m = J.reshape(-1) > 0
    assert C.reshape(-1)[~m].sum() == 0
    assert stats.chisquare(C.reshape(-1)[m], J.reshape(-1)[m] * n).pvalue > 1e-3


def test_sampling_capacity_cap_is_lossless():
    R, d1, d2 = 4, 1, 2
    prov = HashReadouts(V=4, R=R, noise=2.5, seed=4)
    J = _exact_joint(prov, 1.0, 1.0, R)
    n = 3000
    C = np.zeros_like(J)
    for s in range(n):
        res = L.decode_loopspec(prov, R, d1, d2, 2, L.Sampler(1.0, seed=7000 + s), max_branches=2)
        C[res.tokens[0], res.tokens[1]] += 1
    m = J.reshape(-1) > 0
    assert stats.chisquare(C.reshape(-1)[m], J.reshape(-1)[m] * n).pvalue > 1e-3


def test_sampling_third_token_marginal():
    R, d1, d2 = 4, 1, 2
    prov = HashReadouts(V=4, R=R, noise=2.0, seed=21)
    root = prov.root()
    law = np.zeros(4)
    p1 = D.readout_dist(prov.logits(root, R), 1.0)
    for a, b in itertools.product(range(4), range(4)):
        pa = prov.child(root, a)
        p2 = D.readout_dist(prov.logits(pa, R), 1.0)
        law += p1[a] * p2[b] * D.readout_dist(prov.logits(prov.child(pa, b), R), 1.0)
    n = 3000
    c = np.zeros(4)
    for s in range(n):
        c[L.decode_loopspec(prov, R, d1, d2, 3, L.Sampler(1.0, seed=50000 + s)).tokens[2]] += 1
    assert stats.chisquare(c, law * n).pvalue > 1e-3


# ---------------------------------------------------------------------------
# switching (d1, d2) while decoding (depth re-planning) and the TV records
# ---------------------------------------------------------------------------
SWITCHES = [{5: (3, 5), 12: (1, 0), 20: (2, 6)}, {2: (6, 7), 9: (1, 2), 10: (4, 0)}]


@pytest.mark.parametrize("sw", SWITCHES)
def test_greedy_lossless_with_switches(sw):
    """Greedy tokens equal vanilla decoding across pair switches; the step
    count follows the cost of each commit (d1 / d2 / R after source 1 / 2 /
    restart), except right after a switch, where the root continues from its
    depth if it is below the new d1 and from depth 0 otherwise."""
    R, N = 8, 30
    for seed in range(4):
        prov = HashReadouts(V=7, R=R, seed=seed)
        v = L.decode_vanilla(prov, R, N, L.Sampler(0.0))
        s = L.decode_loopspec(prov, R, 2, 4, N, L.Sampler(0.0), switches=sw)
        assert s.tokens == v.tokens
        d1, d2, steps = 2, 4, R
        for i, src in enumerate(s.sources[:-1]):
            cost = {1: d1, 2: d2, 0: R}[src]
            if i + 2 in sw:                  # the commit that brings the count to i + 2
                d1, d2 = sw[i + 2]
                r = R - cost
                cost = R - (r if r < d1 else 0)
            steps += cost
        assert s.steps == steps
        # one-hot readouts: TV is the argmax mismatch, and the first proposal
        # is accepted exactly when it matches the target
        assert set(s.tv1) <= {0.0, 1.0} and set(s.tv2) <= {0.0, 1.0}
        assert s.n_acc1 == sum(t == 0.0 for t in s.tv1)
        for src, t1, t2 in zip(s.sources, s.tv1, s.tv2):
            if src == 2:
                assert t1 == 1.0 and t2 == 0.0


def test_sampling_lossless_with_switch_chi_square():
    """The third token's marginal equals the target law when the pair changes
    after the second commit (a root at depth >= the new d1 restarts)."""
    R = 4
    prov = HashReadouts(V=4, R=R, noise=2.0, seed=21)
    root = prov.root()
    law = np.zeros(4)
    p1 = D.readout_dist(prov.logits(root, R), 1.0)
    for a, b in itertools.product(range(4), range(4)):
        pa = prov.child(root, a)
        p2 = D.readout_dist(prov.logits(pa, R), 1.0)
        law += p1[a] * p2[b] * D.readout_dist(prov.logits(prov.child(pa, b), R), 1.0)
    n = 3000
    c = np.zeros(4)
    for s in range(n):
        res = L.decode_loopspec(prov, R, 2, 3, 3, L.Sampler(1.0, seed=80000 + s), switches={2: (1, 2)})
        c[res.tokens[2]] += 1
    assert stats.chisquare(c, law * n).pvalue > 1e-3


def test_sampling_tv_record_is_one_minus_the_acceptance_rate():
    """Speculative sampling accepts a draft x ~ q against p with probability
    sum_x min(p, q) = 1 - TV(p, q): given the history, each verification's
    first acceptance is a Bernoulli(1 - tv1) draw, so the acceptance count
    minus the sum of (1 - tv1) is a martingale (z-score below 4)."""
    R, d1, d2 = 4, 1, 2
    prov = HashReadouts(V=6, R=R, noise=1.8, seed=31)
    dev = var = 0.0
    for s in range(300):
        res = L.decode_loopspec(prov, R, d1, d2, 12, L.Sampler(1.0, seed=90000 + s))
        for src, t in zip(res.sources, res.tv1):
            dev += (src == 1) - (1.0 - t)
            var += t * (1.0 - t)
    assert var > 50
    assert abs(dev) / np.sqrt(var) < 4.0
