"""Pins for cascade verification: losslessness by exact enumeration, Theorem 1,
Lemma 1, acceptance = 1 - TV, greedy reduction, and a Monte Carlo of the
oracle's own Verify + gate + draws against the exact law."""
import numpy as np
import pytest
from scipy import stats

from oracle import dist as D
from oracle import loopspec as L
from oracle import theory as T


def _rand_dists(rng, V, k=3, sparsity=0.3):
    out = []
    for _ in range(k):
        p = rng.dirichlet(np.ones(V) * 0.7)
        p[rng.random(V) < sparsity] = 0
        if p.sum() == 0:
            p[rng.integers(V)] = 1
        out.append(p / p.sum())
    return out


@pytest.mark.parametrize("gate", ["gated", "open", "closed"])
def test_cascade_is_lossless_exact(gate):
    rng = np.random.default_rng(1)
    for _ in range(300):
        V = int(rng.integers(2, 9))
        p, q1, q2t = _rand_dists(rng, V)
        law, a1, a2, rs = T.cascade_law(p, q1, q2t, gate)
        assert np.allclose(law, p, atol=1e-13), (p, q1, q2t)
        assert np.isclose(a1 + a2 + rs, 1.0)


def test_accept1_is_one_minus_tv():
    rng = np.random.default_rng(2)
    for _ in range(200):
        p, q1, q2t = _rand_dists(rng, 6)
        _, a1, _, _ = T.cascade_law(p, q1, q2t)
        assert np.isclose(a1, 1 - D.tv(p, q1))


def test_theorem1_restart_bounds_and_closed_form():
    rng = np.random.default_rng(3)
    for _ in range(500):
        p, q1, q2t = _rand_dists(rng, int(rng.integers(2, 9)), sparsity=0.1)
        eps2 = D.tv(q2t, p)
        _, _, _, r_gated = T.cascade_law(p, q1, q2t, "gated")
        _, _, _, r_open = T.cascade_law(p, q1, q2t, "open")
        assert r_gated <= 2 * eps2 + 1e-12
        assert r_open <= eps2 + 1e-12
        # closed form: sum_{x in G} [q1-p]_+(x) TV(rho1, q2) + sum_{x not in G} [q1-p]_+(x)
        rho1, _ = D.residual(p, q1)
        q2, _ = D.residual(q2t, q1)
        G = q2t < q1
        qp = D.positive_part(q1, p)
        closed = qp[G].sum() * D.tv(rho1, q2) + qp[~G].sum()
        assert np.isclose(r_gated, closed, atol=1e-13)


def test_lemma1():
    rng = np.random.default_rng(4)
    n = 0
    for _ in range(2000):
        p, q1, q2t = _rand_dists(rng, int(rng.integers(2, 9)), sparsity=0.0)
        e1, e2 = D.tv(q1, p), D.tv(q2t, p)
        if e1 <= 0 or np.allclose(q1, q2t):
            continue
        nu1, _ = D.residual(q2t, q1)
        nu2, _ = D.residual(p, q1)
        assert D.tv(nu1, nu2) <= e2 / e1 + 1e-12
        n += 1
    assert n > 1000


class _Fixed:
    """A one-branch tree whose readouts at d1, d2, R are fixed distributions."""

    def __init__(self, p, q1, q2t, d1, d2, R):
        self.d = {d1: q1, d2: q2t, R: p}
        self.V = p.size

    def root(self):
        return ()

    def child(self, node, t):
        return node + (t,)

    def position(self, node):
        return len(node) + 10


class _S(L.Sampler):
    """Sampler whose readout 'dist' passes fixed distributions straight through."""

    def dist(self, w):
        return w


def test_oracle_verify_monte_carlo_matches_exact_law():
    rng = np.random.default_rng(5)
    p, q1, q2t = _rand_dists(rng, 5, sparsity=0.0)
    q2t = 0.5 * q2t + 0.5 * p              # a deeper readout closer to the target
    law, a1, a2, rs = T.cascade_law(p, q1, q2t, "gated")
    R, d1, d2 = 4, 1, 2
    prov = _Fixed(p, q1, q2t, d1, d2, R)

    class Prov(_Fixed):
        def logits(self, node, r):
            return self.d[r] if len(node) == 1 else p   # deeper prefixes: irrelevant

    prov = Prov(p, q1, q2t, d1, d2, R)
    n = 6000
    counts = np.zeros(5)
    src = np.zeros(3)
    for s in range(n):
        res = L.decode_loopspec(prov, R, d1, d2, 2, _S(1.0, 1.0, seed=11, seq=s))
        counts[res.tokens[1]] += 1
        src[res.sources[0]] += 1
    # the prefill token is drawn from p_R at the root; the first Verify commit follows law == p
    assert stats.chisquare(counts, law * n).pvalue > 1e-3
    exp_src = np.array([rs, a1, a2]) * n
    assert stats.chisquare(src, exp_src).pvalue > 1e-3


def test_greedy_reduction():
    # one-hot readouts: the cascade is argmax comparisons
    V = 6
    e = np.eye(V)
    for t in range(V):
        for a1 in range(V):
            for a2 in range(V):
                law, acc1, acc2, rs = T.cascade_law(e[t], e[a1], e[a2], "gated")
                assert law.argmax() == t and law.max() == 1
                if a1 == t:
                    assert acc1 == 1
                elif a2 != a1 and a2 == t:      # gate open (argmax q2~ != x1) and match
                    assert acc2 == 1
                else:
                    assert rs == 1


# ---- second-proposal variants of the ablation (Ablation Study, Table 3) ----------

@pytest.mark.parametrize("variant", [L.SP_GATED, L.SP_RESIDUAL, L.SP_NAIVE])
def test_second_proposal_variants_lossless_exact(variant):
    rng = np.random.default_rng(21 + variant)
    for _ in range(300):
        V = int(rng.integers(2, 9))
        p, q1, q2t = _rand_dists(rng, V)
        law, a1, a2, rs = T.cascade_law_variant(p, q1, q2t, variant)
        assert np.allclose(law, p, atol=1e-13), (variant, p, q1, q2t)
        assert np.isclose(a1 + a2 + rs, 1.0)


def test_gated_variant_is_the_gated_cascade():
    rng = np.random.default_rng(24)
    for _ in range(200):
        p, q1, q2t = _rand_dists(rng, int(rng.integers(2, 9)))
        got = T.cascade_law_variant(p, q1, q2t, L.SP_GATED)
        ref = T.cascade_law(p, q1, q2t, "gated")
        assert np.allclose(got[0], ref[0]) and np.allclose(got[1:], ref[1:])


@pytest.mark.parametrize("variant", [L.SP_RESIDUAL, L.SP_NAIVE])
def test_masked_second_proposal_differs_from_first(variant):
    rng = np.random.default_rng(25 + variant)
    for _ in range(300):
        V = int(rng.integers(2, 9))
        _, q1, q2t = _rand_dists(rng, V)
        for x1 in range(V):
            q2, _ = L.second_proposal(q1, q2t, x1, variant)
            if q2 is None:          # nothing left once x1 is masked out
                base = q2t if variant == L.SP_NAIVE else D.residual(q2t, q1)[0]
                assert np.all(np.delete(base, x1) == 0)
                continue
            assert q2[x1] == 0 and np.isclose(q2.sum(), 1.0) and np.all(q2 >= 0)


def test_residual_variant_needs_no_mask_where_the_gate_opens():
    # where q2~(x1) < q1(x1), (q2~ (-) q1)(x1) is already zero: masking changes nothing
    rng = np.random.default_rng(27)
    n = 0
    for _ in range(300):
        V = int(rng.integers(2, 9))
        _, q1, q2t = _rand_dists(rng, V, sparsity=0.0)
        for x1 in range(V):
            if q2t[x1] < q1[x1]:
                g, _ = L.second_proposal(q1, q2t, x1, L.SP_GATED)
                r, _ = L.second_proposal(q1, q2t, x1, L.SP_RESIDUAL)
                assert np.allclose(g, r, atol=1e-15)
                n += 1
    assert n > 300


def test_naive_variant_monte_carlo_matches_exact_law():
    rng = np.random.default_rng(28)
    p, q1, q2t = _rand_dists(rng, 5, sparsity=0.0)
    law, a1, a2, rs = T.cascade_law_variant(p, q1, q2t, L.SP_NAIVE)
    R, d1, d2 = 4, 1, 2

    class Prov(_Fixed):
        def logits(self, node, r):
            return self.d[r] if len(node) == 1 else p

    prov = Prov(p, q1, q2t, d1, d2, R)
    n = 6000
    counts = np.zeros(5)
    src = np.zeros(3)
    for s in range(n):
        res = L.decode_loopspec(prov, R, d1, d2, 2, _S(1.0, 1.0, seed=13, seq=s), variant=L.SP_NAIVE)
        counts[res.tokens[1]] += 1
        src[res.sources[0]] += 1
    assert stats.chisquare(counts, law * n).pvalue > 1e-3
    assert stats.chisquare(src, np.array([rs, a1, a2]) * n).pvalue > 1e-3


def test_ungated_variants_need_sampling():
    p = np.array([0.5, 0.5])
    prov = _Fixed(p, p, p, 1, 2, 4)
    with pytest.raises(ValueError):
        L.decode_loopspec(prov, 4, 1, 2, 3, L.Sampler(0.0), variant=L.SP_NAIVE)
