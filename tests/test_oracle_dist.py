"""Pins for readout distributions, the residual operator, draws and Philox."""
import numpy as np
import pytest
from scipy import special, stats

from oracle import dist as D
from oracle import philox as PX


def test_softmax_matches_scipy():
    z = np.random.default_rng(0).standard_normal(50) * 3
    for T in (0.5, 1.0, 2.0):
        assert np.allclose(D.readout_dist(z, T), special.softmax(z / T), atol=1e-15)


def test_greedy_is_one_hot_lowest_id():
    z = np.array([0.1, 3.0, -1.0, 3.0])
    p = D.readout_dist(z, 0.0)
    assert p.tolist() == [0, 1, 0, 0]


def test_top_p_hand_example():
    # probabilities 0.5, 0.3, 0.15, 0.05 (from logs); top_p = 0.79:
    # ranked-before masses 0, 0.5, 0.8, 0.95 -> keep the first two, renormalise
    p0 = np.array([0.15, 0.5, 0.05, 0.3])
    p = D.readout_dist(np.log(p0), 1.0, 0.79)
    assert np.allclose(p, [0, 0.625, 0, 0.375])
    # top_p above 0.8 keeps the third
    p = D.readout_dist(np.log(p0), 1.0, 0.81)
    assert np.allclose(p, np.array([0.15, 0.5, 0, 0.3]) / 0.95)
    # at least one token survives
    assert D.readout_dist(np.log(p0), 1.0, 1e-9).tolist() == [0, 1, 0, 0]


def test_top_p_ties_by_lower_id():
    p0 = np.array([0.25, 0.25, 0.25, 0.25])
    p = D.readout_dist(np.log(p0), 1.0, 0.5)
    assert np.allclose(p, [0.5, 0.5, 0, 0])


def test_residual_and_tv_closed_forms():
    mu = np.array([0.5, 0.3, 0.2])
    nu = np.array([0.2, 0.5, 0.3])
    r, zm = D.residual(mu, nu)
    assert not zm and np.allclose(r, [1, 0, 0])
    assert np.isclose(D.tv(mu, nu), 0.5 * np.abs(mu - nu).sum())
    assert np.isclose(D.tv(mu, nu), D.tv(nu, mu))
    mu = np.array([0.6, 0.1, 0.3])
    nu = np.array([0.2, 0.3, 0.5])
    r, _ = D.residual(mu, nu)
    assert np.allclose(r, [1, 0, 0])
    r, zm = D.residual(mu, mu)
    assert zm and np.allclose(r, mu)


def test_race_sample_distribution():
    w = np.array([0.1, 0.0, 0.4, 0.2, 0.3])
    n = 40000
    counts = np.zeros(5)
    for s in range(n // 1000):
        U = PX.vocab_uniforms(7, s, 0, PX.TARGET, 5 * 1000).reshape(1000, 5)
        for u in U:
            counts[D.race_sample(w, u)[0]] += 1
    assert counts[1] == 0
    nz = w > 0
    chi = stats.chisquare(counts[nz], w[nz] * n)
    assert chi.pvalue > 1e-3


@pytest.mark.parametrize("seed", range(5))
def test_philox_matches_numpy(seed):
    rng = np.random.default_rng(seed)
    key = rng.integers(0, 2 ** 63, 2, dtype=np.uint64)
    ctr = rng.integers(1, 2 ** 63, 4, dtype=np.uint64)
    bg = np.random.Philox(key=key, counter=ctr - np.array([1, 0, 0, 0], np.uint64))
    ref = bg.random_raw(4)                      # numpy bumps the counter before output
    got = PX.philox4x64([int(c) for c in ctr], [int(k) for k in key])
    assert list(got) == [int(x) for x in ref]
    vec = PX.philox4x64_vec(np.array([ctr[0]]), int(ctr[1]), int(ctr[2]), int(ctr[3]),
                            [int(k) for k in key])[0]
    assert [int(x) for x in vec] == [int(x) for x in ref]


def test_uniforms_exact_in_fp32_and_distributed():
    u = PX.vocab_uniforms(1, 0, 5, PX.TARGET, 100000)
    assert np.all(u.astype(np.float32).astype(np.float64) == u)
    assert u.min() > 0 and u.max() < 1
    assert stats.kstest(u, "uniform").pvalue > 1e-3
    s = np.array([PX.scalar_uniform(3, 0, p, PX.ACC1) for p in range(3000)])
    assert np.all(s.astype(np.float32).astype(np.float64) == s)
    assert stats.kstest(s, "uniform").pvalue > 1e-3
