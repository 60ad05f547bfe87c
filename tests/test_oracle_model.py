"""Pins for the fp64 looped forward: textbook operations checked against
independent formulations, the per-depth KV cache against a cache-free
recomputation, and the alpha = 0 special case."""
import numpy as np
import pytest
from scipy import special

import synth
from oracle import model as M


def test_rmsnorm_properties():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 64)) * 3
    g = np.ones(64)
    y = M.rms_norm(x, g, 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0)
    assert np.allclose(M.rms_norm(7.5 * x, g, 0.0), y)          # scale invariance
    g2 = rng.standard_normal(64)
    assert np.allclose(M.rms_norm(x, g2, 0.0), y * g2)
    # eps enters under the root: a zero vector maps to zero, not NaN
    assert np.all(M.rms_norm(np.zeros((1, 4)), np.ones(4), 1e-6) == 0)


def test_rope_equals_complex_rotation():
    rng = np.random.default_rng(1)
    T, H, dh, base = 7, 3, 16, 10000.0
    x = rng.standard_normal((T, H, dh))
    pos = np.array([0, 1, 5, 17, 100, 1023, 8191])
    y = M.rope(x, pos, base)
    half = dh // 2
    z = x[..., :half] + 1j * x[..., half:]
    theta = np.exp(1j * pos[:, None] * base ** (-np.arange(0, dh, 2) / dh))
    w = z * theta[:, None, :]
    assert np.allclose(y[..., :half], w.real) and np.allclose(y[..., half:], w.imag)
    assert np.allclose(M.rope(x, np.zeros(T), base), x)


def test_rope_relative_position():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 1, 32))
    k = rng.standard_normal((1, 1, 32))
    d = [float((M.rope(q, np.array([m + 3]), 1e4) * M.rope(k, np.array([m]), 1e4)).sum())
         for m in (0, 10, 500)]
    assert np.allclose(d, d[0])


def test_attention_against_loops():
    rng = np.random.default_rng(3)
    Tq, Tk, H, dh = 3, 6, 2, 8
    q = rng.standard_normal((Tq, H, dh))
    K = rng.standard_normal((Tk, H, dh))
    V = rng.standard_normal((Tk, H, dh))
    qpos = np.array([3, 4, 5])
    kpos = np.arange(Tk)
    out = M.causal_attention(q, K, V, qpos, kpos)
    for i in range(Tq):
        for h in range(H):
            s = np.array([q[i, h] @ K[j, h] / np.sqrt(dh) for j in range(qpos[i] + 1)])
            w = special.softmax(s)
            ref = sum(w[j] * V[j, h] for j in range(qpos[i] + 1))
            assert np.allclose(out[i, h], ref)
    # identical keys: the output is the mean of the visible values
    out = M.causal_attention(q[:1], np.ones((Tk, H, dh)), V, np.array([5]), kpos)
    assert np.allclose(out[0], V.mean(axis=0))


def test_silu():
    x = np.linspace(-10, 10, 101)
    assert np.allclose(M.silu(x), x * special.expit(x))


@pytest.mark.parametrize("name", ["micro", "small_raven"])
def test_cached_forward_equals_cache_free(name):
    spec = synth.preset(name, gain_noise=0.1)
    lm = M.LoopedLM(spec, synth.make_weights(spec, seed=5))
    prompt = synth.make_prompt(spec.vocab, 9, seed=6)
    extra = [3, 1, 4, 1, 5]
    node = lm.prefill(prompt)
    nodes = [node]
    for t in extra:
        node = lm.extend(node, t)
        nodes.append(node)
    full = lm.forward_full(list(prompt) + extra)
    for r in range(1, spec.R + 1):
        for i, nd in enumerate(nodes):
            ref = full[r][len(prompt) - 1 + i]
            got = lm.logits(nd, r)
            assert np.allclose(got, ref, rtol=1e-12, atol=1e-12), (r, i)


def test_sibling_prefixes_do_not_mix():
    # extending the same prefix by different tokens gives the cache-free values of each
    spec = synth.preset("micro")
    lm = M.LoopedLM(spec, synth.make_weights(spec))
    prompt = [1, 2, 3]
    root = lm.prefill(prompt)
    a = lm.extend(lm.extend(root, 4), 5)
    b = lm.extend(lm.extend(root, 6), 5)
    for r in (1, spec.R):
        assert np.allclose(lm.logits(a, r), lm.forward_full(prompt + [4, 5])[r][-1], atol=1e-12)
        assert np.allclose(lm.logits(b, r), lm.forward_full(prompt + [6, 5])[r][-1], atol=1e-12)


def test_alpha_zero_all_depths_identical():
    spec = synth.preset("micro", alpha=0.0)
    lm = M.LoopedLM(spec, synth.make_weights(spec))
    node = lm.prefill([5, 7, 9])
    for r in range(1, spec.R + 1):
        assert np.array_equal(lm.logits(node, r), lm.logits(node, spec.R))
    # and they equal the bare embedding readout: W_head RMSNorm(E[x])
    W = lm.W
    x = W["embed"][9]
    ref = W["head"] @ (x / np.sqrt(np.mean(x * x) + spec.rms_eps))
    assert np.allclose(lm.logits(node, 1), ref)
