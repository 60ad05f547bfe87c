"""Shared set-up for the GPU parity tests: seeded models, the oracle's greedy
trajectory, and the comparison tolerances."""
import functools
import sys

import numpy as np

import synth
from oracle import loopspec as OL
from oracle import model as OM

# Tolerances on readout logits.  bf16 weights with bf16-rounded activations and
# fp32 accumulation: max-abs 5e-2 on logits, and top-1 must agree wherever the
# fp64 top-2 margin exceeds 0.1.  fp32 models: fp32 rounding only.
TOL = {"bf16": 5e-2, "f32": 1e-3}
MARGIN = {"bf16": 0.1, "f32": 2e-3}


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@functools.lru_cache(maxsize=None)
def model(name, **over):
    spec = synth.preset(name, **dict(over))
    return spec, synth.make_weights(spec, seed=0)


@functools.lru_cache(maxsize=None)
def oracle_lm(name, **over):
    spec, w = model(name, **over)
    return OM.LoopedLM(spec, w)


def prompt(spec, n, seq=0):
    return synth.make_prompt(spec.vocab, n, seed=1, seq=seq)


def oracle_greedy(name, n_prompt, n_tok, seq=0, **over):
    """The oracle's vanilla greedy trajectory and its per-position fp64 logits at
    every depth for the prefixes prompt || y_1 .. y_k."""
    spec, _ = model(name, **over)
    lm = oracle_lm(name, **over)
    pr = prompt(spec, n_prompt, seq)
    node = lm.prefill(list(pr))
    toks, logits = [], []
    z = lm.logits(node, spec.R)
    toks.append(int(np.argmax(z)))
    for _ in range(n_tok - 1):
        node = lm.extend(node, toks[-1])
        logits.append(np.stack([lm.logits(node, r) for r in range(1, spec.R + 1)]))
        toks.append(int(np.argmax(logits[-1][-1])))
    node = lm.extend(node, toks[-1])
    logits.append(np.stack([lm.logits(node, r) for r in range(1, spec.R + 1)]))
    return pr, toks, np.stack(logits), z


def oracle_trajectory(spec, w, pr, n_tok, cache64=True):
    """Like oracle_greedy for an explicit (spec, weights) pair, without caching
    the fp64 model: (greedy tokens, fp64 logits [n_tok, R, V] of the prefixes
    prompt || y_1 .. y_k, the first token's logits)."""
    lm = OM.LoopedLM(spec, w, cache64=cache64)
    node = lm.prefill(list(pr))
    z0 = lm.logits(node, spec.R)
    toks, logits = [int(np.argmax(z0))], []
    for k in range(n_tok):
        node = lm.extend(node, toks[-1])
        logits.append(np.stack([lm.logits(node, r) for r in range(1, spec.R + 1)]))
        if k + 1 < n_tok:
            toks.append(int(np.argmax(logits[-1][-1])))
    return toks, np.stack(logits), z0
