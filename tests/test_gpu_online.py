"""Switching the proposal depths while decoding (loopspec_set_depths), the
TV statistics the decode gathers for re-planning, and the online planner
loop, against the fp64 oracle's Alg. 1 run with the same switches.

* greedy at R = 8: tokens across four pair switches equal vanilla decoding
  on the same kernels (bf16 and fp32 models); on fp32 models they equal the
  oracle's tokens, and the commit sources and summed argmax mismatches at d1
  and d2 equal the oracle's records;
* a prelude + core + coda model: mid-sequence only pairs whose readout depths
  the generated positions' coda caches cover are accepted (others: ESTATE),
  any pair after a rewind, and both stay lossless;
* sampled, keyed draws (one shard per row at V = 16, four at V = 4096):
  tokens equal the oracle's keyed run with the same switches up to its first
  near-tie decision, and the TV sums TV(p_R, p_d1), TV(p_R, p_d2) equal the
  oracle's per-verification records (fp32 against fp64);
* decode_adaptive (segments, re-plan, switch) stays lossless; bad pairs are
  refused with the right error code and leave the handle usable.
"""
import numpy as np
import pytest

from oracle import loopspec as OL
from oracle import model as OM
from paper_2609_17184_amd import depths as PD

from gpu_common import log, model, prompt

pytestmark = pytest.mark.gpu

FRAGILE = {"race": 1e-4, "accept": 1e-4, "topp": 1e-4, "gate": 1e-4}
ARGMAX_MARGIN = {"bf16": 0.1, "f32": 2e-3}
SCALE = 2.0 ** -32


def _compared(res, argmax_margin):
    """Leading committed tokens of the oracle's run that no near-tie decision
    precedes (a decision at step t may change every commit from step t on)."""
    th = dict(FRAGILE, argmax=argmax_margin)
    bad = [d[1] for d in res.decisions if d[2] < th[d[0]]]
    if not bad:
        return len(res.tokens)
    f = min(bad)
    return 1 + sum(1 for c in res.commit_steps if c < f) if f > 0 else 0


def _segments(dec, first, pairs):
    """Decode segment by segment, switching to the next pair between them;
    returns the token list (prefill token first) and the oracle's switch map."""
    toks, sw, done = [first], {}, 1
    for i, (n, d1, d2) in enumerate(pairs):
        if i:
            dec.set_depths(d1, d2)
            sw[done] = (d1, d2)
        toks += list(dec.decode(n)[0])
        done += n
    return toks, sw


PAIRS8 = [(9, 2, 4), (7, 3, 5), (8, 1, 0), (6, 2, 6), (9, 1, 3)]


@pytest.mark.parametrize("name,alpha,n_prompt,oracle", [("micro", 0.6, 9, True), ("micro", 2.0, 12, True),
                                                        ("small_bf16", 0.3, 12, False)])
def test_greedy_switches_match_vanilla_and_oracle(name, alpha, n_prompt, oracle):
    """Greedy decoding across four pair switches at R = 8 equals vanilla
    decoding; on the fp32 models (drafts rejected at most positions, no
    near-tie in the oracle's run) the tokens, commit sources and TV records
    equal the oracle's Alg. 1 run with the same switches."""
    over = {"R": 8, "alpha": alpha}
    spec, w = model(name, **over)
    pr = prompt(spec, n_prompt)
    R = spec.R
    N = 1 + sum(p[0] for p in PAIRS8)
    from paper_2609_17184_amd import Decoder
    dec = Decoder(spec, w, R=R, d1=PAIRS8[0][1], d2=PAIRS8[0][2], max_ctx=128, max_slots=64)
    first = dec.prefill(0, pr)
    toks, sw = _segments(dec, first, PAIRS8)
    st = dec.stats()
    dec.rewind(0)
    van = [first] + list(dec.vanilla_decode(N - 1)[0])
    dec.close()
    assert toks == van
    assert st["tv_count"] == st["committed"] == N - 1
    assert st["spawn_refused"] == 0 and st["zero_mass"] == 0
    # a first proposal is accepted exactly when it is the target's argmax
    assert st["tv_d1"] * SCALE == st["tv_count"] - st["n_acc1"]
    if not oracle:
        return
    lm = OM.LoopedLM(spec, w)
    res = OL.decode_loopspec(OL.ModelReadouts(lm, pr), R, PAIRS8[0][1], PAIRS8[0][2], N, OL.Sampler(0.0),
                             switches=sw)
    # greedy: only the argmax decisions can be near-ties (the gate compares one-hot readouts)
    thr = ARGMAX_MARGIN[spec.weight_dtype]
    bad = [d[1] for d in res.decisions if d[0] == "argmax" and d[2] < thr]
    log(f"[online greedy] {name} alpha={alpha} switches {sw}: gpu acc1={st['n_acc1']} acc2={st['n_acc2']} "
        f"restart={st['n_restart']} tv_d1={st['tv_d1'] * SCALE:.0f} tv_d2={st['tv_d2'] * SCALE:.0f}; oracle "
        f"acc1={res.n_acc1} acc2={res.n_acc2} restart={res.n_restart} tv1={sum(res.tv1):.0f} "
        f"tv2={sum(res.tv2):.0f}; near-ties {len(bad)}")
    assert not bad, "the oracle's run has a near-tie: pick another prompt"
    assert toks == res.tokens
    assert (st["n_acc1"], st["n_acc2"], st["n_restart"]) == (res.n_acc1, res.n_acc2, res.n_restart)
    assert st["tv_d1"] * SCALE == sum(res.tv1) and st["tv_d2"] * SCALE == sum(res.tv2)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name,pairs,T,top_p,variant", [
    ("micro", [(9, 1, 2), (8, 2, 3), (7, 1, 0), (9, 1, 3)], 1.0, 1.0, OL.SP_GATED),
    ("micro", [(9, 1, 2), (8, 2, 3), (9, 1, 3)], 1.0, 0.9, OL.SP_RESIDUAL),
    ("tiny", [(9, 1, 2), (8, 2, 3), (7, 1, 0), (9, 1, 3)], 1.0, 1.0, OL.SP_GATED),
])
def test_sampled_switches_match_the_oracle(name, pairs, T, top_p, variant):
    spec, w = model(name)
    pr = prompt(spec, 9)
    R, seed = spec.R, 11
    N = 1 + sum(p[0] for p in pairs)
    from paper_2609_17184_amd import Decoder
    dec = Decoder(spec, w, R=R, d1=pairs[0][1], d2=pairs[0][2], temperature=T, top_p=top_p, seed=seed,
                  max_ctx=128, max_slots=16, second_proposal=variant)
    first = dec.prefill(0, pr)
    toks, sw = _segments(dec, first, pairs)
    st = dec.stats()
    dec.close()
    lm = OM.LoopedLM(spec, w)
    res = OL.decode_loopspec(OL.ModelReadouts(lm, pr), R, pairs[0][1], pairs[0][2], N,
                             OL.Sampler(T, top_p, seed=seed, seq=0), variant=variant, switches=sw)
    k = _compared(res, 0.0)
    log(f"[online sampled] {name} T={T} top_p={top_p} variant={variant} switches {sw}: gpu "
        f"acc1={st['n_acc1']} acc2={st['n_acc2']} restart={st['n_restart']} tv_d1={st['tv_d1'] * SCALE:.5f} "
        f"tv_d2={st['tv_d2'] * SCALE:.5f}; oracle acc1={res.n_acc1} acc2={res.n_acc2} restart={res.n_restart} "
        f"tv1={sum(res.tv1):.5f} tv2={sum(res.tv2):.5f}; compared {k}/{N}")
    assert k >= 10
    assert toks[:k] == res.tokens[:k]
    assert st["tv_count"] == st["committed"] == N - 1
    if k == N:
        assert (st["n_acc1"], st["n_acc2"], st["n_restart"]) == (res.n_acc1, res.n_acc2, res.n_restart)
        # fp32 readouts and sums in 2^-40 fixed point against fp64
        tol = 1e-4 * (N - 1)
        assert abs(st["tv_d1"] * SCALE - sum(res.tv1)) < tol
        assert abs(st["tv_d2"] * SCALE - sum(res.tv2)) < tol
    assert st["zero_mass"] == 0


def test_decode_adaptive_is_lossless_and_replans():
    """The planner loop on the R = 8 model, greedy: the tokens equal vanilla
    decoding whatever pairs it picks, every segment after the first two
    measured depths carries a plan, and the planned pairs fit the pool."""
    name = "small_bf16"
    spec, w = model(name, R=8)
    pr = prompt(spec, 12)
    from paper_2609_17184_amd import Decoder
    from paper_2609_17184_amd.binding import worst_case_branches
    dec = Decoder(spec, w, R=spec.R, d1=2, d2=4, max_ctx=160, max_slots=32)
    first = dec.prefill(0, pr)
    toks, plans = PD.decode_adaptive(dec, 72, every=12, margin=0.0, min_count=4)
    dec.rewind(0)
    van = dec.vanilla_decode(72)[0]
    slots = dec.capacity()[0]
    dec.close()
    assert list(toks[0]) == list(van)
    made = [p for p in plans if p["plan"] is not None]
    log(f"[online adaptive] first {first}: " + "; ".join(
        f"{p['tokens']} tok at ({p['d1']},{p['d2']}) -> {p.get('switched_to', '-')}" for p in plans))
    assert made, "no plan was made"
    for p in made:
        d1, d2 = p["plan"]["d1"], p["plan"]["d2"]
        assert 0 < worst_case_branches(spec.R, d1, d2) <= slots
        assert p["plan"]["steps_bound"] <= p["plan"]["current_bound"] + 1e-12


def test_coda_model_switches_within_its_coda_caches():
    """Prelude + core + coda model, greedy: after decoding at (2, 4) the
    generated positions hold coda keys / values at depths 2, 4 and R only, so
    (3, 5) is refused (ESTATE) and (4, 0) accepted mid-sequence; after a
    rewind (3, 5) is accepted; every run equals vanilla decoding."""
    from paper_2609_17184_amd import Decoder, LoopSpecError
    spec, w = model("small_raven")
    pr = prompt(spec, 10)
    dec = Decoder(spec, w, R=spec.R, d1=2, d2=4, max_ctx=96, max_slots=16)
    first = dec.prefill(0, pr)
    a = list(dec.decode(12)[0])
    assert dec.can_set_depths(3, 5) == -5 and dec.can_set_depths(4, 0) == 0 and dec.can_set_depths(2, 0) == 0
    with pytest.raises(LoopSpecError) as e:
        dec.set_depths(3, 5)
    assert e.value.code == -5 and "coda" in str(e.value)
    dec.set_depths(4, 0)
    a += list(dec.decode(12)[0])
    assert dec.can_set_depths(2, 4) == -5           # depth 2 was not read out at (4, 0)
    dec.rewind(0)
    assert dec.can_set_depths(3, 5) == 0
    dec.set_depths(3, 5)
    b = list(dec.decode(24)[0])
    dec.rewind(0)
    van = list(dec.vanilla_decode(24)[0])
    st = dec.stats()
    dec.close()
    log(f"[online coda] first {first}: switched run {a[:8]}..., rewound run {b[:8]}...")
    assert a == van and b == van
    assert st["zero_mass"] == 0


def test_set_depths_refuses_bad_pairs():
    from paper_2609_17184_amd import Decoder, LoopSpecError
    spec, w = model("small_raven")
    pr = prompt(spec, 6)
    dec = Decoder(spec, w, R=spec.R, d1=2, d2=4, max_ctx=64)
    first = dec.prefill(0, pr)
    ref = dec.decode(10)[0]
    codes = {}
    for d1, d2 in ((0, 2), (4, 4), (2, 8), (8, 0), (1, 2)):
        with pytest.raises(LoopSpecError) as e:
            dec.set_depths(d1, d2)
        codes[(d1, d2)] = e.value.code
    # (1, 2) at R = 8 needs 54 slots per sequence; the pool was sized for (2, 4)
    assert codes[(1, 2)] == -4 and all(c == -1 for k, c in codes.items() if k != (1, 2)), codes
    dec.set_depths(2, 4)                                     # the same pair: nothing happens
    dec.rewind(0)
    again = dec.decode(10)[0]
    dec.close()
    assert list(again) == list(ref), (first, ref, again)
