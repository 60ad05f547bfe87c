"""In-flight branches read out mid-decode against the fp64 oracle.

After a few LoopSpec steps the tree holds branches at several depths, each a
prefix of committed tokens plus in-flight ancestors whose keys and values
live in their own branch slots.  Every live branch is read out (through the
C ABI) at its current depth -- the hidden state the decode step itself
produced -- and at every shallower depth by recomputation, and the logits are
compared with the oracle's readout of the same prefix at the same depth: the
first proposal's q1 = C(H^(d1)) and the gate's q2~ = C(H^(d2)) in particular
(Alg. 1; Sec. 4.2-4.3).  The launch configurations covered are the persistent
pass (<= 16 slots), the 64-row per-kernel path (more than 16 slots), the
per-kernel attention over more than 32 chunks of 64 positions, the
shared-prefix task attention, and a model with prelude and coda blocks.  Also: one vanilla token per call equals the
vanilla decode."""
import numpy as np
import pytest

from oracle import dist as OD
from oracle import model as OM

from gpu_common import MARGIN, TOL, log, model, prompt

pytestmark = pytest.mark.gpu


def _oracle_node(lm, cache, pr, prefix):
    """Oracle node of the token prefix (memoised along shared prefixes)."""
    key = tuple(int(t) for t in prefix)
    if key in cache:
        return cache[key]
    if len(key) == len(pr):
        node = lm.prefill(list(pr))
    else:
        node = lm.extend(_oracle_node(lm, cache, pr, key[:-1]), key[-1])
    cache[key] = node
    return node


def _check_tree(dec, spec, lm, pr, d1, d2, cache, what, coda=False):
    """Compare every live branch's readouts with the oracle; returns the
    number of (branch, depth) pairs compared and the depths seen."""
    dtype = spec.weight_dtype
    n = 0
    depths = set()
    for slot, info, prefix in dec.branches():
        assert list(prefix[:len(pr)]) == [int(t) for t in pr]
        cur = info["depth"]
        if cur < 1:
            continue
        node = _oracle_node(lm, cache, pr, prefix)
        want = range(1, cur + 1) if not coda else [d for d in (d1, d2, dec.R) if d and d <= cur]
        for r in want:
            got = dec.debug_readout(slot, r).astype(np.float64)
            ref = lm.logits(node, r)
            err = float(np.abs(got - ref).max())
            assert err <= TOL[dtype], (what, slot, info, r, err)
            if OD.top2_margin(ref) > MARGIN[dtype]:
                assert int(np.argmax(got)) == int(np.argmax(ref)), (what, slot, r)
            # the greedy draft recorded at d1 is the argmax of that readout
            if r == d1 and info["x1"] >= 0:
                assert info["x1"] == int(np.argmax(got)), (what, slot, info)
            n += 1
            depths.add(r)
    log(f"{what}: {n} (branch, depth) readouts within {TOL[dtype]} of the oracle; depths {sorted(depths)}")
    return n, depths


@pytest.mark.parametrize("name,n_prompt,max_slots,max_ctx,per_kernel,d1,d2,shared", [
    ("small_bf16", 70, 0, 256, False, 1, 2, False),      # persistent pass (<= 16 slots)
    ("small_bf16", 70, 24, 256, False, 1, 2, False),     # 64-row per-kernel path
    ("small_bf16", 1100, 0, 2600, True, 1, 2, False),    # per-kernel attention over 41 chunks
    ("small_bf16", 1100, 24, 2600, False, 1, 2, False),  # 64-row path, long context
    ("small_bf16", 1100, 0, 2600, True, 1, 2, True),     # shared-prefix task attention
    ("small_bf16", 70, 24, 256, False, 1, 2, True),      # shared-prefix, 64-row path
    ("tiny", 32, 0, 256, False, 1, 3, False),            # fp32 model
    ("tiny", 32, 0, 256, True, 1, 3, True),              # fp32, shared-prefix
])
def test_inflight_readouts_match_oracle(name, n_prompt, max_slots, max_ctx, per_kernel, d1, d2, shared):
    from paper_2609_17184_amd import Decoder
    spec, w = model(name)
    lm = OM.LoopedLM(spec, w)
    pr = prompt(spec, n_prompt)
    dec = Decoder(spec, w, R=spec.R, d1=d1, d2=d2, max_ctx=max_ctx, max_slots=max_slots, per_kernel=per_kernel,
                  shared_prefix=shared)
    slots = dec.capacity()[0]
    log(f"[debug] {name} prompt {n_prompt} slots {slots} max_ctx {max_ctx} per_kernel {per_kernel} "
        f"pass {dec.pass_attention}")
    if max_slots > 16 or per_kernel:
        assert not dec.pass_kernel
    dec.prefill(0, pr)
    cache = {}
    total, seen = 0, set()
    for step in range(7):
        dec.decode_step()
        n, d = _check_tree(dec, spec, lm, pr, d1, d2, cache, f"  step {step + 1}")
        total += n
        seen |= d
    assert total > 0 and {d1, d2} <= seen
    dec.close()


def test_inflight_readouts_with_coda_match_oracle():
    """Prelude and coda blocks: the readout at d1, d2 and R goes through the
    coda blocks with their per-readout-depth caches."""
    from paper_2609_17184_amd import Decoder
    spec, w = model("small_raven")
    lm = OM.LoopedLM(spec, w)
    pr = prompt(spec, 40)
    d1, d2 = 2, 5
    dec = Decoder(spec, w, R=spec.R, d1=d1, d2=d2, max_ctx=256)
    dec.prefill(0, pr)
    cache = {}
    total, seen = 0, set()
    for step in range(12):
        dec.decode_step()
        n, d = _check_tree(dec, spec, lm, pr, d1, d2, cache, f"  coda step {step + 1}", coda=True)
        total += n
        seen |= d
    assert {d1, d2} <= seen
    # a depth without coda caches for in-flight positions is refused
    slot = next(s for s, info, _ in dec.branches() if info["depth"] >= 3)
    with pytest.raises(RuntimeError):
        dec.debug_readout(slot, 3)
    dec.close()


@pytest.mark.parametrize("name", ["small_bf16", "small_raven"])
def test_vanilla_step_equals_vanilla_decode(name):
    from paper_2609_17184_amd import Decoder
    spec, w = model(name)
    d1, d2 = (1, 2) if spec.R == 4 else (2, 4)
    dec = Decoder(spec, w, R=spec.R, d1=d1, d2=d2, max_seqs=2, max_ctx=256)
    for q in range(2):
        dec.prefill(q, prompt(spec, 20 + 7 * q, seq=q))
    steps = np.stack([dec.vanilla_step() for _ in range(6)], axis=1)
    # LoopSpec decoding of a sequence on the vanilla schedule needs a rewind
    with pytest.raises(RuntimeError):
        dec.decode(1)
    for q in range(2):
        dec.rewind(q)
    ref = dec.vanilla_decode(6)
    assert np.array_equal(steps, ref), (steps, ref)
    for q in range(2):
        dec.rewind(q)
    assert np.array_equal(dec.decode(6), ref)          # greedy: LoopSpec == vanilla
    dec.close()


def test_debug_calls_reject_bad_arguments():
    from paper_2609_17184_amd import Decoder
    spec, w = model("micro")
    dec = Decoder(spec, w, R=spec.R, d1=1, d2=2, max_ctx=64)
    slots = dec.capacity()[0]
    with pytest.raises(RuntimeError):
        dec.branch(slots)                               # outside the pool
    dec.prefill(0, prompt(spec, 5))
    live = dec.branches()
    assert len(live) == 1 and live[0][1]["depth"] == 0 and live[0][1]["parent"] == -1
    with pytest.raises(RuntimeError):
        dec.debug_readout(live[0][0], 1)                # depth above the branch's current depth
    empty = next(s for s in range(slots) if s != live[0][0])
    with pytest.raises(RuntimeError):
        dec.debug_readout(empty, 1)                     # no branch in the slot
    dec.close()
