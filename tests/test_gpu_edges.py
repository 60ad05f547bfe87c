"""Edge cases of the decode path on the GPU: rejected prompts, a context that
fills up during decoding, zero-token calls, and a persistent pass holding its
maximum of 16 rows (capacity-limited spawning) that stays lossless."""
import numpy as np
import pytest

from paper_2609_17184_amd import binding as B
from paper_2609_17184_amd import Decoder

from gpu_common import log, model, prompt

pytestmark = pytest.mark.gpu


def test_prefill_rejects_bad_prompts():
    spec, w = model("micro")
    dec = Decoder(spec, w, R=4, d1=1, d2=2, max_ctx=32)
    with pytest.raises(B.LoopSpecError) as e:
        dec.prefill(0, [])
    assert e.value.code == B.EINVAL
    with pytest.raises(B.LoopSpecError) as e:
        dec.prefill(0, prompt(spec, 31))                 # prompt + 2 > max_ctx
    assert e.value.code == B.ECAPACITY
    with pytest.raises(B.LoopSpecError) as e:
        dec.prefill(0, [0, spec.vocab])                  # id out of range
    assert e.value.code == B.EINVAL
    assert 0 <= dec.prefill(0, prompt(spec, 30)) < spec.vocab   # the largest prompt that fits
    assert np.array_equal(dec.decode(0), np.zeros((1, 0), np.int32))
    dec.close()


@pytest.mark.parametrize("vanilla", [False, True])
def test_decode_up_to_full_context(vanilla):
    """A request past max_ctx is refused before any launch and leaves the
    sequence as it was; decoding right up to the last position works (branches
    that would run past it are not spawned) and stays lossless."""
    spec, w = model("micro")
    dec = Decoder(spec, w, R=4, d1=1, d2=2, max_ctx=24)
    run = dec.vanilla_decode if vanilla else dec.decode
    dec.prefill(0, prompt(spec, 10))
    with pytest.raises(B.LoopSpecError) as e:
        run(12)                                          # 10 + 1 + 12 + 2 > 24
    assert e.value.code == B.ECAPACITY
    full = run(11)
    with pytest.raises(B.LoopSpecError) as e:
        run(1)
    assert e.value.code == B.ECAPACITY
    dec.rewind(0)
    head = run(5)
    tail = run(6)
    assert np.array_equal(full, np.concatenate([head, tail], axis=1))
    dec.rewind(0)
    ref = dec.decode(11) if vanilla else dec.vanilla_decode(11)
    assert np.array_equal(full, ref)
    dec.close()


def test_decode_steps_until_full_context():
    """Single steps commit until the context is full, then report ECAPACITY."""
    spec, w = model("micro")
    dec = Decoder(spec, w, R=4, d1=1, d2=2, max_ctx=24)
    dec.prefill(0, prompt(spec, 10))
    steps = 0
    with pytest.raises(B.LoopSpecError) as e:
        while steps < 200:
            dec.decode_step()
            steps += 1
    assert e.value.code == B.ECAPACITY
    st = dec.stats()
    log(f"[steps] {steps} steps, committed {st['committed']}")
    assert steps >= 11            # the prefill committed one token; a step commits at most one more
    dec.rewind(0)
    assert dec.decode(11).shape == (1, 11)
    dec.close()


def test_pass_with_sixteen_rows_is_lossless():
    """Three sequences share a pool of 16 branch slots (the persistent pass's
    row limit; their worst case would need 21): spawns are refused when the
    pool is full and the output still equals vanilla decoding."""
    name = "small_bf16"
    spec, w = model(name)
    Q = 3
    dec = Decoder(spec, w, R=4, d1=1, d2=2, max_seqs=Q, max_ctx=160, max_slots=16)
    assert dec.pass_kernel and dec.capacity()[0] == 16
    for q in range(Q):
        dec.prefill(q, prompt(spec, 30 + 5 * q, seq=q))
    dec.reset_stats()
    a = dec.decode(40)
    st = dec.stats()
    for q in range(Q):
        dec.rewind(q)
    b = dec.vanilla_decode(40)
    log(f"[rows16] maxM={st['max_M']} refused={st['spawn_refused']} committed={st['committed']}")
    assert np.array_equal(a, b)
    assert st["max_M"] <= 16 and st["committed"] >= Q * 40
    dec.close()


@pytest.mark.parametrize("d1,d2,temperature", [(1, 2, 0.0), (2, 3, 0.0), (1, 2, 1.0)])
def test_single_steps_commit_what_decode_commits(d1, d2, temperature):
    """One step per call (the one-step graph) commits the same tokens as a
    decode of the same length (which replays multi-step graphs); sampled
    draws are keyed by position, so they agree too."""
    spec, w = model("small_bf16")
    dec = Decoder(spec, w, R=4, d1=d1, d2=d2, temperature=temperature, top_p=0.9 if temperature else 1.0,
                  max_ctx=128)
    dec.prefill(0, prompt(spec, 20))
    ref = [int(t) for t in dec.decode(24)[0]]
    dec.rewind(0)
    toks = []
    for _ in range(24 * 4 + 8):
        if len(toks) == 24:
            break
        tok, _ = dec.decode_step()
        if tok[0] >= 0:
            toks.append(int(tok[0]))
    assert toks == ref
    dec.close()


@pytest.mark.parametrize("vanilla", [False, True])
def test_sampled_decode_in_two_calls_equals_one(vanilla):
    """Sampled decoding split over two calls commits the same tokens as one
    call (keyed draws; the tree carries over between LoopSpec calls)."""
    spec, w = model("micro")
    dec = Decoder(spec, w, R=4, d1=1, d2=2, temperature=1.0, top_p=0.9, seed=7, max_ctx=64)
    run = dec.vanilla_decode if vanilla else dec.decode
    dec.prefill(0, prompt(spec, 10))
    full = run(20)
    dec.rewind(0)
    head = run(7)
    tail = run(13)
    assert np.array_equal(full, np.concatenate([head, tail], axis=1))
    dec.close()


def test_unprefilled_sequence_is_left_alone():
    """A handle with room for three sequences and two prefilled: the empty
    one's output row stays untouched and the others decode as they do alone."""
    spec, w = model("micro")
    dec = Decoder(spec, w, R=4, d1=1, d2=2, max_seqs=3, max_ctx=64)
    prs = {0: prompt(spec, 8, seq=0), 2: prompt(spec, 13, seq=2)}
    for q, pr in prs.items():
        dec.prefill(q, pr)
    out = dec.decode(10)
    assert (out[1] == -1).all()
    dec.close()
    for q, pr in prs.items():
        one = Decoder(spec, w, R=4, d1=1, d2=2, max_ctx=64)
        one.prefill(0, pr)
        assert np.array_equal(one.decode(10)[0], out[q])
        one.close()


def test_prefill_again_mid_decode():
    """Prefilling a sequence again in the middle of a decode replaces it (its
    branches and cache) while the other sequence carries on."""
    spec, w = model("micro")
    dec = Decoder(spec, w, R=4, d1=1, d2=2, max_seqs=2, max_ctx=64)
    pa, pb, pc = prompt(spec, 9, seq=0), prompt(spec, 12, seq=1), prompt(spec, 7, seq=2)
    dec.prefill(0, pa)
    dec.prefill(1, pb)
    first = dec.decode(5)
    dec.prefill(1, pc)
    second = dec.decode(6)
    dec.close()
    ref = {}
    for key, pr, n in (("a", pa, 11), ("c", pc, 6)):
        one = Decoder(spec, w, R=4, d1=1, d2=2, max_ctx=64)
        one.prefill(0, pr)
        ref[key] = one.decode(n)[0]
        one.close()
    assert np.array_equal(np.concatenate([first[0], second[0]]), ref["a"])
    assert np.array_equal(second[1], ref["c"])
