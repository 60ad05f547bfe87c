"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle, and
greedy LoopSpec against vanilla looped decoding on the same kernels."""
import numpy as np
import pytest

from oracle import dist as OD
from oracle import loopspec as OL
from oracle import model as OM
import synth

from gpu_common import MARGIN, TOL, log, model, oracle_greedy, oracle_lm, prompt

pytestmark = pytest.mark.gpu


def decoder(name, R=4, d1=1, d2=2, max_seqs=1, max_ctx=256, per_kernel=False, **over):
    from paper_2609_17184_amd import Decoder
    spec, w = model(name, **over)
    return spec, Decoder(spec, w, R=R, d1=d1, d2=d2, max_seqs=max_seqs, max_ctx=max_ctx,
                         per_kernel=per_kernel)


def _check_logits(got, ref, dtype, what):
    err = np.abs(got.astype(np.float64) - ref).max()
    log(f"{what}: max |gpu - oracle| = {err:.3e} (tol {TOL[dtype]})")
    assert err <= TOL[dtype], what
    # top-1 agreement where the oracle's top-2 margin is wide enough
    for g, r in zip(got.reshape(-1, got.shape[-1]), ref.reshape(-1, ref.shape[-1])):
        if OD.top2_margin(r) > MARGIN[dtype]:
            assert int(np.argmax(g)) == int(np.argmax(r))


@pytest.mark.parametrize("name,n_prompt,n_tok,over,per_kernel,max_ctx", [
    ("micro", 7, 6, (), False, 256), ("tiny", 32, 5, (), False, 256), ("small_bf16", 70, 5, (), False, 256),
    ("small_bf16", 70, 5, (), True, 256), ("small_bf16", 20, 4, (("gain_noise", 0.2),), False, 256),
    ("micro", 9, 4, (("gain_noise", 0.3),), False, 256), ("small_raven", 40, 4, (), False, 256),
    ("small_raven", 40, 4, (), True, 256),
    # long contexts: 18 chunks per row over one workgroup's 8 waves (max_ctx
    # 2048), and the chunk-task attention of longer-context handles
    ("small_bf16", 1100, 4, (), False, 2048), ("small_bf16", 1100, 4, (), False, 2600),
    ("tiny", 32, 5, (), False, 2600)])
def test_teacher_forced_logits(name, n_prompt, n_tok, over, per_kernel, max_ctx):
    """Readout logits at every depth along the oracle's greedy trajectory; the
    decode passes run as the persistent kernel (per_kernel False, when the model
    fits it) or as one launch per kernel."""
    over = dict(over)
    log(f"[teacher-forced] {name} prompt {n_prompt} tokens {n_tok} {over} per_kernel={per_kernel} "
        f"max_ctx={max_ctx}")
    spec, dec = decoder(name, R=synth.preset(name).R, d1=1, d2=2, per_kernel=per_kernel, max_ctx=max_ctx,
                        **over)
    log(f"  persistent pass kernel: {dec.pass_kernel} (attention mode {dec.pass_attention})")
    if per_kernel:
        assert not dec.pass_kernel
    elif name != "small_raven":
        assert dec.pass_attention == (1 if max_ctx <= 2048 else 2)
    pr, toks, ref, z0 = oracle_greedy(name, n_prompt, n_tok, **over)
    first = dec.prefill(0, pr)
    if OD.top2_margin(z0) > MARGIN[spec.weight_dtype]:
        assert first == toks[0]
    lg, am = dec.forced_readout(0, toks)
    _check_logits(lg, ref, spec.weight_dtype, f"{name} logits [n, R, V]")
    dec.close()


@pytest.mark.parametrize("name,depths,per_kernel,max_ctx", [
    ("micro", [(1, 2), (1, 3), (2, 3), (1, 0), (2, 0)], False, 256),
    ("tiny", [(1, 2), (2, 3)], False, 256),
    ("small_bf16", [(1, 2), (1, 3), (2, 0)], False, 256),
    ("small_bf16", [(1, 2)], True, 256),
    ("small_bf16", [(1, 2), (2, 0)], False, 2600),       # chunk-task attention in the pass
    ("small_raven", [(2, 4), (1, 5), (3, 0)], False, 256)])
def test_greedy_loopspec_equals_vanilla(name, depths, per_kernel, max_ctx):
    spec = synth.preset(name)
    R = spec.R
    pr = prompt(spec, 33)
    for d1, d2 in depths:
        log(f"[lossless] {name} R={R} d1={d1} d2={d2} per_kernel={per_kernel} max_ctx={max_ctx}")
        _, dec = decoder(name, R=R, d1=d1, d2=d2, per_kernel=per_kernel, max_ctx=max_ctx)
        dec.prefill(0, pr)
        a = dec.decode(48)
        st = dec.stats()
        dec.rewind(0)
        b = dec.vanilla_decode(48)
        log(f"  acc1={st['n_acc1']} acc2={st['n_acc2']} restart={st['n_restart']} steps={st['steps']} "
            f"maxM={st['max_M']}")
        assert np.array_equal(a, b)
        assert st["n_acc1"] + st["n_acc2"] + st["n_restart"] == st["committed"] == 48
        cost = st["n_acc1"] * d1 + st["n_acc2"] * (d2 or R) + st["n_restart"] * R
        # first root needs R steps, then each commit's source sets the next gap;
        # the last commit's own gap is not stepped
        assert abs(st["steps"] - cost) <= R
        dec.close()


def test_loopspec_matches_oracle_simulator():
    """Tokens and commit sources equal the oracle's Alg. 1 run (fp32 model: no
    near-tie decisions in this trajectory)."""
    name, R, d1, d2, N = "micro", 4, 1, 2, 40
    spec, w = model(name)
    lm = OM.LoopedLM(spec, w)
    pr = prompt(spec, 9)
    s = OL.Sampler(0.0)
    res = OL.decode_loopspec(OL.ModelReadouts(lm, pr), R, d1, d2, N, s)
    fragile = [d for d in res.decisions if d[0] == "argmax" and d[2] < MARGIN["f32"]]
    log(f"[sim] oracle acc1={res.n_acc1} acc2={res.n_acc2} restart={res.n_restart} steps={res.steps} "
        f"fragile={len(fragile)}")
    _, dec = decoder(name, R=R, d1=d1, d2=d2)
    first = dec.prefill(0, pr)
    toks = [first] + list(dec.decode(N - 1)[0])
    st = dec.stats()
    if not fragile:
        assert toks == res.tokens
        assert (st["n_acc1"], st["n_acc2"], st["n_restart"]) == (res.n_acc1, res.n_acc2, res.n_restart)
        assert st["steps"] == res.steps
        assert st["max_M"] == max(res.M)
        assert st["gate_eval"] == res.gate_eval and st["gate_open"] == res.gate_open
    else:
        k = min(res.commit_steps.index(c) for c in res.commit_steps if c >= fragile[0][1]) + 1
        assert toks[:k] == res.tokens[:k]
    dec.close()


@pytest.mark.parametrize("Q,max_ctx", [(2, 160), (3, 160), (2, 2600)])
def test_batch_invariance_across_sequences(Q, max_ctx):
    """Within one handle, a sequence decodes to the same tokens whether it runs
    alone or batched with other sequences (other rows, another M every step).
    Q = 2 keeps the (4, 1, 2) slot pool at 14 rows (persistent pass kernel;
    with max_ctx 2600 its chunk-task attention); Q = 3 needs 21 (per-kernel
    launches with 64-row tiles)."""
    name = "small_bf16"
    spec, w = model(name)
    from paper_2609_17184_amd import Decoder
    dec = Decoder(spec, w, R=4, d1=1, d2=2, max_seqs=Q, max_ctx=max_ctx)
    dec.prefill(0, prompt(spec, 40, seq=0))
    a = dec.decode(40)[0]
    dec.rewind(0)
    for q in range(1, Q):
        dec.prefill(q, prompt(spec, 40 + 7 * q, seq=q))
    b = dec.decode(40)
    st = dec.stats()
    log(f"[batch] Q={Q} slots={dec.capacity()[0]} pass={dec.pass_kernel} maxM={st['max_M']} "
        f"committed={st['committed']}")
    assert dec.pass_kernel == (Q == 2)
    assert np.array_equal(a, b[0])
    dec.close()


def test_decode_step_api():
    spec, dec = decoder("micro")
    dec.prefill(0, prompt(spec, 5))
    toks = []
    for _ in range(30):
        t, src = dec.decode_step()
        if t[0] >= 0:
            assert src[0] in (0, 1, 2)
            toks.append(int(t[0]))
    dec.rewind(0)
    ref = dec.vanilla_decode(len(toks))[0]
    assert toks == list(ref)
    dec.close()
