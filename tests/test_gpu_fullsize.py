"""The benchmarked shapes on the GPU.

* Full width against the oracle: the Ouro-1.4B shape (h 2048, 16x128 heads,
  FFN 5632, V 49152, bf16, R 4) with two shared blocks instead of 24 runs the
  persistent pass in the launch configuration of the benchmark (the same work
  items per phase, tiles, k-slices, grid and LDS; the layer count only sets
  the loop length), so its readout logits at every depth are checked against
  the fp64 oracle along the oracle's greedy trajectory, after a 160-token
  prompt (two full 64-position chunks and a ragged one).
* Full size, properties that hold at any size: the 24-block Ouro-1.4B shape
  after a 512-token prompt (the benchmark's workload) decodes greedily to the
  same tokens with LoopSpec as with vanilla looped decoding, for the
  benchmark's depth pair and the paper's; three sequences sharing a 16-row
  pool (the pass's row limit) do too; and the sampled Ouro-2.6B shape
  (T 1, top-p 0.95) repeats its draws exactly under the same key."""
import numpy as np
import pytest

import synth

from gpu_common import log, prompt
from test_gpu_parity import _check_logits

pytestmark = pytest.mark.gpu


@pytest.mark.timeout(400)
def test_full_width_readouts_match_oracle():
    from paper_2609_17184_amd import Decoder
    from oracle import model as OM
    spec = synth.preset("ouro14", n_core=2)
    w = synth.make_weights(spec, seed=0)
    pr = list(prompt(spec, 160))
    log("[full-width] oracle prefill (fp64) ...")
    lm = OM.LoopedLM(spec, w)
    node = lm.prefill(pr)
    z0 = lm.logits(node, spec.R)
    toks = [int(np.argmax(z0))]
    ref = []
    for _ in range(3):
        node = lm.extend(node, toks[-1])
        ref.append(np.stack([lm.logits(node, r) for r in range(1, spec.R + 1)]))
        toks.append(int(np.argmax(ref[-1][-1])))
    ref = np.stack(ref)
    log("[full-width] oracle done; GPU")
    dec = Decoder(spec, w, R=spec.R, d1=2, d2=3, max_ctx=1024)
    assert dec.pass_kernel and dec.pass_attention == 1
    first = dec.prefill(0, pr)
    lg, _ = dec.forced_readout(0, toks[:3])
    _check_logits(lg, ref, "bf16", "ouro14 width, 2 blocks: logits [3, R, V]")
    log(f"[full-width] first token gpu {first} oracle {toks[0]}")
    from gpu_common import MARGIN
    from oracle import dist as OD
    if OD.top2_margin(z0) > MARGIN["bf16"]:
        assert first == toks[0]
    dec.close()


@pytest.mark.timeout(900)
def test_full_depth_readouts_match_oracle():
    """All 24 shared blocks of the Ouro-1.4B shape (96 block applications per
    token at R = 4) after a 64-token prompt: readout logits at every depth of
    three forced tokens within max-abs 5e-2 of the fp64 oracle, top-1 agreeing
    wherever the oracle's top-2 margin exceeds 0.1, and the first token after
    prefill equal to the oracle's where its margin does."""
    from paper_2609_17184_amd import Decoder
    from gpu_common import MARGIN, oracle_trajectory
    from oracle import dist as OD
    spec = synth.preset("ouro14")
    w = synth.make_weights(spec, seed=0)
    pr = list(prompt(spec, 64))
    log("[full-depth] fp64 oracle over 24 blocks ...")
    toks, ref, z0 = oracle_trajectory(spec, w, pr, 3)
    log(f"[full-depth] oracle tokens {toks}; GPU")
    dec = Decoder(spec, w, R=spec.R, d1=2, d2=3, max_ctx=1024)
    assert dec.pass_kernel
    first = dec.prefill(0, pr)
    log(f"[full-depth] first token gpu {first} oracle {toks[0]} (margin {OD.top2_margin(z0):.3f})")
    if OD.top2_margin(z0) > MARGIN["bf16"]:
        assert first == toks[0]
    lg, _ = dec.forced_readout(0, toks)
    _check_logits(lg, ref, "bf16", "ouro14 full depth (24 blocks): logits [3, R, V]")
    dec.close()


@pytest.fixture(scope="module")
def ouro14():
    spec = synth.preset("ouro14")
    return spec, synth.make_weights(spec, seed=0)


@pytest.mark.parametrize("d1,d2", [(2, 3), (1, 2)])
def test_full_size_greedy_loopspec_equals_vanilla(ouro14, d1, d2):
    from paper_2609_17184_amd import Decoder
    spec, w = ouro14
    dec = Decoder(spec, w, R=spec.R, d1=d1, d2=d2, max_ctx=1024)
    assert dec.pass_kernel
    dec.prefill(0, prompt(spec, 512))
    a = dec.decode(32)
    st = dec.stats()
    dec.rewind(0)
    b = dec.vanilla_decode(32)
    log(f"[full-size] ({d1},{d2}) acc1={st['n_acc1']} acc2={st['n_acc2']} restart={st['n_restart']} "
        f"maxM={st['max_M']}")
    assert np.array_equal(a, b)
    dec.close()


def test_full_size_sixteen_rows_lossless(ouro14):
    from paper_2609_17184_amd import Decoder
    spec, w = ouro14
    Q = 3
    dec = Decoder(spec, w, R=spec.R, d1=1, d2=2, max_seqs=Q, max_ctx=1024, max_slots=16)
    assert dec.pass_kernel and dec.capacity()[0] == 16
    for q in range(Q):
        dec.prefill(q, prompt(spec, 512 - 37 * q, seq=q))
    dec.reset_stats()
    a = dec.decode(24)
    st = dec.stats()
    for q in range(Q):
        dec.rewind(q)
    b = dec.vanilla_decode(24)
    log(f"[full-size rows] maxM={st['max_M']} refused={st['spawn_refused']}")
    assert np.array_equal(a, b)
    dec.close()


def test_full_size_sampling_repeats_under_the_same_key():
    from paper_2609_17184_amd import Decoder
    spec = synth.preset("ouro26")
    w = synth.make_weights(spec, seed=0)
    dec = Decoder(spec, w, R=spec.R, d1=1, d2=2, temperature=1.0, top_p=0.95, seed=2, max_ctx=1024)
    dec.prefill(0, prompt(spec, 512))
    a = dec.decode(24)
    st = dec.stats()
    dec.rewind(0)
    dec.set_seed(2)
    b = dec.decode(24)
    log(f"[full-size sampled] acc1={st['n_acc1']} acc2={st['n_acc2']} restart={st['n_restart']}")
    assert np.array_equal(a, b)
    assert a.min() >= 0 and a.max() < spec.vocab
    dec.close()
