"""The Raven/Huginn-shaped width on the GPU against the fp64 oracle.

Hidden 5280 (55 heads of 96), FFN 17920, vocabulary 65536, bf16: the widths
of the benchmarked prelude / core / coda model, with one block per stack and
R = 4 so that the fp64 oracle stays within seconds.  Every decode GEMM of
this width streams K = 5280 or 17920 in more k steps than one wave holds,
so the weight stream is split over several workgroups per output tile; the
test checks the readout logits at every depth (teacher-forced along the
oracle's greedy trajectory) and the first token after prefill, with a branch
pool of at most 16 slots (16-row stream-K launches), of 24 (32-row launches)
and of 64 (64-row launches): at this width the QKV, gate/up, down and LM-head
launches of more than 16 rows stream their weights stream-K too, the O
projection takes the 64-row tiles.  Prefill runs 64-row launches.
Sec. 3.1 (Eq. loop-recurrence), Fig. 2."""
import numpy as np
import pytest

import synth
from oracle import dist as OD

from gpu_common import MARGIN, log, oracle_trajectory, prompt
from test_gpu_parity import _check_logits

pytestmark = pytest.mark.gpu

N_PROMPT, N_TOK, R = 70, 3, 4


@pytest.fixture(scope="module")
def raven_width():
    spec = synth.preset("raven", n_prelude=1, n_core=1, n_coda=1, R=R)
    log("[raven-width] weights ...")
    w = synth.make_weights(spec, seed=0)
    pr = prompt(spec, N_PROMPT)
    log("[raven-width] fp64 oracle ...")
    toks, ref, z0 = oracle_trajectory(spec, w, pr, N_TOK)
    log(f"[raven-width] oracle tokens {toks}")
    return spec, w, pr, toks, ref, z0


@pytest.mark.timeout(900)
@pytest.mark.parametrize("max_slots", [0, 24, 64])
def test_raven_width_readouts_match_oracle(raven_width, max_slots):
    from paper_2609_17184_amd import Decoder
    spec, w, pr, toks, ref, z0 = raven_width
    dec = Decoder(spec, w, R=R, d1=1, d2=2, max_ctx=128, max_slots=max_slots)
    slots = dec.capacity()[0]
    log(f"[raven-width] slots {slots} (direct GEMM path: {slots <= 16}); persistent pass {dec.pass_kernel}")
    assert (slots <= 16) == (max_slots == 0)
    first = dec.prefill(0, pr)
    m0 = OD.top2_margin(z0)
    log(f"[raven-width] first token gpu {first} oracle {toks[0]} (oracle top-2 margin {m0:.3f})")
    if m0 > MARGIN["bf16"]:
        assert first == toks[0]
    lg, _ = dec.forced_readout(0, toks)
    _check_logits(lg, ref, "bf16", f"raven width, slots {slots}: logits [{N_TOK}, R, V]")
    dec.close()
