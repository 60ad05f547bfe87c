"""Proposal-depth planning from the library's teacher-forced readouts (GPU)
against the oracle's depth analysis of the same model and positions."""
import numpy as np
import pytest

from oracle import depths as ODP
from oracle import model as OM
from paper_2609_17184_amd import depths as PD

from gpu_common import log, model, prompt

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,alpha,T,top_p", [("small_bf16", 0.3, 1.0, 0.7), ("tiny", 0.3, 1.0, 0.7),
                                                ("small_bf16", 0.1, 1.0, 1.0)])
def test_select_depths_matches_oracle(name, alpha, T, top_p):
    spec, w = model(name, alpha=alpha)
    toks = prompt(spec, 48)
    k0 = 8
    from paper_2609_17184_amd import Decoder
    dec = Decoder(spec, w, R=spec.R, d1=1, d2=2, max_ctx=64)
    dec.prefill(0, toks[:k0])
    got = PD.select_depths(dec, 0, toks[k0:], T, top_p)
    dec.close()
    lm = OM.LoopedLM(spec, w)
    tv = ODP.teacher_forced_tv(lm, toks, T, top_p, first=k0)
    ref = ODP.predict(tv, spec.R)
    log(f"[depths] {name} alpha={alpha}: gpu tv {got['tv']} -> ({got['d1']},{got['d2']}); "
        f"oracle tv {ref['tv']} -> ({ref['integer_argmin']['d1']},{ref['integer_argmin']['d2']})")
    for r in range(1, spec.R):
        assert abs(got["tv"][r] - tv[r]) < 0.02, (r, got["tv"][r], tv[r])
    f = sorted(ref["f"].values())
    if len(f) > 1 and f[1] - f[0] > 0.02 * f[0]:      # a clear minimum: the same pair
        assert (got["d1"], got["d2"]) == (ref["integer_argmin"]["d1"], ref["integer_argmin"]["d2"])
