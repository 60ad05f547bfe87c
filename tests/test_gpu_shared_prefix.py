"""Shared-prefix decode attention (loopspec_config.shared_prefix) on the
per-kernel path.

The rows of one sequence at one recurrent depth read the same committed keys
and values (KV cache management of the pipelined decode); the attention
launch groups them, loads each committed chunk once and scores it against
every member's query.  A row's arithmetic is the same whether it runs in a
group or alone, so:

* the readout of every branch that shared a group, taken from the hidden
  state the grouped decode step produced, is bit-identical to the readout of
  the same prefix at the same depth computed alone (teacher-forced on the
  vanilla schedule, one row per pass), for committed prefixes of 4 and of
  18 chunks, on the 16-row and the 64-row GEMM paths;
* greedy LoopSpec stays bit-identical to vanilla decoding.
The element-wise comparison of such branches with the fp64 oracle is in
test_gpu_debug (its shared-prefix cases)."""
import collections

import numpy as np
import pytest

from gpu_common import log, model, prompt

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n_prompt,max_ctx,max_slots", [(200, 2100, 24), (1100, 2600, 0), (1100, 2600, 24)])
def test_grouped_rows_equal_rows_computed_alone(n_prompt, max_ctx, max_slots):
    from paper_2609_17184_amd import Decoder
    spec, w = model("small_bf16")
    pr = prompt(spec, n_prompt)
    dec = Decoder(spec, w, R=spec.R, d1=1, d2=2, max_ctx=max_ctx, max_slots=max_slots, per_kernel=True,
                  shared_prefix=True)
    assert not dec.pass_kernel
    dec.prefill(0, pr)
    samples, groups = [], []
    for step in range(10):
        dec.decode_step()
        by_depth = collections.defaultdict(list)
        for slot, info, prefix in dec.branches():
            if info["depth"] >= 1:
                by_depth[info["depth"]].append((slot, prefix))
        for depth, members in by_depth.items():
            if len(members) < 2:
                continue
            groups.append((step + 1, depth, len(members)))
            for slot, prefix in members:
                samples.append((prefix, depth, dec.debug_readout(slot, depth)))
    log(f"[shared prefix] prompt {n_prompt} slots {dec.capacity()[0]}: groups (step, depth, rows) {groups}")
    assert groups, "no two branches of the sequence shared a depth"
    n0 = len(pr)
    for prefix, depth, lg in samples:
        ids = [int(t) for t in prefix[n0:]]
        ref, _ = dec.forced_readout(0, ids)
        alone = ref[len(ids) - 1, depth - 1]
        assert np.array_equal(alone, lg), (len(ids), depth, float(np.abs(alone - lg).max()))
    log(f"[shared prefix] {len(samples)} grouped readouts bit-identical to the same prefixes computed alone")
    dec.rewind(0)
    a = dec.decode(24)[0]
    dec.rewind(0)
    b = dec.vanilla_decode(24)[0]
    dec.close()
    assert list(a) == list(b)
