"""The allocation-free cascade entry point against the one with a workspace.

loopspec_cascade_noalloc keeps its barrier state in a static device array
instead of a caller's workspace; it must take exactly the decisions and give
exactly the distributions loopspec_cascade gives (the same kernels), also on
two calls in a row where the second is smaller (the array keeps the first
call's contents), with one shard per row (V = 16) and with sixteen
(V = 49152, more rows than one launch holds)."""
import numpy as np
import pytest

from gpu_common import log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("V,rows", [(49152, (150, 40)), (16, (3000, 500))])
def test_cascade_noalloc_equals_workspace_entry_point(V, rows):
    import torch
    from paper_2609_17184_amd.binding import cascade
    for call, n in enumerate(rows):
        rng = np.random.default_rng(77 + call + V)
        base = rng.standard_normal((n, V)).astype(np.float32) * 3.0
        z = [torch.from_numpy(base + rng.standard_normal((n, V)).astype(np.float32) * s).cuda()
             for s in (2.0, 1.5, 1.0)]
        keys = torch.from_numpy(np.stack([np.arange(n) % 5, 10 + np.arange(n)], 1).astype(np.int32)).cuda()
        for variant, top_p in ((0, 0.9), (2, 1.0)):
            ref = cascade(z[0], z[1], z[2], keys, 1.0, top_p, 3 + call, variant)
            got = cascade(z[0], z[1], z[2], keys, 1.0, top_p, 3 + call, variant, noalloc=True)
            for a, b, what in zip(got, ref, ("decisions", "q1", "q2")):
                assert torch.equal(a, b), (V, n, variant, what)
            src = ref[0][:, 1].cpu().numpy()
            log(f"[noalloc] V={V} call {call} rows={n} variant={variant}: equal; sources "
                f"{np.bincount(src, minlength=3).tolist()}")
