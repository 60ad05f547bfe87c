"""The read-stream probe covers its buffer exactly once per pass (the XOR of
the per-thread results equals the buffer's XOR, ragged sizes included) and
reports a positive rate."""
import numpy as np
import pytest

from gpu_common import log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n_words", [4, 4 * 1000003, 1 << 24])
def test_read_probe_reads_every_word_once(n_words):
    import torch
    from paper_2609_17184_amd.binding import read_bandwidth
    rng = np.random.default_rng(n_words)
    host = rng.integers(-2**31, 2**31, size=n_words, dtype=np.int64).astype(np.int32)
    buf = torch.from_numpy(host).to("cuda:0")
    gbps, xor = read_bandwidth(buf, reps=2)
    got = np.bitwise_xor.reduce(xor.cpu().numpy().view(np.uint32))
    want = np.bitwise_xor.reduce(host.view(np.uint32))
    log(f"[probe] {n_words * 4} bytes: {gbps:.0f} GB/s")
    assert got == want and gbps > 0
