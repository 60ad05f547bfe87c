"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every declared call, sizes the branch pool like the oracle, and rejects bad
configurations before touching the device."""
import ctypes
import os
import re

import pytest

import paper_2609_17184_amd as P
from paper_2609_17184_amd import binding as B
from oracle import theory as T

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    txt = open(os.path.join(ROOT, "include", "loopspec.h")).read()
    return sorted(set(re.findall(r"\b(loopspec_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    L = B.load_library()
    names = _declared()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), n


def test_binding_covers_every_declared_symbol():
    src = open(os.path.join(ROOT, "paper_2609_17184_amd", "binding.py")).read()
    for n in _declared():
        assert f'"{n}"' in src, n


@pytest.mark.parametrize("R,d1,d2", [(32, 2, 8), (4, 1, 2), (4, 1, 3), (4, 2, 3), (32, 4, 8), (32, 4, 12),
                                     (32, 8, 12), (32, 8, 16), (32, 16, 20), (32, 16, 24), (4, 1, 0),
                                     (4, 3, 0), (8, 3, 5)])
def test_worst_case_matches_oracle(R, d1, d2):
    ref = max(T.worst_case_branches(R, d1, d2, accept=1), T.worst_case_branches(R, d1, d2, accept=2))
    assert P.worst_case_branches(R, d1, d2) == ref


def test_worst_case_paper_value_and_invalid():
    assert P.worst_case_branches(32, 2, 8) == 249
    assert P.worst_case_branches(4, 2, 2) == -1
    assert P.worst_case_branches(4, 0, 2) == -1
    assert P.worst_case_branches(4, 1, 4) == -1


def _create(dims, cfg):
    L = B.load_library()
    h = ctypes.c_void_p()
    rc = L.loopspec_create(ctypes.byref(dims), ctypes.byref(cfg), None, ctypes.byref(h))
    msg = (L.loopspec_last_error(h) or b"").decode() if h else ""
    L.loopspec_destroy(h)
    return rc, msg


def _dims(**kw):
    d = dict(hidden=256, n_heads=2, head_dim=128, ffn=704, vocab=1000, n_prelude=0, n_core=2, n_coda=0,
             weight_dtype=B.BF16, tied_head=0, rope_base=1e4, rms_eps=1e-6, max_seqs=1, max_ctx=128)
    d.update(kw)
    return B.Dims(**d)


def _cfg(**kw):
    c = dict(R=4, d1=1, d2=2, temperature=0.0, top_p=1.0, seed=2, max_slots=0)
    c.update(kw)
    return B.Config(**c)


@pytest.mark.parametrize("dims,cfg,needle", [
    (_dims(hidden=250), _cfg(), "hidden must equal"),
    (_dims(head_dim=100, hidden=200, n_heads=2), _cfg(), "head_dim must be"),
    (_dims(head_dim=48, hidden=96, n_heads=2), _cfg(), "head_dim must be"),
    (_dims(ffn=700), _cfg(), "multiples of 32"),
    (_dims(n_core=0), _cfg(), "n_core"),
    (_dims(weight_dtype=7), _cfg(), "weight_dtype"),
    (_dims(), _cfg(d1=0), "d1"),
    (_dims(), _cfg(shared_prefix=2), "shared_prefix"),
    (_dims(), _cfg(d1=2, d2=2), "d2"),
    (_dims(), _cfg(d2=4), "d2"),
    (_dims(), _cfg(top_p=0.0), "top_p"),
    (_dims(), _cfg(temperature=-1.0), "temperature"),
    (_dims(max_ctx=2), _cfg(), "max_ctx"),
    (_dims(), _cfg(temperature=1.0, second_proposal=3), "second_proposal"),
    (_dims(), _cfg(second_proposal=1), "temperature > 0"),
    (_dims(), _cfg(temperature=1.0, d2=0, second_proposal=2), "d2 > 0"),
])
def test_create_rejects_bad_config(dims, cfg, needle):
    rc, msg = _create(dims, cfg)
    assert rc == B.EINVAL and needle in msg


def test_create_rejects_too_many_slots():
    # (32, 2, 8) needs 249 branches per sequence: more than one batched pass holds
    rc, msg = _create(_dims(), _cfg(R=32, d1=2, d2=8))
    assert rc == B.ECAPACITY and "64" in msg


def test_product_does_not_import_oracle():
    pkg = os.path.join(ROOT, "paper_2609_17184_amd")
    for dp, _, fs in os.walk(pkg):
        for f in fs:
            if f.endswith((".py", ".cpp", ".hip", ".h")):
                txt = open(os.path.join(dp, f)).read()
                assert "oracle" not in txt.replace("Oracle", ""), f


def test_read_probe_rejects_bad_arguments():
    """The read-stream probe validates its arguments before any GPU call."""
    L = B.load_library()
    f = ctypes.c_float()
    fake = ctypes.c_void_p(1 << 20)                      # never dereferenced: every case is rejected first
    assert L.loopspec_read_bandwidth(None, 1024, 1, None, fake, ctypes.byref(f)) == B.EINVAL
    assert L.loopspec_read_bandwidth(fake, 1000, 1, None, fake, ctypes.byref(f)) == B.EINVAL   # not 16-aligned
    assert L.loopspec_read_bandwidth(fake, 0, 1, None, fake, ctypes.byref(f)) == B.EINVAL
    assert L.loopspec_read_bandwidth(fake, 1024, 0, None, fake, ctypes.byref(f)) == B.EINVAL
    assert L.loopspec_read_bandwidth(fake, 1 << 36, 1, None, fake, ctypes.byref(f)) == B.EINVAL
    assert L.loopspec_read_bandwidth(fake, 1024, 1, None, None, ctypes.byref(f)) == B.EINVAL
