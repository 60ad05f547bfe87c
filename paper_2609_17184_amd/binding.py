"""ctypes binding of libloopspec.so (include/loopspec.h).

Argument marshalling only: every step of the decode path runs in the HIP
library.  PyTorch is used to hold the weights in device memory and to provide
a stream.  Importing this module does not need a GPU; creating a Decoder does,
and it fails loudly if the compiled library is missing.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "libloopspec.so")

OK, EINVAL, ENOMEM, EHIP, ECAPACITY, ESTATE, ENUMERIC = 0, -1, -2, -3, -4, -5, -6
F32, BF16 = 0, 1


class Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "hidden", "n_heads", "head_dim", "ffn", "vocab", "n_prelude", "n_core", "n_coda",
        "weight_dtype", "tied_head")] + [
        ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float),
        ("max_seqs", ctypes.c_int32), ("max_ctx", ctypes.c_int32)]


class Config(ctypes.Structure):
    _fields_ = [("R", ctypes.c_int32), ("d1", ctypes.c_int32), ("d2", ctypes.c_int32),
                ("temperature", ctypes.c_float), ("top_p", ctypes.c_float),
                ("seed", ctypes.c_uint64), ("max_slots", ctypes.c_int32), ("per_kernel", ctypes.c_int32),
                ("second_proposal", ctypes.c_int32), ("shared_prefix", ctypes.c_int32)]


LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd")


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in LAYER_TENSORS]


class Weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("head", ctypes.c_void_p), ("layers", ctypes.POINTER(LayerWeights)),
                ("n_layers", ctypes.c_int32)]


class Stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in (
        "steps", "committed", "n_acc1", "n_acc2", "n_restart", "gate_eval", "gate_open",
        "sum_M", "max_M", "spawn_refused", "zero_mass", "tv_d1", "tv_d2", "tv_count")] + [
        ("hist_M", ctypes.c_int64 * 65)]


class CascadeCfg(ctypes.Structure):
    _fields_ = [("vocab", ctypes.c_int32), ("temperature", ctypes.c_float), ("top_p", ctypes.c_float),
                ("seed", ctypes.c_uint64), ("second_proposal", ctypes.c_int32), ("has_second", ctypes.c_int32)]


class Branch(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "active", "seq", "pos", "depth", "token", "parent", "tdone", "x1", "x2", "gate")]


class LoopSpecError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"loopspec error {code}: {msg}")
        self.code = code


_lib = None


def library_path() -> str:
    return _LIB_PATH


def load_library() -> ctypes.CDLL:
    """Load the compiled HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is missing: build it with paper_2609_17184_amd.build.build()")
    L = ctypes.CDLL(_LIB_PATH)
    P = ctypes.POINTER
    i32p = P(ctypes.c_int32)
    sig = {
        "loopspec_create": (ctypes.c_int, [P(Dims), P(Config), ctypes.c_void_p, P(ctypes.c_void_p)]),
        "loopspec_bind_weights": (ctypes.c_int, [ctypes.c_void_p, P(Weights)]),
        "loopspec_prefill": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, i32p, ctypes.c_int32, i32p]),
        "loopspec_rewind": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32]),
        "loopspec_decode_step": (ctypes.c_int, [ctypes.c_void_p, i32p, i32p]),
        "loopspec_decode": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, i32p]),
        "loopspec_vanilla_decode": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, i32p]),
        "loopspec_forced_readout": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, i32p, ctypes.c_int32,
                                                   P(ctypes.c_float), i32p]),
        "loopspec_vanilla_step": (ctypes.c_int, [ctypes.c_void_p, i32p]),
        "loopspec_set_depths": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32]),
        "loopspec_can_set_depths": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32]),
        "loopspec_debug_branch": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, P(Branch), i32p]),
        "loopspec_debug_readout": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                                  P(ctypes.c_float)]),
        "loopspec_decode_profile": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                                   P(ctypes.c_float), i32p, i32p]),
        "loopspec_get_stats": (ctypes.c_int, [ctypes.c_void_p, P(Stats)]),
        "loopspec_reset_stats": (ctypes.c_int, [ctypes.c_void_p]),
        "loopspec_set_seed": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_uint64]),
        "loopspec_last_decode_ms": (ctypes.c_int, [ctypes.c_void_p, P(ctypes.c_float)]),
        "loopspec_capacity": (ctypes.c_int, [ctypes.c_void_p, i32p, i32p]),
        "loopspec_pass_kernel": (ctypes.c_int, [ctypes.c_void_p, i32p]),
        "loopspec_time_kernels": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                                 P(ctypes.c_float)]),
        "loopspec_time_pass": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                              P(ctypes.c_float), i32p]),
        "loopspec_last_error": (ctypes.c_char_p, [ctypes.c_void_p]),
        "loopspec_destroy": (None, [ctypes.c_void_p]),
        "loopspec_version": (ctypes.c_char_p, []),
        "loopspec_worst_case_branches": (ctypes.c_int32, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
        "loopspec_read_bandwidth": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32,
                                                   ctypes.c_void_p, ctypes.c_void_p, P(ctypes.c_float)]),
        "loopspec_cascade_workspace_bytes": (ctypes.c_uint64, [ctypes.c_int32, ctypes.c_int32]),
        "loopspec_cascade_noalloc": (ctypes.c_int, [P(CascadeCfg), ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                                    ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                    ctypes.c_void_p]),
        "loopspec_cascade": (ctypes.c_int, [P(CascadeCfg), ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64,
                                            ctypes.c_void_p]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def worst_case_branches(R: int, d1: int, d2: int) -> int:
    return int(load_library().loopspec_worst_case_branches(R, d1, d2))


def read_bandwidth(buf, reps: int = 10):
    """HBM read rate (GB/s) of a plain stream over the device tensor `buf` and
    the 65536 per-thread XORs of the words read (their XOR is the buffer's).
    A measurement aid: the practical ceiling for the pass's weight stream."""
    import torch
    xor = torch.empty(65536, dtype=torch.int32, device=buf.device)
    stream = torch.cuda.current_stream(buf.device)
    gbps = ctypes.c_float()
    rc = load_library().loopspec_read_bandwidth(ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size(),
                                                int(reps), ctypes.c_void_p(stream.cuda_stream),
                                                ctypes.c_void_p(xor.data_ptr()), ctypes.byref(gbps))
    if rc:
        raise LoopSpecError(rc, "loopspec_read_bandwidth failed")
    return gbps.value, xor


def cascade(z1, z2, zR, keys, temperature: float, top_p: float = 1.0, seed: int = 2, second_proposal: int = 0,
            noalloc: bool = False):
    """Proposal and verification decisions of independent keyed positions
    (loopspec_cascade, or loopspec_cascade_noalloc with noalloc=True).
    z1 / z2 / zR: device fp32 tensors [rows, V] (or [V], shared by every row;
    z2 may be None for the single-proposal pipeline); keys: device int32
    [rows, 2] (sequence, position).  Returns device tensors (out [rows, 6],
    q1 [rows, V], q2 [rows, V])."""
    import torch
    rows = int(keys.shape[0])
    V = int(zR.shape[-1])
    stride = 0 if zR.dim() == 1 else V
    dev = zR.device
    out = torch.full((rows, 6), -1, dtype=torch.int32, device=dev)
    q1 = torch.zeros((rows, V), dtype=torch.float32, device=dev)
    q2 = torch.zeros((rows, V), dtype=torch.float32, device=dev)
    L = load_library()
    cfg = CascadeCfg(V, float(temperature), float(top_p), int(seed), int(second_proposal), int(z2 is not None))
    stream = torch.cuda.current_stream(dev)
    ptr = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else None
    if noalloc:
        rc = L.loopspec_cascade_noalloc(ctypes.byref(cfg), rows, ptr(z1), ptr(z2), ptr(zR), stride, ptr(keys),
                                        ptr(out), ptr(q1), ptr(q2), ctypes.c_void_p(stream.cuda_stream))
    else:
        nbytes = int(L.loopspec_cascade_workspace_bytes(V, rows))
        ws = torch.empty(max(nbytes, 8), dtype=torch.uint8, device=dev)
        rc = L.loopspec_cascade(ctypes.byref(cfg), rows, ptr(z1), ptr(z2), ptr(zR), stride, ptr(keys), ptr(out),
                                ptr(q1), ptr(q2), ptr(ws), nbytes, ctypes.c_void_p(stream.cuda_stream))
    if rc:
        raise LoopSpecError(rc, "loopspec_cascade_noalloc failed" if noalloc else "loopspec_cascade failed")
    return out, q1, q2


def _i32(a) -> ctypes.Array:
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def make_dims(spec, max_seqs: int, max_ctx: int) -> Dims:
    return Dims(spec.hidden, spec.n_heads, spec.head_dim, spec.ffn, spec.vocab, spec.n_prelude,
                spec.n_core, spec.n_coda, BF16 if spec.weight_dtype == "bf16" else F32,
                int(spec.tied_head), spec.rope_base, spec.rms_eps, max_seqs, max_ctx)


class Decoder:
    """One handle of the library: a looped model bound on cuda:0 and a decoding config."""

    def __init__(self, spec, weights: Dict[str, np.ndarray], R: int, d1: int, d2: int,
                 temperature: float = 0.0, top_p: float = 1.0, seed: int = 2, max_seqs: int = 1,
                 max_ctx: int = 1024, max_slots: int = 0, per_kernel: bool = False, shared_prefix: bool = False,
                 second_proposal: int = 0, device: str = "cuda:0"):
        import torch
        self.L = load_library()
        if not torch.cuda.is_available():
            raise RuntimeError("no GPU visible: the LoopSpec library needs an MI355X")
        self.torch = torch
        self.spec = spec
        self.R, self.d1, self.d2 = R, d1, d2
        self.temperature, self.top_p = float(temperature), float(top_p)
        self.max_seqs, self.max_ctx = max_seqs, max_ctx
        self.device = torch.device(device)
        self._h = ctypes.c_void_p()
        # upload the weights (raw bf16 bits or fp32) and keep the tensors alive
        self._t = {}
        for name, a in weights.items():
            a = np.ascontiguousarray(a)
            src = torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a)
            self._t[name] = src.to(self.device)
        torch.cuda.synchronize(self.device)
        self.stream = torch.cuda.Stream(device=self.device)
        self._dims = make_dims(spec, max_seqs, max_ctx)
        self._cfg = Config(R, d1, d2, float(temperature), float(top_p), int(seed), int(max_slots),
                           int(bool(per_kernel)), int(second_proposal), int(bool(shared_prefix)))
        rc = self.L.loopspec_create(ctypes.byref(self._dims), ctypes.byref(self._cfg),
                                    ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(self._h))
        if rc:
            msg = self.error()
            self.close()
            raise LoopSpecError(rc, msg)
        self._bind()

    # -- helpers ----------------------------------------------------------------
    def error(self) -> str:
        if not self._h:
            return ""
        return (self.L.loopspec_last_error(self._h) or b"").decode()

    def _check(self, rc: int) -> None:
        if rc:
            raise LoopSpecError(rc, self.error())

    def _ptr(self, name: str) -> int:
        return self._t[name].data_ptr()

    def _bind(self) -> None:
        sp = self.spec
        names = [f"{st}.{i}" for st, n in sp.stacks for i in range(n)]
        self._layers = (LayerWeights * len(names))(
            *[LayerWeights(*[self._ptr(f"{n}.{t}") for t in LAYER_TENSORS]) for n in names])
        w = Weights(self._ptr("embed"), self._ptr("final_norm"),
                    self._ptr("head") if "head" in self._t else None,
                    self._layers, len(names))
        self._check(self.L.loopspec_bind_weights(self._h, ctypes.byref(w)))

    # -- API ----------------------------------------------------------------------
    def prefill(self, seq: int, ids: Sequence[int]) -> int:
        a, p = _i32(ids)
        out = ctypes.c_int32(-1)
        self._check(self.L.loopspec_prefill(self._h, seq, p, len(a), ctypes.byref(out)))
        return out.value

    def rewind(self, seq: int) -> None:
        self._check(self.L.loopspec_rewind(self._h, seq))

    def decode(self, n: int) -> np.ndarray:
        out = np.full((self.max_seqs, n), -1, np.int32)
        self._check(self.L.loopspec_decode(self._h, n, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
        return out

    def vanilla_decode(self, n: int) -> np.ndarray:
        out = np.full((self.max_seqs, n), -1, np.int32)
        self._check(self.L.loopspec_vanilla_decode(self._h, n,
                                                   out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
        return out

    def decode_step(self):
        tok = np.full(self.max_seqs, -1, np.int32)
        src = np.full(self.max_seqs, -1, np.int32)
        self._check(self.L.loopspec_decode_step(self._h, tok.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                                src.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
        return tok, src

    PROF = {"pass": 0, "qkv": 1, "attention": 2, "o_proj": 3, "gate_up": 4, "down": 5, "head": 6}

    def decode_profile(self, n: int, kind: str, max_launches: int = 1 << 16):
        """Decode n tokens with HIP events in the dispatch of every launch of one kernel kind:
        (ms [launches], info [launches, 3] = (rows, key/value positions read, step))."""
        ms = np.zeros(max_launches, np.float32)
        info = np.zeros((max_launches, 3), np.int32)
        cnt = ctypes.c_int32()
        self._check(self.L.loopspec_decode_profile(
            self._h, n, self.PROF[kind], max_launches, ms.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
            info.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), ctypes.byref(cnt)))
        k = min(cnt.value, max_launches)
        return ms[:k], info[:k]

    def set_depths(self, d1: int, d2: int) -> None:
        """Switch the proposal depths between decode calls (lossless)."""
        self._check(self.L.loopspec_set_depths(self._h, int(d1), int(d2)))
        self.d1, self.d2 = int(d1), int(d2)

    def can_set_depths(self, d1: int, d2: int) -> int:
        """0 if set_depths(d1, d2) would succeed now, else its error code."""
        return int(self.L.loopspec_can_set_depths(self._h, int(d1), int(d2)))

    def vanilla_step(self) -> np.ndarray:
        """One vanilla token per prefilled sequence (-1 for the others)."""
        tok = np.full(self.max_seqs, -1, np.int32)
        self._check(self.L.loopspec_vanilla_step(self._h, tok.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
        return tok

    def branch(self, slot: int, prefix: bool = True):
        """(info dict, token prefix positions 0..pos or None) of a branch slot."""
        b = Branch()
        buf = np.full(self.max_ctx, -1, np.int32) if prefix else None
        self._check(self.L.loopspec_debug_branch(
            self._h, slot, ctypes.byref(b), buf.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)) if prefix else None))
        info = {n: getattr(b, n) for n, _ in Branch._fields_}
        if not info["active"] or buf is None:
            return info, None
        return info, buf[:info["pos"] + 1].copy()

    def branches(self):
        """Every live branch: list of (slot, info, prefix)."""
        out = []
        for slot in range(self.capacity()[0]):
            info, pre = self.branch(slot)
            if info["active"]:
                out.append((slot, info, pre))
        return out

    def debug_readout(self, slot: int, depth: int) -> np.ndarray:
        """Readout logits [V] of a branch's newest token at a depth <= its current depth."""
        lg = np.zeros(self.spec.vocab, np.float32)
        self._check(self.L.loopspec_debug_readout(self._h, slot, depth,
                                                  lg.ctypes.data_as(ctypes.POINTER(ctypes.c_float))))
        return lg

    def forced_readout(self, seq: int, ids: Sequence[int], logits: bool = True):
        a, p = _i32(ids)
        n = len(a)
        lg = np.zeros((n, self.R, self.spec.vocab), np.float32) if logits else None
        am = np.zeros((n, self.R), np.int32)
        self._check(self.L.loopspec_forced_readout(
            self._h, seq, p, n,
            lg.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if logits else None,
            am.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
        return lg, am

    def stats(self) -> dict:
        s = Stats()
        self._check(self.L.loopspec_get_stats(self._h, ctypes.byref(s)))
        d = {n: getattr(s, n) for n, _ in Stats._fields_ if n != "hist_M"}
        d["hist_M"] = list(s.hist_M)
        return d

    def set_seed(self, seed: int) -> None:
        self._check(self.L.loopspec_set_seed(self._h, int(seed)))

    def reset_stats(self) -> None:
        self._check(self.L.loopspec_reset_stats(self._h))

    def last_decode_ms(self) -> float:
        v = ctypes.c_float()
        self._check(self.L.loopspec_last_decode_ms(self._h, ctypes.byref(v)))
        return v.value

    KERNELS = ("qkv", "attention", "o_proj", "gate_up", "down")

    def time_kernels(self, M: int, reps: int = 3) -> dict:
        """Average ms per launch of each recurrent-pass kernel (HIP events)."""
        ms = (ctypes.c_float * 5)()
        self._check(self.L.loopspec_time_kernels(self._h, M, reps, ms))
        return dict(zip(self.KERNELS, list(ms)))

    def time_pass(self, M: int, reps: int = 5):
        """(ms per launch of the core-stack decode pass at M rows, persistent kernel used)."""
        ms, fused = ctypes.c_float(), ctypes.c_int32()
        self._check(self.L.loopspec_time_pass(self._h, M, reps, ctypes.byref(ms), ctypes.byref(fused)))
        return ms.value, bool(fused.value)

    @property
    def pass_kernel(self) -> bool:
        """True when decode passes run as the persistent pass kernel."""
        return self.pass_attention != 0

    @property
    def pass_attention(self) -> int:
        """0: per-kernel launches; persistent pass with attention 1: per (row,
        head) workgroup, 2: (row, head, chunk) tasks (long contexts)."""
        v = ctypes.c_int32()
        self._check(self.L.loopspec_pass_kernel(self._h, ctypes.byref(v)))
        return int(v.value)

    def capacity(self):
        a, b = ctypes.c_int32(), ctypes.c_int32()
        self._check(self.L.loopspec_capacity(self._h, ctypes.byref(a), ctypes.byref(b)))
        return a.value, b.value

    def close(self) -> None:
        if self._h:
            self.L.loopspec_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
