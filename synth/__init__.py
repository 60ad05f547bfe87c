"""Seeded synthetic inputs shared by the fp64 oracle and the HIP path.

This module only *draws data*: model shapes, weights, prompts.  It contains
none of the looped-transformer or LoopSpec arithmetic, so both the oracle and
the GPU binding may import it without sharing any of the method's code.

Weights follow the synthetic recipe for the paper's model families (Ouro-style:
all blocks recurrent; Raven-style: prelude / recurrent core / coda, Fig. 2 and
the Looped Transformers preliminaries): every matrix is drawn N(0, 0.02); the
residual-branch scale alpha is folded into the two matrices that write into the
residual stream (attention output and FFN down projection) *before* rounding,
so a block is the plain pre-norm form ``x += W_o(...)``, ``x += W_d(...)``.
bf16 models are stored as raw bf16 bit patterns (``numpy.uint16``), rounded to
nearest-even from the fp32 draw; fp32 models are stored as ``numpy.float32``.
"""
from __future__ import annotations

import dataclasses
import os
import zlib
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Iterator, Tuple

import numpy as np

__all__ = [
    "ModelSpec", "PRESETS", "preset", "weight_names", "make_weights",
    "make_prompt", "bf16_bits_to_f32", "f32_to_bf16_bits", "tensor_shape",
]


@dataclasses.dataclass(frozen=True)
class ModelSpec:
    hidden: int
    n_heads: int
    head_dim: int
    ffn: int
    vocab: int
    n_prelude: int
    n_core: int
    n_coda: int
    R: int
    weight_dtype: str = "bf16"      # "bf16" or "f32"
    tied_head: bool = False
    alpha: float = 0.3
    rope_base: float = 10000.0
    rms_eps: float = 1e-6
    std: float = 0.02
    gain_noise: float = 0.0        # RMSNorm gains = 1 + gain_noise * N(0,1)

    def __post_init__(self):
        if self.hidden != self.n_heads * self.head_dim:
            raise ValueError("hidden must equal n_heads * head_dim")
        if self.head_dim % 2:
            raise ValueError("head_dim must be even (RoPE pairs)")
        if self.weight_dtype not in ("bf16", "f32"):
            raise ValueError("weight_dtype must be 'bf16' or 'f32'")

    def replace(self, **kw) -> "ModelSpec":
        return dataclasses.replace(self, **kw)

    @property
    def stacks(self) -> Tuple[Tuple[str, int], ...]:
        return (("prelude", self.n_prelude), ("core", self.n_core), ("coda", self.n_coda))

    def n_params(self) -> int:
        return sum(int(np.prod(tensor_shape(self, n))) for n in weight_names(self))


PRESETS: Dict[str, ModelSpec] = {
    # 2 shared pre-RMSNorm blocks looped R=4, h=256, 4x64 heads, FFN 1024, V=4096, tied, fp32
    "tiny": ModelSpec(256, 4, 64, 1024, 4096, 0, 2, 0, R=4, weight_dtype="f32",
                      tied_head=True, alpha=0.3),
    # Ouro-1.4B-shaped: 24 shared blocks, R=4, h=2048, 16x128, FFN 5632, V=49152, bf16
    "ouro14": ModelSpec(2048, 16, 128, 5632, 49152, 0, 24, 0, R=4, alpha=0.3),
    # Ouro-2.6B-shaped: 48 shared blocks
    "ouro26": ModelSpec(2048, 16, 128, 5632, 49152, 0, 48, 0, R=4, alpha=0.3),
    # Raven/Huginn-shaped: 2 prelude, 4 core x R=32, 2 coda; h=5280, 55x96, FFN 17920, V=65536
    "raven": ModelSpec(5280, 55, 96, 17920, 65536, 2, 4, 2, R=32, alpha=0.3),
    # small shapes used by tests (fast on CPU; several MFMA tiles and ragged tails on GPU)
    "micro": ModelSpec(32, 2, 16, 64, 16, 0, 1, 0, R=4, weight_dtype="f32", tied_head=False,
                       alpha=0.3, std=0.3),
    "small_bf16": ModelSpec(256, 2, 128, 704, 1000, 0, 2, 0, R=4, alpha=0.3),
    "small_raven": ModelSpec(192, 2, 96, 512, 800, 1, 2, 1, R=8, alpha=0.3),
}


def preset(name: str, **overrides) -> ModelSpec:
    return PRESETS[name].replace(**overrides) if overrides else PRESETS[name]


def weight_names(spec: ModelSpec) -> Iterator[str]:
    yield "embed"
    for stack, n in spec.stacks:
        for i in range(n):
            for t in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd"):
                yield f"{stack}.{i}.{t}"
    yield "final_norm"
    if not spec.tied_head:
        yield "head"


def tensor_shape(spec: ModelSpec, name: str) -> Tuple[int, ...]:
    h, F, V = spec.hidden, spec.ffn, spec.vocab
    if name in ("embed", "head"):
        return (V, h)
    if name == "final_norm":
        return (h,)
    kind = name.rsplit(".", 1)[1]
    return {
        "attn_norm": (h,), "ffn_norm": (h,),
        "wq": (h, h), "wk": (h, h), "wv": (h, h), "wo": (h, h),
        "wg": (F, h), "wu": (F, h), "wd": (h, F),
    }[kind]


_CHUNK = 1 << 22   # elements per independently seeded chunk (thread-count independent)


def _rng(seed: int, name: str, chunk: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence([int(seed) & 0xFFFFFFFF, zlib.crc32(name.encode()), chunk])
    return np.random.Generator(np.random.PCG64(ss))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to the nearest bf16 (ties to even); returns raw uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _fill(spec: ModelSpec, seed: int, name: str, out: np.ndarray, c: int) -> None:
    """Draw chunk c of tensor `name` into the flat output array."""
    kind = name.rsplit(".", 1)[-1]
    lo = c * _CHUNK
    hi = min(out.size, lo + _CHUNK)
    rng = _rng(seed, name, c)
    if kind in ("attn_norm", "ffn_norm", "final_norm"):
        a = np.ones(hi - lo, np.float32)
        if spec.gain_noise:
            a += np.float32(spec.gain_noise) * rng.standard_normal(hi - lo, dtype=np.float32)
    else:
        a = rng.standard_normal(hi - lo, dtype=np.float32)
        a *= np.float32(spec.std)
        if kind in ("wo", "wd"):
            a *= np.float32(spec.alpha)
    out[lo:hi] = f32_to_bf16_bits(a) if out.dtype == np.uint16 else a


def make_weights(spec: ModelSpec, seed: int = 0, threads: int = 0) -> Dict[str, np.ndarray]:
    """All tensors of the synthetic model, keyed by name, [out][in] row-major.

    bf16 models: uint16 bf16 bit patterns.  fp32 models: float32.  Each tensor
    is drawn in fixed 4M-element chunks, each chunk from its own seed derived
    from (seed, tensor name, chunk index), so the values do not depend on the
    number of threads used.
    """
    dt = np.uint16 if spec.weight_dtype == "bf16" else np.float32
    out: Dict[str, np.ndarray] = {}
    jobs = []
    for name in weight_names(spec):
        shape = tensor_shape(spec, name)
        flat = np.empty(int(np.prod(shape)), dt)
        out[name] = flat.reshape(shape)
        for c in range((flat.size + _CHUNK - 1) // _CHUNK):
            jobs.append((name, flat, c))
    nt = threads or min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(nt) as ex:
        list(ex.map(lambda j: _fill(spec, seed, j[0], j[1], j[2]), jobs))
    return out


def make_prompt(vocab: int, n: int, seed: int = 1, seq: int = 0) -> np.ndarray:
    """Prompt token ids drawn uniformly from [0, vocab)."""
    rng = _rng(seed, f"prompt/{seq}")
    return rng.integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)
