"""fp64 CPU reference of a Looped Transformer forward pass.

TEST INFRASTRUCTURE: part of the CPU oracle.  Only tests/, the smoke check and
the benchmark's CPU-baseline leg may import it; the product path never does.

What it computes (LoopSpec paper, Preliminaries / Looped Transformers,
Eq. loop-recurrence):
    H^(0) = P(X),   H^(r) = B(H^(r-1)) for r = 1..R,   p_r = C(H^(r)).
Ouro-style models: P = token embedding, C = final RMSNorm + LM head.
Raven-style models: P = embedding + prelude blocks, C = coda blocks + final
RMSNorm + LM head (Fig. 2).

Readings where the paper is silent (the model family is only abstracted):
  * block: pre-RMSNorm, x += Attn(RMSNorm(x)); x += FFN(RMSNorm(x)) with the
    residual scale already folded into W_o and W_d by the generator;
    RMSNorm(x) = x / sqrt(mean(x^2) + eps) * g;
  * attention: multi-head, kv heads = heads, causal softmax(q k^T / sqrt(dh)) v;
  * RoPE: rotate-half layout, pairs (i, i + dh/2), angle pos * base^(-2i/dh),
    absolute 0-based positions, the same at every recurrent depth;
  * FFN: SwiGLU, W_d (silu(W_g n) * (W_u n));
  * KV scope: attention at recurrent depth r and layer l reads the keys and
    values of the prefix computed at the same (r, l); every depth has its own
    cache (implementation details, KV cache management).  Coda layers keep one
    cache per readout depth; the prelude has one cache.

Weights are the synthetic bf16 (or fp32) values; all arithmetic is fp64.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Tuple

import numpy as np

import synth


# ----------------------------------------------------------------------------
# textbook operations
# ----------------------------------------------------------------------------
def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def rope(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """x: [T, H, dh]; rotate-half RoPE at absolute positions pos [T]."""
    dh = x.shape[-1]
    half = dh // 2
    inv = base ** (-(2.0 * np.arange(half)) / dh)
    ang = np.asarray(pos, np.float64)[:, None] * inv[None, :]          # [T, half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def causal_attention(q, K, V, qpos, kpos):
    """q [Tq,H,dh], K/V [Tk,H,dh]; query at qpos attends to keys with kpos <= qpos."""
    dh = q.shape[-1]
    s = np.einsum("qhd,khd->hqk", q, K) / np.sqrt(dh)
    mask = np.asarray(kpos)[None, None, :] > np.asarray(qpos)[None, :, None]
    s = np.where(mask, -np.inf, s)
    s = s - s.max(axis=-1, keepdims=True)
    w = np.exp(s)
    w = w / w.sum(axis=-1, keepdims=True)
    return np.einsum("hqk,khd->qhd", w, V)


def silu(x):
    return x / (1.0 + np.exp(-x))


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------
class Weights64:
    """fp64 view of the synthetic tensors, converted on first use and cached."""

    def __init__(self, spec: synth.ModelSpec, raw: Dict[str, np.ndarray], cache: bool = True):
        self.spec, self.raw, self.cache = spec, raw, cache
        self._c: Dict[str, np.ndarray] = {}

    def __getitem__(self, name: str) -> np.ndarray:
        a = self._c.get(name)
        if a is not None:
            return a
        if name == "head" and self.spec.tied_head:
            return self["embed"]
        r = self.raw[name]
        a = (synth.bf16_bits_to_f32(r) if r.dtype == np.uint16 else r).astype(np.float64)
        if self.cache:
            self._c[name] = a
        return a


# ----------------------------------------------------------------------------
# the looped model
# ----------------------------------------------------------------------------
Space = Tuple[str, int]          # ("P", 0) prelude, ("B", r) core depth r, ("C", r) coda at readout r


class Node:
    """A prefix.  Holds, for its own new positions, the keys/values of every
    (space, layer) and the hidden state after every recurrent depth."""

    __slots__ = ("parent", "tokens", "pos0", "kv", "hidden", "memo", "children")

    def __init__(self, parent, tokens, pos0):
        self.parent: Optional[Node] = parent
        self.tokens = list(tokens)          # tokens at positions pos0 .. pos0+len-1
        self.pos0 = pos0
        self.kv: Dict[Tuple[Space, int], Tuple[np.ndarray, np.ndarray]] = {}
        self.hidden: List[np.ndarray] = []  # per depth 0..R: [len, h]
        self.memo: Dict[int, np.ndarray] = {}
        self.children: Dict[int, Node] = {}

    @property
    def last_pos(self) -> int:
        return self.pos0 + len(self.tokens) - 1

    def chain(self) -> List["Node"]:
        out, n = [], self
        while n is not None:
            out.append(n)
            n = n.parent
        return out[::-1]

    def prefix(self) -> List[int]:
        return [t for n in self.chain() for t in n.tokens]


class LoopedLM:
    def __init__(self, spec: synth.ModelSpec, raw: Dict[str, np.ndarray], cache64: bool = True):
        self.spec = spec
        self.W = Weights64(spec, raw, cache64)
        self.n_fwd_tokens = 0

    # -- one pre-norm block over new rows x [T,h] at positions pos [T] ---------
    def _block(self, stack: str, i: int, x, pos, ctx_k, ctx_v, ctx_pos):
        sp, W = self.spec, self.W
        H, dh = sp.n_heads, sp.head_dim
        p = f"{stack}.{i}."
        n = rms_norm(x, W[p + "attn_norm"], sp.rms_eps)
        q = (n @ W[p + "wq"].T).reshape(-1, H, dh)
        k = (n @ W[p + "wk"].T).reshape(-1, H, dh)
        v = (n @ W[p + "wv"].T).reshape(-1, H, dh)
        q = rope(q, pos, sp.rope_base)
        k = rope(k, pos, sp.rope_base)
        K = np.concatenate([ctx_k, k]) if ctx_k is not None else k
        V = np.concatenate([ctx_v, v]) if ctx_v is not None else v
        kp = np.concatenate([ctx_pos, pos]) if ctx_pos is not None else pos
        a = causal_attention(q, K, V, pos, kp).reshape(-1, H * dh)
        x = x + a @ W[p + "wo"].T
        n2 = rms_norm(x, W[p + "ffn_norm"], sp.rms_eps)
        x = x + (silu(n2 @ W[p + "wg"].T) * (n2 @ W[p + "wu"].T)) @ W[p + "wd"].T
        return x, k, v

    def _ctx(self, parent: Optional[Node], space: Space, layer: int):
        """Keys/values/positions of the whole prefix held by `parent`'s chain."""
        if parent is None:
            return None, None, None
        ks, vs, ps = [], [], []
        for n in parent.chain():
            k, v = n.kv[(space, layer)]
            ks.append(k)
            vs.append(v)
            ps.append(np.arange(n.pos0, n.pos0 + len(n.tokens)))
        return np.concatenate(ks), np.concatenate(vs), np.concatenate(ps)

    def _stack(self, stack: str, n_layers: int, space: Space, x, pos, node: Node):
        for i in range(n_layers):
            ck, cv, cp = self._ctx(node.parent, space, i)
            x, k, v = self._block(stack, i, x, pos, ck, cv, cp)
            node.kv[(space, i)] = (k, v)
        return x

    def _run(self, node: Node) -> Node:
        sp = self.spec
        pos = np.arange(node.pos0, node.pos0 + len(node.tokens))
        x = self.W["embed"][np.asarray(node.tokens)]
        x = self._stack("prelude", sp.n_prelude, ("P", 0), x, pos, node)
        node.hidden = [x]
        for r in range(1, sp.R + 1):
            x = self._stack("core", sp.n_core, ("B", r), x, pos, node)
            node.hidden.append(x)
        self.n_fwd_tokens += len(node.tokens)
        return node

    # -- public ----------------------------------------------------------------
    def prefill(self, tokens) -> Node:
        """Prompt x_{1:n} through P and R applications of B (positions 0..n-1)."""
        return self._run(Node(None, tokens, 0))

    def extend(self, node: Node, token: int) -> Node:
        """The prefix node || token, with all R depths computed (memoised)."""
        token = int(token)
        c = node.children.get(token)
        if c is None:
            c = self._run(Node(node, [token], node.last_pos + 1))
            node.children[token] = c
        return c

    def _coda(self, node: Node, r: int):
        """Coda keys/values at readout depth r for `node` (and, first, its chain)."""
        sp = self.spec
        space = ("C", r)
        for n in node.chain():
            if (space, 0) in n.kv:
                continue
            pos = np.arange(n.pos0, n.pos0 + len(n.tokens))
            out = self._stack("coda", sp.n_coda, space, n.hidden[r], pos, n)
            n.kv[(space, "out")] = out        # coda output rows of this node at depth r
        return node.kv[(space, "out")]

    def logits(self, node: Node, r: int) -> np.ndarray:
        """Readout logits C(H^(r)) for the next token after `node`'s prefix."""
        if r in node.memo:
            return node.memo[r]
        sp = self.spec
        x = self._coda(node, r) if sp.n_coda else node.hidden[r]
        x = rms_norm(x[-1], self.W["final_norm"], sp.rms_eps)
        z = self.W["head"] @ x
        node.memo[r] = z
        return z

    def forget(self, node: Node, keep: Node) -> None:
        """Drop `node`'s other children (memory only; results are unaffected)."""
        node.children = {t: c for t, c in node.children.items() if c is keep}

    # -- cache-free recomputation -------------------------------------------------
    def forward_full(self, tokens) -> Dict[int, np.ndarray]:
        """Logits at every depth for every position, recomputing the whole sequence
        with no cache: returns {r: [T, V]}."""
        sp = self.spec
        T = len(tokens)
        pos = np.arange(T)

        def stack(name, n_layers, x):
            for i in range(n_layers):
                x, _, _ = self._block(name, i, x, pos, None, None, None)
            return x

        x = stack("prelude", sp.n_prelude, self.W["embed"][np.asarray(tokens)])
        out = {}
        for r in range(1, sp.R + 1):
            x = stack("core", sp.n_core, x)
            y = stack("coda", sp.n_coda, x) if sp.n_coda else x
            out[r] = rms_norm(y, self.W["final_norm"], sp.rms_eps) @ self.W["head"].T
        return out
