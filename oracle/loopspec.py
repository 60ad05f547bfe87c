"""LoopSpec decoding (Alg. 1 of the paper) and vanilla looped decoding, on CPU.

TEST INFRASTRUCTURE: part of the CPU oracle.  Only tests/, the smoke check and
the benchmark's CPU-baseline leg may import it.

The simulator follows Alg. 1 ("LoopSpec with two proposals") and Sec. 4:
  * after prefill, the first token x ~ C(H) is committed and a branch is spawned
    on prompt || x at depth 0;
  * every step, all active branches advance one recurrent depth (batched
    recurrence, Sec. 4.2 step 1);
  * a branch reaching d1 reads out q1 = p_{d1}, draws x1 ~ q1 and spawns a child
    on X || x1 (early drafting, Sec. 4.2 step 2);
  * a branch reaching d2 reads out q2~ = p_{d2}; if q2~(x1) < q1(x1) (gating,
    Eq. adaptive-gate) it draws x2 ~ q2 = q2~ (-) q1 (Eq. residual-proposal) and
    spawns a second child;
  * the deepest branch, if it reached R, verifies its proposals against p_R in
    order (Verify: accept x_j w.p. min{1, rho(x_j)/q_j(x_j)}, else
    rho <- rho (-) q_j), else resamples x ~ rho and spawns a fresh branch; the
    token is committed and the set is re-rooted at the chosen child (Reroot).

A readout provider supplies p_r for a prefix.  The model-backed provider wraps
the fp64 LoopedLM; tests also use synthetic providers (any function of the
prefix and the depth), because the decision logic only depends on those values.

Readings (see the distribution module for T / top-p / residual / draws):
  * randomness: every draw is keyed by (seed, sequence, position of the token
    being decided, event); see the Philox module;
  * order inside a step is Alg. 1's: advance and propose for every branch of
    the step's set, then verify the deepest one; children spawned this step
    first advance on the next step; children spawned inside a subtree pruned in
    the same step are dropped with it;
  * only the root can reach R (descendants are strictly shallower); asserted;
  * stopping: after `n_tokens` committed tokens, counting the first token that
    prefill commits; the rest of the speculative tree is discarded;
  * changing (d1, d2) while decoding (re-planning the depths from measured TV,
    Sec. 4.1 Observation with Theorem 2): the pair switches right after the
    step that commits a given token count.  The speculative branches and the
    root's proposals are dropped (they were drawn under the old pair); a root
    below the new d1 keeps its depth, one at or past it restarts at depth 0.
    Every committed token is still verified against p_R, so decoding stays
    lossless;
  * TV(p_R, p_d1) and TV(p_R, p_d2) of each verified root are recorded (the
    measurements the re-planning uses); with greedy readouts they are 0 or 1.
"""
from __future__ import annotations

import dataclasses
from typing import Any, Dict, List, Optional, Tuple

import numpy as np

from . import dist as D
from . import philox as PX


# ----------------------------------------------------------------------------
# draws
# ----------------------------------------------------------------------------
class Sampler:
    """Temperature/top-p readout distributions and keyed random decisions."""

    def __init__(self, temperature: float = 0.0, top_p: float = 1.0, seed: int = 2, seq: int = 0):
        self.T, self.top_p, self.seed, self.seq = float(temperature), float(top_p), seed, seq
        self.decisions: List[tuple] = []   # (kind, position, margin) for fragility analysis
        self.step = 0

    @property
    def greedy(self) -> bool:
        return self.T == 0.0

    def dist(self, logits: np.ndarray) -> np.ndarray:
        if self.greedy:
            self.decisions.append(("argmax", self.step, D.top2_margin(logits)))
        elif self.top_p < 1.0:
            # distance of the nearest ranked-before mass to the top-p cut
            z = np.asarray(logits, np.float64) / self.T
            e = np.exp(z - z.max())
            p = e / e.sum()
            order = np.lexsort((np.arange(p.size), -p))
            before = np.cumsum(p[order]) - p[order]
            self.decisions.append(("topp", self.step, float(np.min(np.abs(before - self.top_p)))))
        return D.readout_dist(logits, self.T, self.top_p)

    def draw(self, w: np.ndarray, event: int, position: int) -> int:
        if self.greedy:
            # a one-hot distribution's only support point (what any race returns)
            nz = np.flatnonzero(w > 0)
            if nz.size == 1:
                return int(nz[0])
        u = PX.vocab_uniforms(self.seed, self.seq, position, event, w.size)
        x, gap = D.race_sample(w, u)
        self.decisions.append(("race", self.step, gap))
        return x

    def accept(self, ratio: float, event: int, position: int) -> bool:
        a = min(1.0, ratio)
        if self.greedy and a in (0.0, 1.0):
            return a == 1.0          # U in [0,1): U < 1 always, U < 0 never
        u = PX.scalar_uniform(self.seed, self.seq, position, event)
        self.decisions.append(("accept", self.step, abs(u - a)))
        return u < a


# ----------------------------------------------------------------------------
# readout providers
# ----------------------------------------------------------------------------
class ModelReadouts:
    """p_r(.|X) from the fp64 looped model, with the sampler's T / top-p."""

    def __init__(self, lm, prompt):
        self.lm = lm
        self.prompt = [int(t) for t in prompt]
        self._root = None

    def root(self):
        if self._root is None:
            self._root = self.lm.prefill(self.prompt)
        return self._root

    def child(self, node, token: int):
        return self.lm.extend(node, token)

    def logits(self, node, r: int) -> np.ndarray:
        return self.lm.logits(node, r)

    def position(self, node) -> int:
        return node.last_pos

    def release(self, node, keep) -> None:
        self.lm.forget(node, keep)


# ----------------------------------------------------------------------------
# results
# ----------------------------------------------------------------------------
@dataclasses.dataclass
class Result:
    tokens: List[int]                    # committed tokens, the prefill token first
    sources: List[int]                   # per Verify commit: 1, 2, or 0 (restart)
    tv1: List[float] = dataclasses.field(default_factory=list)   # per Verify: TV(p_R, p_d1) of the root
    tv2: List[float] = dataclasses.field(default_factory=list)   # per Verify: TV(p_R, p_d2) (0 if d2 = 0)
    steps: int = 0                       # batched recurrent steps after prefill
    M: List[int] = dataclasses.field(default_factory=list)   # |A_cur| per step
    n_acc1: int = 0
    n_acc2: int = 0
    n_restart: int = 0
    gate_eval: int = 0
    gate_open: int = 0
    zero_mass: int = 0
    commit_steps: List[int] = dataclasses.field(default_factory=list)
    decisions: List[tuple] = dataclasses.field(default_factory=list)

    @property
    def n_decode(self) -> int:
        return len(self.sources)

    def gamma(self, R: int, d1: int, d2: int) -> float:
        """Mean accepted length (Implementation and Metrics, gamma)."""
        n = self.n_decode
        den = self.n_acc1 * d1 + self.n_acc2 * (d2 or R) + (n - self.n_acc1 - self.n_acc2) * R
        return n * R / den if den else float("nan")


# ----------------------------------------------------------------------------
# vanilla looped decoding
# ----------------------------------------------------------------------------
def decode_vanilla(prov, R: int, n_tokens: int, sampler: Sampler) -> Result:
    """All R depths of one token before the next (Fig. 1a)."""
    node = prov.root()
    res = Result([], [])
    x = sampler.draw(sampler.dist(prov.logits(node, R)), PX.TARGET, prov.position(node) + 1)
    res.tokens.append(x)
    while len(res.tokens) < n_tokens:
        node = prov.child(node, x)
        res.steps += R
        sampler.step = res.steps
        x = sampler.draw(sampler.dist(prov.logits(node, R)), PX.TARGET, prov.position(node) + 1)
        res.tokens.append(x)
        res.sources.append(0)
        res.commit_steps.append(res.steps)
    res.decisions = sampler.decisions
    return res


# ----------------------------------------------------------------------------
# LoopSpec (Alg. 1)
# ----------------------------------------------------------------------------
class Branch:
    __slots__ = ("node", "r", "Q", "parent", "pos", "q2t")

    def __init__(self, node, pos: int, parent: Optional["Branch"]):
        self.node = node          # prefix X^(b) (its readouts come from the provider)
        self.pos = pos            # position of the newest token of X^(b)
        self.r = 0                # recurrent depth
        self.Q: List[tuple] = []  # proposal records (x_j, q_j, child_j)
        self.parent = parent
        self.q2t = None           # readout distribution at d2


def _descends(b: Branch, c: Branch) -> bool:
    while b is not None:
        if b is c:
            return True
        b = b.parent
    return False


# second-proposal variants (Ablation Study, Table 3)
SP_GATED, SP_RESIDUAL, SP_NAIVE = 0, 1, 2


def second_proposal(q1: np.ndarray, q2t: np.ndarray, x1: int, variant: int = SP_GATED):
    """Distribution the second proposal is drawn from, or None when there is none.

    SP_GATED (Sec. 4.3): q2 = q2~ (-) q1, only when q2~(x1) < q1(x1).
    The ablation's ungated variants always propose, with the first proposal x1
    masked out and the rest renormalised so that the two proposals differ:
    SP_RESIDUAL from q2~ (-) q1, SP_NAIVE from q2~ itself.  Reading: when the
    masking leaves no mass there is no second proposal (as with a closed gate).
    Returns (q2 or None, zero_mass flag of the residual).
    """
    if variant == SP_GATED:
        if not q2t[x1] < q1[x1]:
            return None, False
        return D.residual(q2t, q1)
    zm = False
    if variant == SP_RESIDUAL:
        base, zm = D.residual(q2t, q1)
    elif variant == SP_NAIVE:
        base = np.asarray(q2t, np.float64)
    else:
        raise ValueError("unknown second-proposal variant")
    m = np.array(base, np.float64)
    m[x1] = 0.0
    s = m.sum()
    return (m / s if s > 0.0 else None), zm


def decode_loopspec(prov, R: int, d1: int, d2: int, n_tokens: int, sampler: Sampler,
                    max_branches: Optional[int] = None, variant: int = SP_GATED,
                    switches: Optional[Dict[int, Tuple[int, int]]] = None) -> Result:
    """Alg. 1.  d2 = 0 disables the second proposal (single-proposal pipeline).

    `max_branches` (optional) caps the active set: a proposal whose child would
    exceed it is still drawn and verified but spawns no child (a first proposal
    accepted that way restarts from depth 0; a second proposal is treated as a
    closed gate).  Both keep decoding lossless because the choice never looks at
    the target distribution.  `variant` selects the second proposal (see
    second_proposal; the ungated variants are defined for sampling).
    `switches` maps a committed-token count to the pair (d1, d2) decoding
    continues with once that many tokens are committed (module readings).
    """
    if variant != SP_GATED and (sampler.greedy or not d2):
        raise ValueError("the ungated second-proposal variants need sampling and d2 > 0")
    for a, b in [(d1, d2)] + list((switches or {}).values()):
        if not (1 <= a < R) or (b and not (a < b < R)):
            raise ValueError("need 1 <= d1 < d2 < R (or d2 = 0 and d1 < R)")
        if variant != SP_GATED and not b:
            raise ValueError("the ungated second-proposal variants need d2 > 0")
    res = Result([], [])
    A: List[Branch] = []

    def spawn(node, token: int, parent: Optional[Branch]) -> Branch:
        c = Branch(prov.child(node, token), prov.position(node) + 1, parent)
        A.append(c)
        return c

    def room() -> bool:
        return max_branches is None or len(A) < max_branches

    root_node = prov.root()
    x = sampler.draw(sampler.dist(prov.logits(root_node, R)), PX.TARGET,
                     prov.position(root_node) + 1)
    res.tokens.append(x)
    if len(res.tokens) < n_tokens:
        spawn(root_node, x, None)

    while len(res.tokens) < n_tokens:
        res.steps += 1
        sampler.step = res.steps
        cur = list(A)
        res.M.append(len(cur))
        for b in cur:
            b.r += 1                                             # H_b <- B(H_b)
            if b.r == d1:                                        # first proposal
                q1 = sampler.dist(prov.logits(b.node, d1))
                x1 = sampler.draw(q1, PX.DRAFT1, b.pos + 1)
                c1 = spawn(b.node, x1, b) if room() else None
                b.Q = [(x1, q1, c1)]
            elif d2 and b.r == d2:                               # gated second proposal
                x1, q1, _ = b.Q[0]
                q2t = sampler.dist(prov.logits(b.node, d2))
                b.q2t = q2t
                res.gate_eval += 1
                if variant == SP_GATED:
                    sampler.decisions.append(("gate", sampler.step, abs(q2t[x1] - q1[x1]) / max(q1[x1], 1e-300)))
                q2, zm = second_proposal(q1, q2t, x1, variant)
                if q2 is not None and room():
                    res.gate_open += 1
                    res.zero_mass += zm
                    x2 = sampler.draw(q2, PX.DRAFT2, b.pos + 1)
                    c2 = spawn(b.node, x2, b)
                    b.Q.append((x2, q2, c2))
        rmax = max(b.r for b in A)
        if rmax != R:
            continue
        top = [b for b in A if b.r == R]
        assert len(top) == 1, "only the root can reach depth R"
        b = top[0]
        p = sampler.dist(prov.logits(b.node, R))
        res.tv1.append(D.tv(p, b.Q[0][1]))
        res.tv2.append(D.tv(p, b.q2t) if d2 else 0.0)
        xs, c, src = _verify(b, p, sampler, res)
        if c is None:                                            # accepted, but no child was spawned
            c = spawn(b.node, xs, None)
        res.tokens.append(xs)
        res.sources.append(src)
        res.commit_steps.append(res.steps)
        res.n_acc1 += src == 1
        res.n_acc2 += src == 2
        res.n_restart += src == 0
        A[:] = [a for a in A if _descends(a, c)]                 # Reroot(A, c*)
        c.parent = None
        if hasattr(prov, "release"):
            prov.release(b.node, c.node)
        if switches and len(res.tokens) in switches:              # new proposal depths
            d1, d2 = switches[len(res.tokens)]
            A[:] = [c]
            c.Q, c.q2t = [], None
            if c.r >= d1:
                c.r = 0
    res.decisions = sampler.decisions
    return res


def _verify(b: Branch, p: np.ndarray, sampler: Sampler, res: Result):
    """Verify(b, p) of Alg. 1: cascade over the proposal records, then resample."""
    rho = p
    pos = b.pos + 1
    for j, (xj, qj, cj) in enumerate(b.Q):
        event = PX.ACC1 if j == 0 else PX.ACC2
        if sampler.accept(rho[xj] / qj[xj], event, pos):
            return xj, cj, j + 1
        rho, zm = D.residual(rho, qj)
        res.zero_mass += zm
    x = sampler.draw(rho, PX.RESAMPLE, pos)
    return x, None, 0
