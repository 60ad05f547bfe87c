"""Philox4x64-10 counter-based generator, written from the Random123 definition
(Salmon et al., "Parallel random numbers: as easy as 1, 2, 3", SC'11).

TEST INFRASTRUCTURE: part of the CPU oracle.  Only tests/, the smoke check and
the benchmark's CPU-baseline leg may import it.

The paper only says that fresh uniforms U ~ U(0,1) are drawn in Verify and that
drafts are sampled from their proposal (Alg. 1).  The oracle makes every draw a
pure function of a key and a counter so that an independent implementation fed
the same (seed, sequence, position, event) obtains the same uniforms:

  key     = (seed, seq)                       two 64-bit words
  counter = (block, position, event, 0)       four 64-bit words

``position`` is the absolute index of the token being decided, ``event`` names
the draw (constants below) and ``block`` indexes groups of 4 vocabulary ids for
vocabulary-wide draws (word ``v & 3`` of block ``v >> 2`` belongs to id v).
"""
from __future__ import annotations

import numpy as np

M0 = 0xD2E7470EE14C6C93
M1 = 0xCA5A826395121157
W0 = 0x9E3779B97F4A7C15
W1 = 0xBB67AE8584CAA73B
MASK = (1 << 64) - 1

# draw events
TARGET = 1     # vanilla decoding / first token after prefill: x ~ p_R
DRAFT1 = 2     # first proposal  x1 ~ q1
DRAFT2 = 3     # second proposal x2 ~ q2
ACC1 = 4       # U_1 of Verify
ACC2 = 5       # U_2 of Verify
RESAMPLE = 6   # x ~ rho after all proposals were rejected


def philox4x64(counter, key, rounds: int = 10):
    """One Philox4x64 block: 4 output words for a 4-word counter and 2-word key."""
    x0, x1, x2, x3 = (int(c) & MASK for c in counter)
    k0, k1 = (int(k) & MASK for k in key)
    for r in range(rounds):
        if r:
            k0 = (k0 + W0) & MASK
            k1 = (k1 + W1) & MASK
        p0 = M0 * x0
        p1 = M1 * x2
        hi0, lo0 = p0 >> 64, p0 & MASK
        hi1, lo1 = p1 >> 64, p1 & MASK
        x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
    return x0, x1, x2, x3


def _mulhilo64(a: np.ndarray, b: int):
    """Vectorised 64x64 -> 128-bit product split into (hi, lo) uint64 words."""
    a = a.astype(np.uint64)
    m32 = np.uint64(0xFFFFFFFF)
    s32 = np.uint64(32)
    a_lo, a_hi = a & m32, a >> s32
    b_lo, b_hi = np.uint64(b & 0xFFFFFFFF), np.uint64(b >> 32)
    ll = a_lo * b_lo
    lh = a_lo * b_hi
    hl = a_hi * b_lo
    hh = a_hi * b_hi
    mid = (ll >> s32) + (lh & m32) + (hl & m32)
    lo = (ll & m32) | ((mid & m32) << s32)
    hi = hh + (lh >> s32) + (hl >> s32) + (mid >> s32)
    return hi, lo


def philox4x64_vec(block: np.ndarray, x1: int, x2: int, x3: int, key, rounds: int = 10):
    """Philox4x64 over many counters that differ only in word 0; returns [n, 4] uint64."""
    with np.errstate(over="ignore"):
        c0 = np.asarray(block, dtype=np.uint64)
        c1 = np.full_like(c0, np.uint64(x1 & MASK))
        c2 = np.full_like(c0, np.uint64(x2 & MASK))
        c3 = np.full_like(c0, np.uint64(x3 & MASK))
        k0, k1 = int(key[0]) & MASK, int(key[1]) & MASK
        for r in range(rounds):
            if r:
                k0 = (k0 + W0) & MASK
                k1 = (k1 + W1) & MASK
            hi0, lo0 = _mulhilo64(c0, M0)
            hi1, lo1 = _mulhilo64(c2, M1)
            c0, c1, c2, c3 = hi1 ^ c1 ^ np.uint64(k0), lo1, hi0 ^ c3 ^ np.uint64(k1), lo0
    return np.stack([c0, c1, c2, c3], axis=1)


def u24(word: int) -> float:
    """Uniform on [0,1) from the top 24 bits; exactly representable in fp32 and fp64."""
    return (int(word) >> 40) * 2.0 ** -24


def u23_open(words: np.ndarray) -> np.ndarray:
    """Uniform on (0,1) from the top 23 bits plus one half; exact in fp32 and fp64."""
    return ((np.asarray(words, dtype=np.uint64) >> np.uint64(41)).astype(np.float64) + 0.5) \
        * 2.0 ** -23


def scalar_uniform(seed: int, seq: int, position: int, event: int) -> float:
    """U in [0,1) for an accept test (block 0, word 0)."""
    return u24(philox4x64((0, position, event, 0), (seed, seq))[0])


def vocab_uniforms(seed: int, seq: int, position: int, event: int, vocab: int) -> np.ndarray:
    """U_v in (0,1) for every vocabulary id v (word v & 3 of block v >> 2)."""
    nb = (vocab + 3) // 4
    words = philox4x64_vec(np.arange(nb, dtype=np.uint64), position, event, 0, (seed, seq))
    return u23_open(words.reshape(-1)[:vocab])
