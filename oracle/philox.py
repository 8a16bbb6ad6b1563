"""Philox4x32-10 counter-based generator and the Gumbel keys drawn from it.

The paper samples K rollouts per prompt from the policy (Alg. 1) without
saying how.  Sampling here is Gumbel-max with counter-based random numbers so
that every (seed, sequence, step, vocabulary id) draw is reproducible on any
device and a resumed rollout continues bit-identically.

Philox4x32-10 is the generator of Salmon, Moraes, Dror and Shaw, "Parallel
random numbers: as easy as 1, 2, 3" (SC'11): ten rounds of two 32x32->64-bit
multiplies with the multipliers 0xD2511F53 and 0xCD9E8D57, the key bumped by
the Weyl constants 0x9E3779B9 and 0xBB67AE85 between rounds.

Counter layout for vocabulary id i of sequence ``seq`` at generation step
``step``: ctr = (i >> 2, step, seq, 0), key = (seed mod 2^32, seed >> 32); the
draw is word (i & 3) of the block.  A word w becomes u = (2*(w >> 9) + 1) * 2^-24,
an odd multiple of 2^-24 strictly inside (0, 1).
"""
from __future__ import annotations

import numpy as np

M0, M1 = 0xD2511F53, 0xCD9E8D57
W0, W1 = 0x9E3779B9, 0xBB67AE85
_MASK = 0xFFFFFFFF


def philox4x32_10(ctr: np.ndarray, key: tuple[int, int]) -> np.ndarray:
    """ctr: uint [n, 4] counters -> uint32 [n, 4] output blocks."""
    c = np.asarray(ctr, dtype=np.uint64) & np.uint64(_MASK)
    c0, c1, c2, c3 = (c[:, j].copy() for j in range(4))
    k0, k1 = int(key[0]) & _MASK, int(key[1]) & _MASK
    m0, m1, msk = np.uint64(M0), np.uint64(M1), np.uint64(_MASK)
    for r in range(10):
        if r:
            k0 = (k0 + W0) & _MASK
            k1 = (k1 + W1) & _MASK
        p0 = m0 * c0
        p1 = m1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & msk
        hi1, lo1 = p1 >> np.uint64(32), p1 & msk
        c0, c1, c2, c3 = (hi1 ^ c1 ^ np.uint64(k0), lo1, hi0 ^ c3 ^ np.uint64(k1), lo0)
    return np.stack([c0, c1, c2, c3], axis=1).astype(np.uint32)


def split_seed(seed: int) -> tuple[int, int]:
    seed = int(seed) & ((1 << 64) - 1)
    return seed & _MASK, seed >> 32


def vocab_words(seed: int, step: int, seq: int, vocab: int) -> np.ndarray:
    """uint32 [vocab] raw draws for every vocabulary id of one sampling step."""
    nblk = (vocab + 3) // 4
    ctr = np.zeros((nblk, 4), np.uint64)
    ctr[:, 0] = np.arange(nblk, dtype=np.uint64)
    ctr[:, 1] = np.uint64(step & _MASK)
    ctr[:, 2] = np.uint64(seq & _MASK)
    return philox4x32_10(ctr, split_seed(seed)).reshape(-1)[:vocab]


def philox_uniform24(words: np.ndarray) -> np.ndarray:
    """u = (2*(w >> 9) + 1) * 2^-24 in float64 (exact)."""
    w = np.asarray(words, np.uint32).astype(np.uint64)
    return (2.0 * (w >> np.uint64(9)).astype(np.float64) + 1.0) * 2.0 ** -24


def gumbel_keys(seed: int, step: int, seq: int, vocab: int) -> np.ndarray:
    """Gumbel(0,1) noise g_i = -ln(-ln u_i) for every vocabulary id."""
    u = philox_uniform24(vocab_words(seed, step, seq, vocab))
    return -np.log(-np.log(u))
