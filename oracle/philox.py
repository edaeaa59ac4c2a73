"""Philox counter-based random numbers (oracle side).

The paper draws every Bernoulli handoff coin (and the sampling noise) from a
per-request seeded generator so that a rollout's authorship is reproducible
from its seed (reproducibility appendix, word-level handoff details).  It does
not name the generator; the oracle and the library use Philox4x32-10 of Salmon, Moraes, Dror
and Shaw, "Parallel random numbers: as easy as 1, 2, 3" (SC'11), written here
from that published description:

  * state: a 4-word counter and a 2-word key;
  * one round: multiply counter words 0 and 2 by the round multipliers into
    (hi, lo) double-width products, then the new counter is
        (hi1 ^ c1 ^ k0,  lo1,  hi0 ^ c3 ^ k1,  lo0);
  * between rounds the key is bumped by the Weyl constants;
  * Philox4x32-10 runs 10 rounds with 32-bit words.

Counter layout used by the library and this oracle (the paper fixes none):
  key = (seed mod 2^32, seed >> 32)
  sampling noise for vocab entry v:  ctr = (v >> 2, t, s, 0), word v & 3
  handoff coin:                      ctr = (0,      t, s, 1), word 0
where s is the global sequence id and t the 1-based step.

Pins: philox_generic with 64-bit words equals NumPy's Philox4x64-10 bit
generator; the 32-bit variant equals the published known-answer vectors
(tests/golden/philox_kat.txt); philox4x32 (vectorised) equals philox_generic.
"""
from __future__ import annotations

import numpy as np

_CONST = {
    32: dict(M=(0xD2511F53, 0xCD9E8D57), W=(0x9E3779B9, 0xBB67AE85)),
    64: dict(M=(0xD2E7470EE14C6C93, 0xCA5A826395121157),
             W=(0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)),
}


def philox_generic(ctr, key, width=32, rounds=10):
    """Scalar Philox4xW-R on Python integers (W = 32 or 64). Returns 4 ints."""
    M, W = _CONST[width]["M"], _CONST[width]["W"]
    mask = (1 << width) - 1
    c0, c1, c2, c3 = (int(x) & mask for x in ctr)
    k0, k1 = (int(x) & mask for x in key)
    for r in range(rounds):
        if r:
            k0 = (k0 + W[0]) & mask
            k1 = (k1 + W[1]) & mask
        p0 = M[0] * c0
        p1 = M[1] * c2
        c0, c1, c2, c3 = ((p1 >> width) ^ c1 ^ k0, p1 & mask,
                          (p0 >> width) ^ c3 ^ k1, p0 & mask)
    return [c0, c1, c2, c3]


def philox4x32(ctr: np.ndarray, key, rounds: int = 10) -> np.ndarray:
    """Vectorised Philox4x32-R. ctr: uint32 array [..., 4]; key: 2 ints.

    Products of two 32-bit words are formed exactly in uint64.
    """
    ctr = np.asarray(ctr, dtype=np.uint64)
    M0, M1 = (np.uint64(m) for m in _CONST[32]["M"])
    W0, W1 = _CONST[32]["W"]
    mask = np.uint64(0xFFFFFFFF)
    sh = np.uint64(32)
    c0, c1, c2, c3 = (ctr[..., i].copy() for i in range(4))
    k0, k1 = int(key[0]) & 0xFFFFFFFF, int(key[1]) & 0xFFFFFFFF
    for r in range(rounds):
        if r:
            k0 = (k0 + W0) & 0xFFFFFFFF
            k1 = (k1 + W1) & 0xFFFFFFFF
        p0 = M0 * c0
        p1 = M1 * c2
        c0, c1, c2, c3 = ((p1 >> sh) ^ c1 ^ np.uint64(k0), p1 & mask,
                          (p0 >> sh) ^ c3 ^ np.uint64(k1), p0 & mask)
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def seed_key(seed: int):
    seed = int(seed)
    return (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)


def philox_words(seed: int, s: int, t: int, stream: int, n_words: int) -> np.ndarray:
    """The first n_words 32-bit outputs of the (s, t, stream) sequence.

    Word v comes from counter (v >> 2, t, s, stream), output lane v & 3.
    """
    nblk = (n_words + 3) // 4
    ctr = np.zeros((nblk, 4), dtype=np.uint64)
    ctr[:, 0] = np.arange(nblk, dtype=np.uint64)
    ctr[:, 1] = np.uint64(t & 0xFFFFFFFF)
    ctr[:, 2] = np.uint64(s & 0xFFFFFFFF)
    ctr[:, 3] = np.uint64(stream & 0xFFFFFFFF)
    return philox4x32(ctr, seed_key(seed)).reshape(-1)[:n_words]


def coin_threshold(p: float) -> int:
    """Integer threshold for a Bernoulli(p) coin on a 32-bit word x: x < thr.

    thr = min(2^32, floor(p * 2^32)); p = 0 never fires and p = 1 always does.
    """
    if not (0.0 <= p <= 1.0):
        raise ValueError("p must lie in [0, 1]")
    return min(1 << 32, int(np.floor(np.float64(p) * 4294967296.0)))


def coin(seed: int, s: int, t: int, thr: int) -> bool:
    """The handoff coin of sequence s after step t (t = 0: the first owner)."""
    x = int(philox_words(seed, s, t, 1, 1)[0])
    return x < thr
