"""Pins of the oracle's Philox generator and its uniform map (CPU only)."""
import os

import numpy as np
import pytest
from scipy import stats

from oracle.philox import philox_generic, philox4x32, philox_words, coin_threshold
from oracle.sampler import uniform_from_words

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox_kat.txt")


def _kat_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            w = [int(x, 16) for x in line.split()]
            rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


def test_philox4x32_known_answers():
    rows = _kat_rows()
    assert len(rows) == 3
    for ctr, key, out in rows:
        assert philox_generic(ctr, key, 32) == out
        got = philox4x32(np.array([ctr], dtype=np.uint32), key)[0].tolist()
        assert got == out


def test_round_structure_matches_numpy_philox4x64():
    # NumPy's Philox bit generator is Philox4x64-10; it increments the counter
    # before each block, so its first block is philox(counter + 1).
    rng = np.random.default_rng(7)
    for _ in range(20):
        key = [int(x) for x in rng.integers(0, 2**63, size=2)]
        ctr = [int(x) for x in rng.integers(0, 2**62, size=4)]
        bg = np.random.Philox(key=key, counter=ctr)
        raw = [int(x) for x in bg.random_raw(4)]
        nxt = [ctr[0] + 1] + ctr[1:]
        assert philox_generic(nxt, key, 64) == raw


def test_vectorised_equals_scalar():
    rng = np.random.default_rng(3)
    ctr = rng.integers(0, 2**32, size=(64, 4), dtype=np.uint64).astype(np.uint32)
    key = [int(x) for x in rng.integers(0, 2**32, size=2)]
    vec = philox4x32(ctr, key)
    for i in range(64):
        assert vec[i].tolist() == philox_generic(ctr[i].tolist(), key, 32)


def test_word_layout():
    # word v of stream (s, t, stream) is lane v & 3 of counter (v >> 2, t, s, stream)
    seed = (0x1234 << 32) | 0xABCD
    w = philox_words(seed, s=5, t=9, stream=0, n_words=11)
    for v in range(11):
        blk = philox_generic([v >> 2, 9, 5, 0], [0xABCD, 0x1234], 32)
        assert int(w[v]) == blk[v & 3]


def test_uniform_map_is_exact_and_open():
    u = uniform_from_words(np.array([0, 511, 512, 2**32 - 1], dtype=np.uint32))
    assert u.dtype == np.float32
    assert u[0] == np.float32(2.0 ** -24)
    assert u[1] == u[0]                      # the low 9 bits are dropped
    assert u[2] == np.float32(3 * 2.0 ** -24)
    assert u[3] == np.float32(1.0 - 2.0 ** -24)
    assert np.all((u > 0) & (u < 1))


def test_uniformity_and_independence():
    x = philox_words(99, s=1, t=1, stream=0, n_words=200_000)
    u = uniform_from_words(x).astype(np.float64)
    hist, _ = np.histogram(u, bins=64, range=(0, 1))
    assert stats.chisquare(hist).pvalue > 1e-3
    r = np.corrcoef(u[:-1], u[1:])[0, 1]
    assert abs(r) < 4.0 / np.sqrt(u.size)
    # neighbouring (s, t) streams are uncorrelated too
    y = uniform_from_words(philox_words(99, s=2, t=1, stream=0, n_words=200_000)).astype(np.float64)
    assert abs(np.corrcoef(u, y)[0, 1]) < 4.0 / np.sqrt(u.size)


@pytest.mark.parametrize("p,thr", [(0.0, 0), (1.0, 2**32), (0.5, 2**31), (0.1, 429496729)])
def test_coin_threshold(p, thr):
    assert coin_threshold(p) == thr


def test_coin_threshold_rejects_out_of_range():
    with pytest.raises(ValueError):
        coin_threshold(1.5)
    with pytest.raises(ValueError):
        coin_threshold(-0.1)
