"""Pins of the oracle's sampler, senior log-probs and handoff rule (CPU only)."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st
from scipy import stats
from scipy.special import log_softmax, softmax

from oracle.philox import coin_threshold, philox_words
from oracle.sampler import (gumbel_noise, gumbel_argmax, senior_logprob, scores, handoff,
                            first_owner, SWITCH_REDRAW, SWITCH_FLIP, SWITCH_ALTERNATE, SENIOR, JUNIOR)


def test_gumbel_max_histogram_matches_softmax():
    # 2e5 draws over distinct (s, t) counters against softmax, chi-square
    rng = np.random.default_rng(0)
    V = 512
    s = rng.standard_normal(V) * 1.5
    n = 200_000
    counts = np.zeros(V)
    for i in range(n // 1000):
        for j in range(1000):
            g = gumbel_noise(1234, s=i, t=j + 1, V=V)
            y, _ = gumbel_argmax(s, g)
            counts[y] += 1
    p = softmax(s)
    exp = p * n
    keep = exp >= 5
    obs = np.append(counts[keep], counts[~keep].sum())
    ex = np.append(exp[keep], exp[~keep].sum())
    assert stats.chisquare(obs, ex).pvalue > 1e-3


def test_low_temperature_is_argmax():
    rng = np.random.default_rng(1)
    z = rng.standard_normal(300)
    for t in range(1, 30):
        g = gumbel_noise(5, 0, t, 300)
        y, _ = gumbel_argmax(scores(z, 1e-4), g)
        assert y == int(np.argmax(z))


def test_ties_go_to_smallest_id_and_margin():
    s = np.array([0.0, 2.0, 1.0, 2.0])
    y, m = gumbel_argmax(s, np.zeros(4, np.float32))
    assert y == 1 and m == 0.0
    y, m = gumbel_argmax(np.array([0.0, 1.0, 3.0]), np.zeros(3, np.float32))
    assert y == 2 and m == pytest.approx(2.0)


def test_logprob_matches_scipy_and_normalises():
    rng = np.random.default_rng(2)
    z = rng.standard_normal(2000) * 3
    s = scores(z, 0.6, eos_id=7, eos_bias=-2.0)
    ref = log_softmax(s)
    for y in (0, 7, 1999):
        assert senior_logprob(s, y) == pytest.approx(ref[y], abs=1e-12)
    lp = np.array([senior_logprob(s, y) for y in range(2000)])
    assert abs(np.exp(lp).sum() - 1) < 1e-10 and np.all(lp <= 0)


def test_scores_bias_and_temperature():
    z = np.array([1.0, 2.0, 3.0])
    np.testing.assert_allclose(scores(z, 0.5, eos_id=1, eos_bias=4.0), [2.0, 12.0, 6.0])
    np.testing.assert_allclose(scores(z, 2.0), [0.5, 1.0, 1.5])


# ---------------------------------------------------------------- handoff rule

def _run(mode, p, owner0, toks, bnd, K, seed=3, s=0):
    thr = coin_threshold(p)
    a, c, owners, decs = owner0, 0, [], []
    for t, y in enumerate(toks, start=1):
        owners.append(a)
        a, c, d = handoff(mode, a, c, y, bnd, K, seed, s, t, thr)
        decs.append(d)
    return owners, decs


def test_switch_p1_token_level_alternates():
    owners, decs = _run(SWITCH_FLIP, 1.0, SENIOR, list(range(40)), None, -1)
    assert owners == [SENIOR, JUNIOR] * 20 and all(decs)


def test_switch_p0_is_solo_senior():
    owners, _ = _run(SWITCH_FLIP, 0.0, SENIOR, list(range(200)), None, -1)
    assert set(owners) == {SENIOR}


def test_redraw_extremes():
    o1, _ = _run(SWITCH_REDRAW, 1.0, JUNIOR, list(range(50)), None, -1)
    assert o1 == [JUNIOR] + [SENIOR] * 49
    o0, _ = _run(SWITCH_REDRAW, 0.0, SENIOR, list(range(50)), None, -1)
    assert o0 == [SENIOR] + [JUNIOR] * 49


def test_alternate_ignores_the_coin():
    bnd = np.zeros(10, bool)
    bnd[3] = True
    toks = [1, 3, 1, 1, 3, 3, 1]
    owners, decs = _run(SWITCH_ALTERNATE, 0.0, SENIOR, toks, bnd, -1)
    assert decs == [False, True, False, False, True, True, False]
    assert owners == [SENIOR, SENIOR, JUNIOR, JUNIOR, JUNIOR, SENIOR, JUNIOR]


@pytest.mark.parametrize("K", [0, 3, 31])
def test_cap_fires_every_k_plus_one_tokens(K):
    bnd = np.zeros(8, bool)
    _, decs = _run(SWITCH_FLIP, 0.5, SENIOR, [1] * 200, bnd, K)
    fired = [t for t, d in enumerate(decs, start=1) if d]
    assert fired == list(range(K + 1, 201, K + 1))


def test_boundary_token_resets_span_counter():
    bnd = np.zeros(8, bool)
    bnd[5] = True
    toks = [1, 1, 5, 1, 1, 1, 1]
    _, decs = _run(SWITCH_FLIP, 0.5, SENIOR, toks, bnd, 3)
    # boundary at t=3 resets c; the cap then fires at t = 3 + 4 = 7
    assert decs == [False, False, True, False, False, False, True]


@settings(max_examples=60, deadline=None)
@given(st.lists(st.integers(0, 15), min_size=1, max_size=120), st.integers(0, 6),
       st.sampled_from([SWITCH_REDRAW, SWITCH_FLIP]), st.integers(0, 2**31))
def test_no_run_longer_than_cap_plus_one(toks, K, mode, seed):
    bnd = np.zeros(16, bool)
    bnd[:3] = True
    _, decs = _run(mode, 0.5, SENIOR, toks, bnd, K, seed=seed)
    gap = 0
    for t, (y, d) in enumerate(zip(toks, decs)):
        gap += 1
        assert gap <= K + 1
        if bnd[y]:
            assert d                     # a boundary token always decides
        if d:
            gap = 0


@pytest.mark.parametrize("p", [0.1, 0.3, 0.5])
def test_switch_rate_matches_p(p):
    thr = coin_threshold(p)
    n, flips = 0, 0
    for s in range(40):
        a, c = SENIOR, 0
        for t in range(1, 501):
            b, c, d = handoff(SWITCH_FLIP, a, c, 0, None, -1, 77, s, t, thr)
            n += 1
            flips += int(b != a)
            a = b
    sigma = np.sqrt(p * (1 - p) / n)
    assert abs(flips / n - p) < 4 * sigma


@pytest.mark.parametrize("p", [0.2, 0.5])
def test_redraw_senior_share_matches_p(p):
    thr = coin_threshold(p)
    n, sen = 0, 0
    for s in range(40):
        a, c = first_owner(2, 11, s, thr), 0
        for t in range(1, 301):
            n += 1
            sen += int(a == SENIOR)
            a, c, _ = handoff(SWITCH_REDRAW, a, c, 0, None, -1, 11, s, t, thr)
    assert abs(sen / n - p) < 4 * np.sqrt(p * (1 - p) / n) * 1.5


def test_first_owner_draw_uses_t0_coin():
    thr = coin_threshold(0.5)
    for s in range(20):
        x = int(philox_words(9, s, 0, 1, 1)[0])
        assert first_owner(2, 9, s, thr) == (SENIOR if x < thr else JUNIOR)
    assert first_owner(SENIOR, 9, 0, 0) == SENIOR
    assert first_owner(JUNIOR, 9, 0, 2**32) == JUNIOR
