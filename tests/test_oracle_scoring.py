"""Pins of the oracle's dual-distribution scores (CPU only)."""
import numpy as np
from scipy import stats
from scipy.special import softmax

from oracle.scoring import dual_scores, dual_scores_rows


def test_identical_distributions():
    # alpha = 1, KL = 0, cross-entropy = -log p(y) of the common distribution
    z = np.array([0.3, -1.2, 2.0, 0.0, 0.7])
    ce, a, kl = dual_scores(z, z, 2)
    p = np.exp(z) / np.exp(z).sum()
    assert abs(a - 1.0) < 1e-15
    assert abs(kl) < 1e-15
    assert abs(ce - (-np.log(p[2]))) < 1e-14


def test_logit_shift_changes_nothing():
    # softmax is invariant to adding a constant to all logits
    rng = np.random.default_rng(1)
    zs, zj = rng.standard_normal(50), rng.standard_normal(50)
    base = dual_scores(zs, zj, 7)
    shifted = dual_scores(zs + 123.0, zj - 45.0, 7)
    np.testing.assert_allclose(shifted, base, rtol=0, atol=1e-12)


def test_two_token_closed_form():
    # p_sen = (a, 1 - a), p_jun = (b, 1 - b): alpha = min(a, b) + min(1-a, 1-b),
    # KL = a log(a/b) + (1-a) log((1-a)/(1-b)), cross-entropy of token 1 = -log(1-b)
    a, b = 0.8, 0.35
    zs = np.log([a, 1 - a])
    zj = np.log([b, 1 - b])
    ce, al, kl = dual_scores(zs, zj, 1)
    assert abs(al - (min(a, b) + min(1 - a, 1 - b))) < 1e-15
    assert abs(kl - (a * np.log(a / b) + (1 - a) * np.log((1 - a) / (1 - b)))) < 1e-15
    assert abs(ce - (-np.log(1 - b))) < 1e-15


def test_overlap_is_one_minus_total_variation_and_kl_matches_scipy():
    # sum_v min(p, q) = 1 - (1/2) sum_v |p - q|; KL against scipy's relative entropy
    rng = np.random.default_rng(2)
    for _ in range(20):
        V = int(rng.integers(2, 400))
        zs, zj = rng.standard_normal(V) * 2, rng.standard_normal(V) * 2
        ce, al, kl = dual_scores(zs, zj, int(rng.integers(0, V)))
        p, q = softmax(zs), softmax(zj)
        assert abs(al - (1 - 0.5 * np.abs(p - q).sum())) < 1e-12
        assert abs(kl - stats.entropy(p, q)) < 1e-12
        assert kl >= 0 and 0 <= al <= 1


def test_disjoint_distributions():
    # nearly disjoint supports: alpha -> 0, KL and the cross-entropy of the
    # senior's token grow with the logit gap
    zs = np.array([40.0, 0.0, 0.0])
    zj = np.array([0.0, 40.0, 40.0])
    ce, al, kl = dual_scores(zs, zj, 0)
    assert al < 1e-16
    assert abs(ce - (40 + np.log(2))) < 1e-9
    assert abs(kl - (40 + np.log(2))) < 1e-9


def test_rows():
    rng = np.random.default_rng(3)
    zs, zj = rng.standard_normal((4, 30)), rng.standard_normal((4, 30))
    y = np.array([0, 5, 29, 11])
    out = dual_scores_rows(zs, zj, y)
    for r in range(4):
        np.testing.assert_array_equal(out[r], dual_scores(zs[r], zj[r], y[r]))
