"""Pins of the oracle's senior-only GRPO loss pieces (CPU only)."""
import numpy as np

from oracle.grpo import group_advantages, senior_mask, clipped_loss, STD_EPS


def test_advantages_closed_forms():
    # one success among four: mean 1/4, sample std sqrt(1/4) = 1/2
    A = group_advantages(np.array([1.0, 0.0, 0.0, 0.0]), 4)
    np.testing.assert_allclose(A, np.array([0.75, -0.25, -0.25, -0.25]) / (0.5 + STD_EPS), rtol=0, atol=1e-15)
    # constant rewards carry no signal
    np.testing.assert_array_equal(group_advantages(np.ones(8), 8), np.zeros(8))
    # groups are independent; each group's advantages sum to zero
    r = np.random.default_rng(0).integers(0, 2, 24).astype(float)
    A = group_advantages(r, 8)
    np.testing.assert_allclose(A.reshape(3, 8).sum(axis=1), 0.0, atol=1e-12)
    np.testing.assert_allclose(A[8:16], group_advantages(r[8:16], 8), atol=0)


def test_mask_takes_senior_positions_before_the_length():
    owner = np.array([[1, 0, 1, 1], [0, 0, 1, 0]])
    m = senior_mask(owner, np.array([3, 4]))
    np.testing.assert_array_equal(m, [[True, False, True, False], [False, False, True, False]])


def test_ratio_one_reduces_to_the_plain_policy_gradient():
    # logp_new = logp_old: rho = 1, L = -(1/N) sum A over the masked positions,
    # dL/dlogp = -A/N there (the L_TRL equation's gradient)
    rng = np.random.default_rng(1)
    lp = -rng.random((3, 6))
    owner = rng.integers(0, 2, (3, 6))
    mask = senior_mask(owner, np.array([6, 4, 5]))
    adv = np.array([0.7, -1.2, 0.3])
    loss, n, g = clipped_loss(lp, lp, adv, mask)
    assert n == mask.sum()
    assert abs(loss - (-(adv[:, None] * mask).sum() / n)) < 1e-15
    np.testing.assert_allclose(g, np.where(mask, -adv[:, None] / n, 0.0), atol=1e-15)


def test_gradient_matches_finite_differences():
    rng = np.random.default_rng(2)
    S, T = 4, 7
    lo = -rng.random((S, T)) * 3
    ln = lo + rng.normal(0, 0.3, (S, T))       # ratios on both sides of the clip band
    mask = senior_mask(rng.integers(0, 2, (S, T)), np.full(S, T))
    adv = rng.normal(0, 1, S)
    loss, n, g = clipped_loss(ln, lo, adv, mask)
    h = 1e-6
    for s in range(S):
        for t in range(T):
            d = np.zeros((S, T)); d[s, t] = h
            num = (clipped_loss(ln + d, lo, adv, mask)[0] - clipped_loss(ln - d, lo, adv, mask)[0]) / (2 * h)
            assert abs(num - g[s, t]) < 1e-7, (s, t, num, g[s, t])


def test_junior_positions_and_clipped_terms_carry_no_gradient():
    lo = np.zeros((1, 4))
    ln = np.log(np.array([[2.0, 0.5, 1.1, 3.0]]))       # rho = 2, 0.5, 1.1, 3
    mask = np.array([[True, True, True, False]])
    loss, n, g = clipped_loss(ln, lo, np.array([1.0]), mask)
    # A > 0: min(rho, clip(rho)) -> 1.2 (clipped, no gradient), 0.5 (unclipped), 1.1 (inside)
    assert n == 3
    assert abs(loss - (-(1.2 + 0.5 + 1.1) / 3)) < 1e-15
    np.testing.assert_allclose(g, [[0.0, -0.5 / 3, -1.1 / 3, 0.0]], atol=1e-15)
    # changing a junior position changes nothing
    ln2 = ln.copy(); ln2[0, 3] = -5.0
    assert clipped_loss(ln2, lo, np.array([1.0]), mask)[0] == loss
