"""Oracle of the senior-only GRPO loss pieces — TEST INFRASTRUCTURE ONLY.

Section 3.4 (tandem policy update) and Algorithm 1's update half: every
rollout y^(j,i) gets a scalar reward r^(j,i); the advantage is GRPO's
group-relative one, computed from the G rewards of its prompt and
normalised by their standard deviation (the advantage-estimator entry of
the hyperparameter table); the senior is updated with GRPO's clipped
surrogate (clip ratio 0.2 in that table, no KL term) on the
positions it emitted only (the response mask narrowed by the authorship
mask m), junior-emitted positions contributing nothing.  Where the paper
defers to standard GRPO, this takes: the sample standard deviation (Bessel's
correction) plus 1e-6, the advantage shared by every position of a rollout,
and the loss averaged over all masked positions of the batch.

Plain float64 NumPy.  Pins: tests/test_oracle_grpo.py.
"""
from __future__ import annotations

import numpy as np

STD_EPS = 1e-6


def group_advantages(rewards: np.ndarray, G: int) -> np.ndarray:
    """A[j G + i] = (r[j G + i] - mean_j) / (std_j + 1e-6), std with Bessel's correction."""
    r = np.asarray(rewards, dtype=np.float64).reshape(-1, G)
    mean = r.mean(axis=1, keepdims=True)
    std = r.std(axis=1, ddof=1, keepdims=True) if G > 1 else np.zeros_like(mean)
    return ((r - mean) / (std + STD_EPS)).reshape(-1)


def senior_mask(owner: np.ndarray, length: np.ndarray) -> np.ndarray:
    """m[s][t] = 1 where the senior emitted position t < length[s] of sequence s."""
    owner = np.asarray(owner)
    T = owner.shape[1]
    return (owner != 0) & (np.arange(T)[None, :] < np.asarray(length)[:, None])


def clipped_loss(logp_new: np.ndarray, logp_old: np.ndarray, adv: np.ndarray, mask: np.ndarray,
                 eps: float = 0.2):
    """GRPO's clipped surrogate over the masked positions, averaged over them:
    L = -(1/N) sum_{masked} min(rho A, clip(rho, 1 - eps, 1 + eps) A), rho = e^(logp_new - logp_old).
    Returns (L, N, dL/dlogp_new [S][T])."""
    mask = np.asarray(mask, dtype=bool)
    n = int(mask.sum())
    ln = np.where(mask, np.asarray(logp_new, dtype=np.float64), 0.0)
    lo = np.where(mask, np.asarray(logp_old, dtype=np.float64), 0.0)
    rho = np.exp(ln - lo)
    A = np.asarray(adv, dtype=np.float64)[:, None] * np.ones_like(rho)
    un = rho * A
    cl = np.clip(rho, 1.0 - eps, 1.0 + eps) * A
    term = np.minimum(un, cl)
    if n == 0:
        return 0.0, 0, np.zeros_like(rho)
    loss = -float(np.sum(np.where(mask, term, 0.0))) / n
    # d min(rho A, clip(rho) A) / d logp_new = rho A where the unclipped term is
    # the minimum (ties included: there clip(rho) = rho), 0 where the clipped
    # constant is strictly smaller
    grad = np.where(mask & (un <= cl), -un / n, 0.0)
    return loss, n, grad
