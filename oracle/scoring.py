"""Oracle of the dual-distribution scores of a token stream — TEST INFRASTRUCTURE ONLY.

At one position, both models' next-token distributions over the shared
vocabulary (temperature 1, no sampling bias: the models' own distributions;
the paper states no temperature for these measures) and the token y that
the stream emits there give:

* the junior's cross-entropy of y, -log p_jun(y), in nats (the per-token
  junior legibility measure of the evaluation section on junior legibility);
* the distribution overlap alpha = sum_v min(p_sen(v), p_jun(v)) (the same
  section; 0 for disjoint supports, 1 for identical distributions);
* KL(p_sen || p_jun) = sum_v p_sen(v) (log p_sen(v) - log p_jun(v)), the
  per-position divergence of the senior from the junior (the ablation section's
  KL regularisation towards the junior uses this direction).

Plain float64 NumPy, written from those definitions.  Pins:
tests/test_oracle_scoring.py.
"""
from __future__ import annotations

import numpy as np


def _log_softmax(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.float64)
    m = np.max(z)
    return z - (m + np.log(np.sum(np.exp(z - m))))


def dual_scores(z_sen: np.ndarray, z_jun: np.ndarray, y: int):
    """(junior cross-entropy of y, overlap alpha, KL(p_sen || p_jun)) of one
    position, from the two models' logits z_sen, z_jun (length V) and the
    emitted token y."""
    ls = _log_softmax(z_sen)
    lj = _log_softmax(z_jun)
    ps, pj = np.exp(ls), np.exp(lj)
    ce = -lj[int(y)]
    alpha = float(np.sum(np.minimum(ps, pj)))
    kl = float(np.sum(ps * (ls - lj)))
    return float(ce), alpha, kl


def dual_scores_rows(z_sen: np.ndarray, z_jun: np.ndarray, y: np.ndarray) -> np.ndarray:
    """dual_scores of every row: [R][3] (cross-entropy, alpha, KL)."""
    return np.array([dual_scores(z_sen[r], z_jun[r], y[r]) for r in range(len(y))], dtype=np.float64)
