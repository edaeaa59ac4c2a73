"""Oracle sampling, senior log-probabilities and the handoff rule.

* Sampling (Algorithm 1: the active model samples y_t from its own
  next-token distribution at temperature T).  Realised as Gumbel-max:
  y = argmax_v (s_v + g_v) with g_v = -log(-log u_v), u_v uniform in (0, 1),
  which draws y ~ softmax(s) exactly.  Only the owner's distribution is
  sampled: the owner a_t is fixed before step t, so keeping y^{a_t} of two
  independent samples has the same law.  The decision is taken
  in float32, the GPU kernel's precision.
* Senior log-probability (the L_TRL equation of Section 3.4): the loss
  needs log pi_sen(y_t | x . y_<t) at senior-owned positions; it is returned
  at every position, taken from the sampling distribution (the paper does
  not say at which temperature; the sampling one is what GRPO's pi_old is).
* Handoff (Algorithm 1's boundary-or-cap block; word-level handoff details
  in the appendix): after y_t is emitted, if y_t is a boundary token or the
  span counter c has reached K, a Bernoulli(p) draw picks the next owner and
  c resets; otherwise the owner is kept and c grows by one.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from .philox import philox_words

SWITCH_REDRAW, SWITCH_FLIP, SWITCH_ALTERNATE = 0, 1, 2
JUNIOR, SENIOR = 0, 1

_TWO_M24 = np.float32(2.0 ** -24)


def scores(z: np.ndarray, T: float, eos_id: int = -1, eos_bias: float = 0.0) -> np.ndarray:
    """Sampling scores s = (z + b * e_eos) / T (float64)."""
    s = np.array(z, dtype=np.float64, copy=True)
    if eos_id >= 0:
        s[..., eos_id] += eos_bias
    return s / T


def uniform_from_words(x: np.ndarray) -> np.ndarray:
    """u = (2 * (x >> 9) + 1) * 2^-24: 2^23 equally spaced points strictly inside (0, 1), exact in fp32."""
    k = (np.asarray(x, dtype=np.uint32) >> np.uint32(9)).astype(np.float32)
    return (k * np.float32(2.0) + np.float32(1.0)) * _TWO_M24


def gumbel_noise(seed: int, s: int, t: int, V: int) -> np.ndarray:
    """Standard Gumbel noise g_v = -log(-log u_v) for v < V, in float32."""
    u = uniform_from_words(philox_words(seed, s, t, 0, V))
    return -np.log(-np.log(u))


def gumbel_argmax(s_owner: np.ndarray, g: np.ndarray):
    """Gumbel-max decision in float32: returns (token, margin best - second).

    Ties go to the smallest token id (the paper does not say).
    """
    val = s_owner.astype(np.float32) + g.astype(np.float32)
    y = int(np.argmax(val))                       # first maximum = smallest id
    best = val[y]
    rest = np.delete(val, y)
    second = rest.max() if rest.size else np.float32(-np.inf)
    return y, float(best - second)


def logsumexp(s: np.ndarray) -> float:
    m = np.max(s)
    return float(m + np.log(np.sum(np.exp(s - m))))


def senior_logprob(s_senior: np.ndarray, y: int) -> float:
    """log softmax(s_senior)[y] in float64."""
    return float(s_senior[y] - logsumexp(s_senior))


def handoff(mode: int, owner: int, c: int, y: int, boundary: Optional[np.ndarray],
            cap_k: int, seed: int, s: int, t: int, thr: int):
    """One application of the handoff block after y_t is emitted.

    Returns (next_owner, next_c, decided) where decided tells whether a
    decision point was reached (boundary token or span cap).
      REDRAW:    next owner = senior iff the coin fires (the paper's rule);
      SWITCH:    next owner flips iff the coin fires;
      ALTERNATE: next owner always flips (the deterministic step schedule).
    The coin is word 0 of Philox counter (0, t, s, 1), firing iff x < thr.
    """
    is_bnd = True if boundary is None else bool(boundary[y])
    at_cap = cap_k >= 0 and c >= cap_k
    if not (is_bnd or at_cap):
        return owner, c + 1, False
    x = int(philox_words(seed, s, t, 1, 1)[0])
    fire = x < thr
    if mode == SWITCH_REDRAW:
        nxt = SENIOR if fire else JUNIOR
    elif mode == SWITCH_FLIP:
        nxt = (1 - owner) if fire else owner
    elif mode == SWITCH_ALTERNATE:
        nxt = 1 - owner
    else:
        raise ValueError(mode)
    return nxt, 0, True


def first_owner(choice: int, seed: int, s: int, thr: int) -> int:
    """a_1: SENIOR / JUNIOR as given, or DRAW = Bernoulli(p) with the t = 0 coin."""
    if choice in (JUNIOR, SENIOR):
        return choice
    x = int(philox_words(seed, s, 0, 1, 1)[0])
    return SENIOR if x < thr else JUNIOR
