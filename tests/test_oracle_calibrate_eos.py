"""Pins of the EOS-bias calibration of the long-CoT workload
(oracle/calibrate_eos.py): the mean EOS probability against a direct
softmax, the bisection against its target, the logit samples against a full
causal recompute, and the stored biases against a fresh seeded batch."""
import numpy as np
import pytest
from scipy.special import logsumexp, softmax

import workloads as W
from oracle.calibrate_eos import TARGET, eos_logits, mean_p, solve
from oracle.rollout import build_models


def _samples(z, eos):
    return np.stack([z[:, eos], logsumexp(np.delete(z, eos, axis=1), axis=1)], axis=1)


def test_mean_p_is_the_softmax_probability_of_the_biased_eos():
    rng = np.random.default_rng(3)
    z = rng.standard_normal((40, 64)) * 2.0
    eos = 5
    smp = _samples(z, eos)
    for b in (-3.0, 0.0, 2.2608, 7.5):
        zb = z.copy()
        zb[:, eos] += b
        direct = softmax(zb, axis=1)[:, eos].mean()
        assert mean_p(smp, b) == pytest.approx(direct, rel=1e-12)
    # no bias: the plain softmax probability of the EOS entry
    assert mean_p(smp, 0.0) == pytest.approx(softmax(z, axis=1)[:, eos].mean(), rel=1e-12)


def test_solve_reaches_the_target_and_p_grows_with_the_bias():
    rng = np.random.default_rng(4)
    z = rng.standard_normal((30, 512))
    smp = _samples(z, 7)
    b = solve(smp)
    assert mean_p(smp, b) == pytest.approx(TARGET, rel=1e-9)
    grid = [mean_p(smp, x) for x in np.linspace(-10, 10, 41)]
    assert all(a < c for a, c in zip(grid, grid[1:]))
    assert solve(smp, 0.5) > b


def test_eos_logits_follow_a_full_causal_recompute():
    """The greedy calibration decode, rebuilt step by step from full prefills
    of the growing sequence (no cache reuse): same EOS logits, same
    log-sum-exp of the other entries, same greedy tokens."""
    wl = W.workload("tiny").replace(gain_jitter=0.1)
    ws, wj, _, _ = W.make_all(wl)
    sen, _ = build_models(wl, ws, wj)
    rng = np.random.default_rng(8)
    prompts = [rng.integers(0, wl.senior.vocab, size=n).astype(np.int32) for n in (9, 4)]
    eos, steps = 11, 5
    got = eos_logits(sen, prompts, eos, steps, seed=0)
    want = []
    for x in prompts:
        seq = list(int(v) for v in x)
        for _ in range(steps):
            c = sen.new_cache(len(seq) + 1)
            z = sen.prefill(c, seq)[-1]
            want.append((z[eos], logsumexp(np.delete(z, eos))))
            zz = z.copy()
            zz[eos] = -np.inf
            seq.append(int(np.argmax(zz)))
    np.testing.assert_allclose(got, np.array(want), rtol=0, atol=1e-9)


def test_stored_biases_give_the_target_rate_on_a_fresh_batch():
    """The long-CoT workload's stored biases, on prompts the calibration never
    saw: the mean EOS probability of each model stays within a factor of 1.5
    of 1/4000 (stop lengths of mean about 4000 tokens), and a fresh bisection
    lands within 0.4 of the stored bias (a factor of 1.5 in probability)."""
    wl = W.workload("longcot")
    ws, wj, _, _ = W.make_all(wl)
    sen, jun = build_models(wl, ws, wj)
    rng = np.random.default_rng(2024)
    eos = wl.sample.eos_id
    prompts = [rng.integers(0, eos, size=48).astype(np.int32) for _ in range(2)]
    for model, stored in ((sen, wl.sample.eos_bias_senior), (jun, wl.sample.eos_bias_junior)):
        smp = eos_logits(model, prompts, eos, 12, seed=0)
        p = mean_p(smp, stored)
        assert TARGET / 1.5 < p < TARGET * 1.5, (stored, p)
        assert abs(solve(smp) - stored) < 0.4
