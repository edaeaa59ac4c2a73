"""GPU parity of the senior-only GRPO loss pieces (tandem_grpo_loss) against
the oracle, on seeded synthetic batches and on the arenas of a rollout.

Tolerances (float32 kernels against the float64 oracle):
* advantages: the mean and sample deviation of G rewards in float32, a few
  ulps: rtol 1e-5, atol 1e-6;
* gradient: -rho A / N per position, exp and two products in float32:
  rtol 1e-5;  where the oracle's ratio lies within 1e-5 of a clip edge the
  float32 comparison may take the other branch, and both values are valid;
* loss: float32 terms summed in runs of at most 1024 (four serial adds, a
  wave and a workgroup tree), then in double: |dL| <= 1e-5 * mean |term|.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle.grpo import group_advantages, senior_mask, clipped_loss
from tests import parity as P

pytestmark = pytest.mark.gpu

EPS = 0.2


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")


def _gpu(rewards, owner, length, lo, ln, G, want_grad=True, workspace=None):
    from paper_2606_28166_amd.engine import grpo_loss
    out = grpo_loss(_dev(rewards), _dev(owner), _dev(length), _dev(lo), None if ln is None else _dev(ln), G,
                    EPS, want_grad=want_grad, workspace=workspace)
    torch.cuda.synchronize()
    return {k: (v.cpu().numpy() if v is not None else None) for k, v in out.items()}


def _check(got, rewards, owner, length, lo, ln, G):
    adv = group_advantages(rewards, G)
    mask = senior_mask(owner, length)
    loss, n, grad = clipped_loss(lo if ln is None else ln, lo, adv, mask, EPS)
    np.testing.assert_allclose(got["advantages"], adv, rtol=1e-5, atol=1e-6)
    assert int(got["n_masked"][0]) == n
    rho = np.exp(np.where(mask, (lo if ln is None else ln).astype(np.float64) - lo, 0.0))
    terms = np.where(mask, np.minimum(rho * adv[:, None], np.clip(rho, 1 - EPS, 1 + EPS) * adv[:, None]), 0.0)
    scale = np.abs(terms).sum() / max(n, 1)
    assert abs(float(got["loss"][0]) - loss) <= 1e-5 * scale + 1e-12, (got["loss"][0], loss)
    if got["grad"] is not None:
        g = got["grad"].astype(np.float64)
        edge = mask & ((np.abs(rho - (1 - EPS)) < 1e-5) | (np.abs(rho - (1 + EPS)) < 1e-5))
        ok = np.isclose(g, grad, rtol=1e-5, atol=1e-12)
        alt = edge & (np.isclose(g, 0.0, atol=0) | np.isclose(g, -rho * adv[:, None] / max(n, 1), rtol=1e-5))
        assert np.all(ok | alt), np.argwhere(~(ok | alt))[:5]
        assert np.all(g[~mask] == 0.0)
        return int(edge.sum())
    return 0


@pytest.mark.parametrize("n_groups,G,T", [(16, 8, 3000), (3, 5, 7), (4, 1, 1030), (3, 8, 1024)])
def test_grpo_loss_matches_oracle(n_groups, G, T):
    """Paper batch (16 prompts x G 8, 3000-token arenas: two full chunks and a
    952-position tail), a batch smaller than one chunk, G = 1 (every advantage
    is 0) and an exact one-chunk stride."""
    P.log(f"case grpo loss {n_groups}x{G} rollouts, stride {T}")
    batch = W.make_grpo_batch(n_groups, G, T, seed=11 + T)
    got = _gpu(*batch, G)
    edges = _check(got, *batch, G)
    P.log(f"  loss {got['loss'][0]:.6f}, {got['n_masked'][0]} masked positions, {edges} at a clip edge")


def test_grpo_ratio_one_no_gradient_and_empty_mask():
    """logp_new = NULL (the first update of a GRPO step, where the policy is
    still pi_old: every ratio is 1) without a gradient buffer; then an
    all-junior batch: N = 0, loss 0, zero gradient."""
    P.log("case grpo loss: ratio 1 without gradient, then an empty mask")
    r, o, l, lo, ln = W.make_grpo_batch(4, 8, 500, seed=3)
    got = _gpu(r, o, l, lo, None, 8, want_grad=False)
    assert got["grad"] is None
    _check(got, r, o, l, lo, None, 8)
    got = _gpu(r, np.zeros_like(o), l, lo, ln, 8)
    assert int(got["n_masked"][0]) == 0 and float(got["loss"][0]) == 0.0
    assert np.all(got["grad"] == 0.0)


def test_grpo_zero_clip_band_and_out_of_range_lengths():
    """eps = 0 (the band collapses to ratio 1: a term keeps its gradient only
    on the side the sign of A allows) and lengths outside [0, T] (clamped:
    a negative length masks nothing, one beyond T masks the whole row)."""
    global EPS
    P.log("case grpo loss: eps 0, lengths -5 and T + 100")
    r, o, l, lo, ln = W.make_grpo_batch(4, 4, 700, seed=7)
    l[2], l[3] = -5, 800
    saved, EPS = EPS, 0.0
    try:
        _check(_gpu(r, o, l, lo, ln, 4), r, o, l, lo, ln, 4)
    finally:
        EPS = saved
    _check(_gpu(r, o, l, lo, ln, 4), r, o, l, lo, ln, 4)


def test_grpo_workspace_reused_across_batches():
    """One workspace serves a large batch and then a smaller one: the counts
    and partial sums left by the first call do not leak into the second."""
    from paper_2606_28166_amd import _lib as L
    P.log("case grpo loss: one workspace, 16x8x3000 then 2x4x100")
    ws = torch.empty(L.tandem_grpo_workspace_size(L.GrpoCfg(16, 8, 3000, EPS)), dtype=torch.uint8,
                     device="cuda:0")
    big = W.make_grpo_batch(16, 8, 3000, seed=21)
    _check(_gpu(*big, 8, workspace=ws), *big, 8)
    small = W.make_grpo_batch(2, 4, 100, seed=22)
    _check(_gpu(*small, 4, workspace=ws), *small, 4)


def test_grpo_on_rollout_arenas():
    """End to end: the loss pieces over the owner, log-prob and length arenas
    that tandem_step writes, against the oracle's pieces over the oracle
    rollout of the same workload (teacher-forced on the oracle's tokens, so
    the authorship streams agree bit for bit and the log-probs within the
    bf16 bound).  The current policy's log-probs are the recorded ones plus
    the same seeded offsets on both sides."""
    from paper_2606_28166_amd.engine import TandemEngine
    from oracle.rollout import rollout, build_models
    P.log("case grpo loss on rollout arenas (small shapes, 2 prompts x G 4, 24 steps)")
    wl = _small_rollout_workload()
    steps = wl.sample.max_new
    ws, wj, prompts, bnd = W.make_all(wl)
    sen, jun = build_models(wl, ws, wj)
    ref = rollout(sen, jun, prompts, wl.group, wl.switch, wl.sample, wl.philox_seed, bnd, max_steps=steps)
    n = wl.n_seqs
    eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed, max_seqs=n,
                       max_ctx=max(len(p) for p in prompts) - 1 + steps, boundary_words=W.boundary_bits(bnd))
    eng.prefill(prompts, wl.group)
    for t in range(1, steps + 1):
        eng.step_forced(ref.tokens[:, t - 1], debug=False)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(eng.owner[:n].cpu().numpy(), ref.owner)
    np.testing.assert_array_equal(eng.length[:n].cpu().numpy(), ref.length)
    rng = np.random.default_rng(31)
    rewards = (rng.random(n) < 0.5).astype(np.float32)
    delta = rng.normal(0.0, 0.15, size=(n, steps)).astype(np.float32)
    from paper_2606_28166_amd.engine import grpo_loss
    got = grpo_loss(_dev(rewards), eng.owner[:n], eng.length[:n], eng.logprob[:n], eng.logprob[:n] + _dev(delta),
                    wl.group, EPS)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in got.items()}
    lo = ref.logprob.astype(np.float64)
    adv = group_advantages(rewards, wl.group)
    mask = senior_mask(ref.owner, ref.length)
    loss, cnt, grad = clipped_loss(lo + delta, lo, adv, mask, EPS)
    assert int(got["n_masked"][0]) == cnt
    np.testing.assert_allclose(got["advantages"], adv, rtol=1e-5, atol=1e-6)
    # rho = exp(delta) on both sides up to float32 rounding of (logprob + delta) - logprob
    assert abs(float(got["loss"][0]) - loss) <= 1e-4 * (np.abs(adv).mean() + 1e-6)
    eng.close()
    P.log(f"  loss {got['loss'][0]:.6f} (oracle {loss:.6f}), {cnt} senior positions")


def _small_rollout_workload():
    wl = W.workload("small").replace(gain_jitter=0.05, n_prompts=2, group=4, prompt_len=140, prompt_len_min=40)
    wl.senior.n_layers, wl.junior.n_layers = 2, 1
    wl.sample.max_new = 24
    return wl
