"""The allocation-free GRPO entry point (tandem_grpo_loss_noalloc) against
tandem_grpo_loss with a caller workspace, through the C ABI: two calls in a
row, the second with a smaller batch, so the second runs over the device
array the first one left.  Both entry points launch the same kernels, so the
results must agree bit for bit; each is also held to the oracle with the
tolerances of the GRPO parity tests (float32 kernels against the float64
oracle: advantages rtol 1e-5, loss 1e-5 of the mean |term|, exact counts)."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle.grpo import group_advantages, senior_mask, clipped_loss

pytestmark = pytest.mark.gpu

EPS = 0.2


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")


def _call(L, batch, G, noalloc):
    rewards, owner, length, lo, ln = (_dev(x) for x in batch)
    S, T = owner.shape
    cfg = L.GrpoCfg(S // G, G, T, EPS)
    adv = torch.full((S,), float("nan"), dtype=torch.float32, device="cuda:0")
    loss = torch.full((1,), float("nan"), dtype=torch.float32, device="cuda:0")
    n = torch.full((1,), -1, dtype=torch.int32, device="cuda:0")
    grad = torch.full((S, T), float("nan"), dtype=torch.float32, device="cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    args = (rewards.data_ptr(), owner.data_ptr(), length.data_ptr(), lo.data_ptr(), ln.data_ptr(),
            adv.data_ptr(), grad.data_ptr(), loss.data_ptr(), n.data_ptr())
    if noalloc:
        L.tandem_grpo_loss_noalloc(cfg, *args, stream)
    else:
        wsb = L.tandem_grpo_workspace_size(cfg)
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda:0")
        L.tandem_grpo_loss(cfg, *args, ws.data_ptr(), wsb, stream)
    torch.cuda.synchronize()
    return dict(advantages=adv.cpu().numpy(), loss=loss.cpu().numpy(), n_masked=n.cpu().numpy(),
                grad=grad.cpu().numpy())


def _oracle_check(got, batch, G):
    rewards, owner, length, lo, ln = batch
    adv = group_advantages(rewards, G)
    mask = senior_mask(owner, length)
    loss, n, _ = clipped_loss(ln, lo, adv, mask, EPS)
    np.testing.assert_allclose(got["advantages"], adv, rtol=1e-5, atol=1e-6)
    assert int(got["n_masked"][0]) == n
    rho = np.exp(np.where(mask, ln.astype(np.float64) - lo, 0.0))
    terms = np.where(mask, np.minimum(rho * adv[:, None], np.clip(rho, 1 - EPS, 1 + EPS) * adv[:, None]), 0.0)
    assert abs(float(got["loss"][0]) - loss) <= 1e-5 * np.abs(terms).sum() / max(n, 1) + 1e-12


def test_noalloc_matches_workspace_entry_point_twice():
    from paper_2606_28166_amd import _lib as L
    print("no-alloc GRPO: 16 x 8 x 3000 then 3 x 5 x 700", flush=True)
    for (n_groups, G, T), seed in (((16, 8, 3000), 71), ((3, 5, 700), 72)):
        batch = W.make_grpo_batch(n_groups, G, T, seed)
        ref = _call(L, batch, G, noalloc=False)
        got = _call(L, batch, G, noalloc=True)
        for k in ("advantages", "loss", "n_masked", "grad"):
            assert np.array_equal(got[k], ref[k]), k
        _oracle_check(got, batch, G)

