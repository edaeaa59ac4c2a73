"""EOS logit bias of the long-chain-of-thought workload (oracle-side calibration).

The long-CoT workload stops sequences at an EOS token whose logit bias makes
the stop lengths geometric with mean 4000 tokens, i.e. a per-step EOS
probability of 1/4000 under each model's own distribution (a choice of
this implementation: the paper fixes neither the EOS rate nor the bias).  This
script measures, with the float64 oracle, each model's mean EOS probability
over a seeded calibration batch (the workload's first prompts, free-running
decode steps) as a function of the bias b, and finds b by bisection:

    p(b) = mean over (row, step) of  e^(z_eos + b) / (sum_v e^z_v - e^z_eos + e^(z_eos + b))

    python3 oracle/calibrate_eos.py            # prints the two biases

The printed values are the ones stored in the workload definition.  Test
infrastructure only.
"""
from __future__ import annotations

import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

TARGET = 1.0 / 4000.0
CAL_PROMPTS = 4
CAL_STEPS = 24


def eos_logits(model, prompts, eos: int, steps: int, seed: int):
    """(z_eos, log sum_v e^z_v excluding eos) for every (prompt, step) of a greedy decode.

    The decode appends the argmax of the non-EOS logits (a deterministic
    stand-in for sampling; the calibration only needs typical contexts)."""
    out = []
    for x in prompts:
        c = model.new_cache(len(x) + steps + 1)
        if len(x) > 1:
            model.prefill(c, x[:-1])
        tok, pos = int(x[-1]), len(x) - 1
        for _ in range(steps):
            z = model.forward([c], [tok], [pos])[0]
            rest = np.delete(z, eos)
            m = rest.max()
            out.append((z[eos], m + np.log(np.exp(rest - m).sum())))
            zz = z.copy()
            zz[eos] = -np.inf
            tok, pos = int(np.argmax(zz)), pos + 1
    return np.array(out)


def mean_p(samples: np.ndarray, b: float) -> float:
    ze, lse_rest = samples[:, 0], samples[:, 1]
    a = ze + b
    m = np.maximum(a, lse_rest)
    return float(np.mean(np.exp(a - m) / (np.exp(lse_rest - m) + np.exp(a - m))))


def solve(samples: np.ndarray, target: float = TARGET) -> float:
    lo, hi = -20.0, 40.0
    for _ in range(100):
        mid = 0.5 * (lo + hi)
        if mean_p(samples, mid) < target:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def main() -> None:
    import workloads as W
    from oracle.rollout import build_models
    wl = W.workload("longcot")
    wl.n_prompts = CAL_PROMPTS
    ws, wj, prompts, _ = W.make_all(wl)
    sen, jun = build_models(wl, ws, wj)
    eos = wl.sample.eos_id
    for name, model in (("senior", sen), ("junior", jun)):
        smp = eos_logits(model, prompts, eos, CAL_STEPS, wl.philox_seed)
        b = solve(smp)
        print(f"{name}: bias {b:.4f}  (mean p_eos {mean_p(smp, b):.3e}, unbiased {mean_p(smp, 0.0):.3e}, "
              f"{len(smp)} samples)")


if __name__ == "__main__":
    main()
