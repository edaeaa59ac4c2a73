"""Shared driver of the GPU-vs-oracle parity tests (imported by test_gpu_*.py).

The oracle runs free; the library then runs teacher-forced on the oracle's
token stream (tandem_step_forced) and reports its own sample, margin and
logits at chosen steps.  Bars (from the hot path's parity protocol):
  * owner masks, decision points and final sampler state: bit-exact;
  * the library's own sample equals the oracle's wherever the oracle's
    Gumbel margin exceeds 1e-2;
  * logits and senior log-probs: max-abs <= 2e-2 (bf16 weights, fp32
    accumulation); fp32 workloads are held to 1e-3.
"""
from __future__ import annotations

import dataclasses
import sys
import time
from typing import Dict, Optional, Sequence

import numpy as np

import workloads as W
from oracle.rollout import rollout, build_models

MARGIN = 1e-2
TOL_BF16 = 2e-2
TOL_F32 = 1e-3


@dataclasses.dataclass
class Parity:
    ref: object
    out: Dict[str, np.ndarray]
    sampled: np.ndarray
    gpu_margin: np.ndarray
    logits: Dict[int, Dict[str, np.ndarray]]
    state: Dict[str, np.ndarray]
    steps: int
    rows: np.ndarray

    def report(self) -> str:
        r = self.ref
        s = self.steps
        lp = np.abs(self.out["logprob"][:, :s] - r.logprob[:, :s]).max()
        big = r.margin[:, :s] > MARGIN
        mism = int(((self.sampled[:, :s] != r.sampled[:, :s]) & big).sum())
        band = int((~big).sum())
        lg = max((float(np.nanmax(np.abs(v["gpu_" + k] - v[k]))) for v in self.logits.values()
                  for k in ("senior", "junior")), default=0.0)
        return (f"steps={s} rows={len(self.rows)} max|dlogprob|={lp:.3e} max|dlogits|={lg:.3e} "
                f"sample mismatches above margin={mism} in-band tokens={band}")


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def run(wl: W.Workload, steps: Optional[int] = None, logits_at: Sequence[int] = (1,),
        max_prefill_tokens: int = 4096, seq_subset: Optional[Sequence[int]] = None,
        weights=None, before=None) -> Parity:
    """before: called with the engine before this batch's prefill (earlier use of
    the same handle)."""
    from paper_2606_28166_amd.engine import TandemEngine
    steps = steps or wl.sample.max_new
    ws, wj, prompts, bnd = weights if weights is not None else W.make_all(wl)
    sen, jun = build_models(wl, ws, wj)
    t0 = time.time()
    def progress(t, n):
        if n >= 32 and (t % 16 == 0 or t == n):
            log(f"  oracle {wl.name}: step {t}/{n} ({time.time() - t0:.0f}s)")

    ref = rollout(sen, jun, prompts, wl.group, wl.switch, wl.sample, wl.philox_seed, bnd,
                  max_steps=steps, keep_logits_at=logits_at, seq_subset=seq_subset, progress=progress)
    log(f"  oracle {wl.name}: {time.time() - t0:.1f}s")
    rows = ref.seq_ids
    n = wl.n_seqs
    max_ctx = max(len(p) for p in prompts) - 1 + wl.sample.max_new
    eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed,
                       max_seqs=n, max_ctx=max_ctx, max_prefill_tokens=max_prefill_tokens,
                       boundary_words=W.boundary_bits(bnd))
    if before is not None:
        before(eng)
    eng.prefill(prompts, wl.group)
    sampled = np.full((len(rows), wl.sample.max_new), -1, np.int32)
    margin = np.zeros((len(rows), wl.sample.max_new), np.float32)
    logits = {}
    for t in range(1, steps + 1):
        forced = np.full(n, -1, np.int32)
        forced[rows] = ref.tokens[:, t - 1]
        want = t in logits_at
        dbg = eng.step_forced(forced, logits=want)
        sampled[:, t - 1] = dbg["sampled"][:n].cpu().numpy()[rows]
        margin[:, t - 1] = dbg["margin"][:n].cpu().numpy()[rows]
        if want:
            logits[t] = {"senior": ref.logits[t]["senior"], "junior": ref.logits[t]["junior"],
                         "gpu_senior": dbg["logits_senior"][:n].cpu().numpy()[rows],
                         "gpu_junior": dbg["logits_junior"][:n].cpu().numpy()[rows]}
    out = eng.outputs()
    out = {k: v[rows] for k, v in out.items()}
    st = eng.state()
    st = {k: v[rows] for k, v in st.items()}
    eng.close()
    return Parity(ref, out, sampled, margin, logits, st, steps, rows)


def check(p: Parity, tol: float) -> None:
    r, s = p.ref, p.steps
    log("  " + p.report())
    np.testing.assert_array_equal(p.out["tokens"][:, :s], r.tokens[:, :s])
    np.testing.assert_array_equal(p.out["owner"][:, :s], r.owner[:, :s])
    big = r.margin[:, :s] > MARGIN
    np.testing.assert_array_equal(p.sampled[:, :s][big], r.sampled[:, :s][big])
    np.testing.assert_allclose(p.out["logprob"][:, :s], r.logprob[:, :s], rtol=0, atol=tol)
    for t, v in p.logits.items():
        for k in ("senior", "junior"):
            live = ~np.isnan(v[k][:, 0])             # rows still generating at step t
            np.testing.assert_allclose(v["gpu_" + k][live], v[k][live], rtol=0, atol=tol,
                                       err_msg=f"{k} logits, step {t}")
    np.testing.assert_array_equal(p.out["length"], r.length)
    np.testing.assert_array_equal(p.state["owner"], r.final_owner)
    np.testing.assert_array_equal(p.state["c"], r.final_c)
    np.testing.assert_array_equal(p.state["t"], r.final_t)
    np.testing.assert_array_equal(p.state["pos"], r.final_pos)
