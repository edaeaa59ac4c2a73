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
        weights=None, before=None, after=None) -> Parity:
    """before: called with the engine before this batch's prefill (earlier use of
    the same handle); after: called with (engine, prompts, oracle result)
    once the teacher-forced steps are read, before the engine is closed."""
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
    if after is not None:
        after(eng, prompts, ref)
    eng.close()
    return Parity(ref, out, sampled, margin, logits, st, steps, rows)


def free_run(eng, prompts, G: int, steps: int, eager: bool, flags: int = 0) -> Dict[str, np.ndarray]:
    """Prefill and `steps` free-running tandem_step calls on an engine, replayed
    from the step graph (eager=False) or launched kernel by kernel; flags: more
    tandem_timing_enable flags for these steps."""
    from paper_2606_28166_amd import _lib as L
    eng.timing((L.TIMING_EAGER if eager else 0) | flags)
    eng.prefill(prompts, G)
    for _ in range(steps):
        eng.step()
    out = eng.outputs()
    eng.timing(0)
    return out


def first_divergence(gpu: Dict[str, np.ndarray], ref, rows: np.ndarray, steps: int, band: float = MARGIN):
    """Free-running GPU stream against the free-running oracle, per checked
    row: the tokens must agree before the row's first step whose oracle Gumbel
    margin is inside `band` (at that step either token is a correct sample,
    and the two streams may part), the owner bits through that step (they
    depend on the earlier tokens only), and rows without such a step must
    agree in full, length included.  Returns (first divergence step or None,
    rows compared in full, tokens compared)."""
    first, full, n = None, 0, 0
    for i, s in enumerate(rows):
        L = min(steps, int(ref.length[i]))
        inband = np.nonzero(ref.margin[i, :L] <= band)[0]
        upto = int(inband[0]) if inband.size else L
        np.testing.assert_array_equal(gpu["tokens"][s, :upto], ref.tokens[i, :upto], err_msg=f"row {s}")
        np.testing.assert_array_equal(gpu["owner"][s, :min(upto + 1, L)], ref.owner[i, :min(upto + 1, L)],
                                      err_msg=f"row {s}")
        diff = np.nonzero(gpu["tokens"][s, :L] != ref.tokens[i, :L])[0]
        if diff.size:
            first = int(diff[0]) + 1 if first is None else min(first, int(diff[0]) + 1)
        else:
            full += 1
        if not inband.size:
            assert min(steps, int(gpu["length"][s])) == L, f"row {s}: length"
        n += upto
    return first, full, n


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
