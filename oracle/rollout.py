"""Oracle tandem rollout driver (Algorithm 1, rollout half; Section 3.3).

For prompt j and rollout i the global sequence id is s = j * G + i.  Both
models prefill x_j[0 .. P_j - 2]; the last prompt token is the first pending
token, so step t = 1 forwards it through both models at position P_j - 1 and
emits y_1.  Every step then:

  1. forwards the pending token through BOTH models (dual forward on the
     shared history; both caches grow in lockstep),
  2. builds scores s_m = (z_m + b_m e_eos) / T for m in {senior, junior},
  3. samples y_t from the owner a_t by Gumbel-max (or takes a forced token),
  4. records y_t, m_t = 1[a_t = senior], the senior log-prob and the margin,
  5. stops the sequence at EOS (after recording it) or at t = max_new,
  6. otherwise applies the handoff block (EOS breaks before it, as in the
     algorithm; at t = max_new the block still runs, then the loop ends).

``forced`` (teacher forcing) replaces the appended token while the oracle
still reports its own sample; entries < 0 mean "not forced".
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence

import numpy as np

from .model import OracleModel
from .philox import coin_threshold
from .sampler import (SENIOR, JUNIOR, gumbel_noise, gumbel_argmax, handoff,
                      scores, senior_logprob, first_owner)


@dataclasses.dataclass
class RolloutResult:
    tokens: np.ndarray        # int32 [n_seq, max_new]   appended token (forced or sampled)
    sampled: np.ndarray       # int32 [n_seq, max_new]   the oracle's own Gumbel-max sample
    owner: np.ndarray         # uint8 [n_seq, max_new]   m_t = 1[a_t = senior]
    logprob: np.ndarray       # float64 [n_seq, max_new] log pi_sen(y_t | .)
    margin: np.ndarray        # float32 [n_seq, max_new] best - second Gumbel score
    decided: np.ndarray       # uint8 [n_seq, max_new]   a handoff decision point was reached after t
    length: np.ndarray        # int32 [n_seq]
    final_owner: np.ndarray   # int32 [n_seq]
    final_c: np.ndarray       # int32 [n_seq]
    final_t: np.ndarray       # int32 [n_seq]
    final_pos: np.ndarray     # int32 [n_seq]
    logits: Dict[int, Dict[str, np.ndarray]]   # step -> {"senior", "junior"} [n_seq, V] (if requested)
    seq_ids: np.ndarray       # int64 [n_seq] global ids of the rows returned


def rollout(sen: OracleModel, jun: OracleModel, prompts: Sequence[np.ndarray], G: int,
            switch, sample, seed: int, boundary: Optional[np.ndarray] = None,
            forced: Optional[np.ndarray] = None, keep_logits_at: Sequence[int] = (),
            seq_subset: Optional[Sequence[int]] = None, max_steps: Optional[int] = None,
            progress=None) -> RolloutResult:
    """Run the tandem rollout.

    switch: workloads.SwitchSettings; sample: workloads.SampleSettings.
    seq_subset restricts the run to some global sequence ids (each sequence's
    result depends only on the weights, its prompt, the seed and its id).
    max_steps truncates the run (the stop rule still uses sample.max_new).
    forced: int array [n_rows, >= steps] of tokens to append, by row.
    progress: optional callable(step, n_steps), called after prefill (step 0)
    and after every decode step (reporting only; the result does not depend on it).
    """
    V = sen.s.vocab
    if jun.s.vocab != V:
        raise ValueError("senior and junior must share one vocabulary")
    n_all = len(prompts) * G
    ids = np.arange(n_all) if seq_subset is None else np.asarray(seq_subset, dtype=np.int64)
    R = len(ids)
    L = sample.max_new
    steps = L if max_steps is None else min(L, max_steps)
    thr = coin_threshold(switch.p)
    T = sample.temperature

    # prefill once per prompt, then copy the caches to the prompt's rows
    caches_s, caches_j, pos, pending = [], [], np.zeros(R, np.int64), np.zeros(R, np.int64)
    proto = {}
    for r, s in enumerate(ids):
        j = int(s) // G
        x = np.asarray(prompts[j])
        if j not in proto:
            ctx = len(x) + L
            cs, cj = sen.new_cache(ctx), jun.new_cache(ctx)
            if len(x) > 1:
                sen.prefill(cs, x[:-1])
                jun.prefill(cj, x[:-1])
            proto[j] = (cs, cj)
        cs, cj = proto[j]
        caches_s.append(cs.copy())
        caches_j.append(cj.copy())
        pos[r] = len(x) - 1
        pending[r] = int(x[-1])
    del proto

    if progress is not None:
        progress(0, steps)
    owner = np.array([first_owner(switch.first_owner, seed, int(s), thr) for s in ids], np.int64)
    c = np.zeros(R, np.int64)
    t = np.ones(R, np.int64)
    done = np.zeros(R, bool)

    out_tok = np.full((R, L), -1, np.int32)
    out_smp = np.full((R, L), -1, np.int32)
    out_own = np.zeros((R, L), np.uint8)
    out_lp = np.zeros((R, L), np.float64)
    out_mg = np.zeros((R, L), np.float32)
    out_dec = np.zeros((R, L), np.uint8)
    length = np.zeros(R, np.int32)
    kept: Dict[int, Dict[str, np.ndarray]] = {}

    for step in range(steps):
        act = np.nonzero(~done)[0]
        if act.size == 0:
            break
        zs = sen.forward([caches_s[r] for r in act], pending[act], pos[act])
        zj = jun.forward([caches_j[r] for r in act], pending[act], pos[act])
        if step + 1 in keep_logits_at:
            kept[step + 1] = {"senior": np.full((R, V), np.nan), "junior": np.full((R, V), np.nan)}
            kept[step + 1]["senior"][act] = zs
            kept[step + 1]["junior"][act] = zj
        for a_i, r in enumerate(act):
            s = int(ids[r])
            tt = int(t[r])
            ss = scores(zs[a_i], T, sample.eos_id, sample.eos_bias_senior)
            sj = scores(zj[a_i], T, sample.eos_id, sample.eos_bias_junior)
            g = gumbel_noise(seed, s, tt, V)
            y_hat, mg = gumbel_argmax(ss if owner[r] == SENIOR else sj, g)
            y = y_hat
            if forced is not None and forced[r, tt - 1] >= 0:
                y = int(forced[r, tt - 1])
            out_tok[r, tt - 1] = y
            out_smp[r, tt - 1] = y_hat
            out_own[r, tt - 1] = 1 if owner[r] == SENIOR else 0
            out_lp[r, tt - 1] = senior_logprob(ss, y)
            out_mg[r, tt - 1] = mg
            length[r] = tt
            is_eos = sample.eos_id >= 0 and y == sample.eos_id
            if not is_eos:
                owner[r], c[r], dec = handoff(switch.mode, int(owner[r]), int(c[r]), y, boundary,
                                             switch.cap_k, seed, s, tt, thr)
                out_dec[r, tt - 1] = 1 if dec else 0
            if is_eos or tt == L:
                done[r] = True
            pending[r] = y
            pos[r] += 1
            t[r] += 1
        if progress is not None:
            progress(step + 1, steps)

    return RolloutResult(out_tok, out_smp, out_own, out_lp, out_mg, out_dec, length,
                         owner.astype(np.int32), c.astype(np.int32), t.astype(np.int32),
                         pos.astype(np.int32), kept, ids)


def build_models(wl, ws, wj):
    """OracleModel pair from workloads-generated weights (float64)."""
    from workloads import weights_as_float
    return (OracleModel(wl.senior, weights_as_float(wl.senior, ws)),
            OracleModel(wl.junior, weights_as_float(wl.junior, wj)))
