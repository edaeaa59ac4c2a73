"""GPU parity of the tandem step against the CPU oracle, through the C ABI."""
import numpy as np
import pytest

import workloads as W
from tests import parity as P

pytestmark = pytest.mark.gpu


def _tiny(dtype="f32", **kw):
    wl = W.workload("tiny").replace(gain_jitter=0.1, **kw)
    wl.senior.dtype = dtype
    wl.junior.dtype = dtype
    return wl


def _small_reduced(n_sen=2, n_jun=1, **kw):
    wl = W.workload("small").replace(gain_jitter=0.05, n_prompts=2, group=4, prompt_len=140,
                                     prompt_len_min=40, **kw)
    wl.senior.n_layers, wl.junior.n_layers = n_sen, n_jun
    wl.sample.max_new = 24
    return wl


def _qwen_reduced():
    wl = W.workload("qwen").replace(gain_jitter=0.05, n_prompts=1, group=4, prompt_len=64)
    wl.senior.n_layers, wl.junior.n_layers = 2, 2
    wl.sample.max_new = 12
    return wl


def test_tiny_fp32_all_valu_paths():
    P.log("case tiny fp32")
    p = P.run(_tiny("f32"), logits_at=(1, 16, 32))
    P.check(p, P.TOL_F32)


def test_tiny_bf16_mfma_gemm_valu_attention():
    P.log("case tiny bf16 (head_dim 32)")
    p = P.run(_tiny("bf16"), logits_at=(1, 32))
    P.check(p, P.TOL_BF16)


def test_small_shapes_bf16_ragged_prompts():
    P.log("case small-shaped bf16, ragged prompts, 2+1 layers")
    wl = _small_reduced()
    p = P.run(wl, logits_at=(1, 24), max_prefill_tokens=256)
    P.check(p, P.TOL_BF16)


def test_vocabulary_not_a_multiple_of_four_takes_the_separate_pass():
    """A bf16 pair whose vocabulary (32001) is not a multiple of 4: the LM
    heads cannot take the sampling epilogue (float4 noise rows), so every
    step stores the logits and samples in the separate pass; parity as for
    the other small shapes."""
    P.log("case vocab 32001 (small shapes 2+1 layers): the separate sampling pass")
    wl = _small_reduced()
    wl.senior.vocab = wl.junior.vocab = 32001
    p = P.run(wl, logits_at=(1, 24), max_prefill_tokens=256)
    P.check(p, P.TOL_BF16)


def test_qwen_shapes_bf16_qk_norm():
    P.log("case qwen-shaped bf16, qk-norm, head_dim 128, 2+2 layers")
    p = P.run(_qwen_reduced(), logits_at=(1, 12))
    P.check(p, P.TOL_BF16)


def test_shared_prompt_prefix_edges():
    """The G sequences of a prompt read its K/V prefix (prompt length - 1,
    rounded down to 16) once per block of rows: prompt lengths on both sides
    of every 16-position boundary (no shared prefix at all below 17 tokens,
    a one-position suffix at the first step for 17, 33, 49), G = 3 rows per
    prompt (row blocks split inside a group), contexts crossing several chunk
    boundaries during the rollout."""
    P.log("case shared prompt prefix: small shapes 2+1 layers, prompt lengths 1..65 around multiples of 16, G=3")
    wl = _small_reduced()
    lengths = [1, 2, 16, 17, 18, 32, 33, 48, 49, 65]
    wl.n_prompts, wl.group, wl.prompt_len, wl.prompt_len_min = len(lengths), 3, max(lengths), None
    wl.sample.max_new = 40
    ws, wj, _, bnd = W.make_all(wl)
    rng = np.random.default_rng(77)
    prompts = [rng.integers(0, wl.senior.vocab, size=n).astype(np.int32) for n in lengths]
    p = P.run(wl, logits_at=(1, 17, 40), weights=(ws, wj, prompts, bnd))
    P.check(p, P.TOL_BF16)


@pytest.mark.parametrize("shape", ["small", "qwen"])
def test_one_sequence_per_prompt_unshared_attention(shape):
    """G = 1: no prompt prefix to share, so decode attention takes the per-row
    kernel over each row's whole context (head_dim 64 and 128)."""
    P.log(f"case G=1 ({shape} shapes): per-row decode attention without a shared prefix")
    if shape == "small":
        wl = _small_reduced()
        wl.n_prompts, wl.group = 5, 1
    else:
        wl = _qwen_reduced()
        wl.n_prompts, wl.group, wl.prompt_len_min = 3, 1, 20
    p = P.run(wl, logits_at=(1, wl.sample.max_new))
    P.check(p, P.TOL_BF16)


@pytest.mark.parametrize("shape", ["small", "qwen"])
def test_dual_distribution_scores(shape):
    """tandem_score_step after every teacher-forced step against the oracle's
    scores of the oracle's own logits of that step (end to end, the bf16
    bound)."""
    from paper_2606_28166_amd.engine import TandemEngine
    from oracle.rollout import rollout, build_models
    from oracle.scoring import dual_scores_rows
    P.log(f"case dual-distribution scores ({shape} shapes)")
    wl = _small_reduced() if shape == "small" else _qwen_reduced()
    steps = 12
    wl.sample.max_new = steps
    ws, wj, prompts, bnd = W.make_all(wl)
    sen, jun = build_models(wl, ws, wj)
    ref = rollout(sen, jun, prompts, wl.group, wl.switch, wl.sample, wl.philox_seed, bnd,
                  max_steps=steps, keep_logits_at=tuple(range(1, steps + 1)))
    n = wl.n_seqs
    eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed, max_seqs=n,
                       max_ctx=max(len(p) for p in prompts) - 1 + steps, boundary_words=W.boundary_bits(bnd))
    eng.prefill(prompts, wl.group)
    worst = 0.0
    for t in range(1, steps + 1):
        forced = ref.tokens[:, t - 1]
        eng.step_forced(forced, debug=False)
        sc = eng.score()[:n].cpu().numpy().astype(np.float64)
        e2e = dual_scores_rows(ref.logits[t]["senior"], ref.logits[t]["junior"], forced)
        np.testing.assert_allclose(sc, e2e, rtol=0, atol=P.TOL_BF16, err_msg=f"step {t}")
        worst = max(worst, float(np.abs(sc - e2e).max()))
    eng.close()
    P.log(f"  max |dscore| {worst:.2e}")


def test_sampling_inside_lm_heads_against_separate_pass():
    """At the Qwen shapes (both LM heads on fp16 streaming GEMMs) the step
    samples inside the LM-head GEMMs by default; with
    TANDEM_TIMING_SEPARATE_SAMPLE it stores the logits and samples in a pass
    over them.  Both free-running streams (graph replays) match the
    free-running oracle up to each row's first in-band step, agree with each
    other wherever their tokens agree (senior log-probs within 1e-3: the two
    sum the log-sum-exp in different orders and form the appended token's
    senior score differently), and the dual-distribution scores after a step
    that stored no logits (both LM heads run again) equal those after a step
    that did."""
    from paper_2606_28166_amd import _lib as L
    from paper_2606_28166_amd.engine import TandemEngine
    from oracle.rollout import rollout, build_models
    P.log("case sampling inside the LM heads vs the separate pass (Qwen shapes, 2+2 layers, 8 rows, 16 steps)")
    wl = _qwen_reduced().replace(n_prompts=2)
    steps = 16
    wl.sample.max_new = steps
    ws, wj, prompts, bnd = W.make_all(wl)
    sen, jun = build_models(wl, ws, wj)
    ref = rollout(sen, jun, prompts, wl.group, wl.switch, wl.sample, wl.philox_seed, bnd)
    n = wl.n_seqs
    eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed, max_seqs=n,
                       max_ctx=max(len(p) for p in prompts) - 1 + steps, boundary_words=W.boundary_bits(bnd))
    runs = {}
    for name, flags in (("fused", 0), ("separate", L.TIMING_SEPARATE_SAMPLE)):
        runs[name] = P.free_run(eng, prompts, wl.group, steps, eager=False, flags=flags)
        first, full, cmp = P.first_divergence(runs[name], ref, np.arange(n), steps)
        P.log(f"  {name}: {full}/{n} rows identical to the oracle, {cmp} tokens compared, first divergence {first}")
    a, b = runs["fused"], runs["separate"]
    worst = 0.0
    for s in range(n):
        same = int(np.argmax(a["tokens"][s] != b["tokens"][s])) if (a["tokens"][s] != b["tokens"][s]).any() else steps
        np.testing.assert_allclose(a["logprob"][s, :same], b["logprob"][s, :same], rtol=0, atol=1e-3)
        if same:
            worst = max(worst, float(np.abs(a["logprob"][s, :same] - b["logprob"][s, :same]).max()))
    P.log(f"  max |dlogprob| fused vs separate {worst:.2e}")
    scores = []
    for flags in (0, L.TIMING_SEPARATE_SAMPLE):
        eng.timing(flags)
        eng.prefill(prompts, wl.group)
        eng.step_forced(ref.tokens[:, 0], debug=False)
        scores.append(eng.score()[:n].cpu().numpy())
    eng.close()
    np.testing.assert_allclose(scores[0], scores[1], rtol=0, atol=1e-4)


def test_second_prefill_on_one_handle():
    """A handle takes a new batch of another shape: a first batch (2 prompts x
    G=4) runs 20 graph-replayed steps, then 3 ragged prompts x G=3 are prefilled
    on the same handle and match the oracle (the shared-prefix tables, the
    attention counters and the step graph are rebuilt or reused)."""
    P.log("case second prefill on one handle: small shapes 2+1 layers, 2x4 rows then 3x3 ragged rows")
    wl = _small_reduced()
    lengths = [33, 90, 17]
    wl.n_prompts, wl.group, wl.prompt_len, wl.prompt_len_min = len(lengths), 3, max(lengths), None
    ws, wj, _, bnd = W.make_all(wl)
    rng = np.random.default_rng(5)
    first = [rng.integers(0, wl.senior.vocab, size=n).astype(np.int32) for n in (70, 41)]
    prompts = [rng.integers(0, wl.senior.vocab, size=n).astype(np.int32) for n in lengths]

    def first_batch(eng):
        eng.prefill(first, 4)
        for _ in range(20):
            eng.step()

    p = P.run(wl, logits_at=(1, 24), weights=(ws, wj, prompts, bnd), before=first_batch)
    P.check(p, P.TOL_BF16)


def test_paper_schedule_redraw_word_boundaries_and_cap():
    P.log("case paper schedule: REDRAW p=0.5, K=3, drawn first owner, 35% boundary bitmap, T=0.6")
    wl = _tiny("bf16")
    wl.switch = W.SwitchSettings(W.REDRAW, 0.5, 3, "random:0.351", W.DRAW)
    wl.sample.temperature = 0.6
    p = P.run(wl, logits_at=(5,))
    P.check(p, P.TOL_BF16)
    assert p.ref.decided.sum() > 0 and 0 < p.ref.owner.mean() < 1


def test_paper_schedule_at_qwen_shapes():
    """The paper's training schedule (word-level REDRAW, p = 0.5, span cap 32,
    drawn first owner, T = 0.6, 35% boundary bitmap) on the Qwen shapes."""
    P.log("case paper schedule at Qwen shapes, 2+2 layers, 40 steps")
    wl = _qwen_reduced()
    paper = W.workload("qwen-paper")
    wl.switch, wl.sample.temperature = paper.switch, paper.sample.temperature
    wl.sample.max_new = 40
    p = P.run(wl, logits_at=(1, 40))
    P.check(p, P.TOL_BF16)
    assert p.ref.decided.sum() > 0 and 0 < p.ref.owner.mean() < 1


def test_eos_stops_sequences():
    P.log("case EOS with logit bias")
    wl = _tiny("f32")
    wl.sample.eos_id, wl.sample.eos_bias_senior, wl.sample.eos_bias_junior = 5, 4.0, 3.0
    p = P.run(wl, logits_at=(2,))
    assert (p.ref.length < wl.sample.max_new).any()
    P.check(p, P.TOL_F32)


def test_free_running_is_deterministic_and_matches_oracle_fp32():
    from paper_2606_28166_amd.engine import TandemEngine
    from oracle.rollout import rollout, build_models
    P.log("case free-running determinism")
    wl = _tiny("f32")
    ws, wj, prompts, bnd = W.make_all(wl)
    outs = []
    for _ in range(2):
        eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed,
                           max_seqs=wl.n_seqs, max_ctx=wl.prompt_len - 1 + wl.sample.max_new)
        eng.prefill(prompts, wl.group)
        n_active = None
        for _ in range(wl.sample.max_new):
            n_active = eng.step(want_active=True)
        assert n_active == 0
        outs.append(eng.outputs())
        eng.close()
    for k in outs[0]:
        np.testing.assert_array_equal(outs[0][k], outs[1][k])
    sen, jun = build_models(wl, ws, wj)
    ref = rollout(sen, jun, prompts, wl.group, wl.switch, wl.sample, wl.philox_seed, bnd)
    np.testing.assert_array_equal(outs[0]["tokens"], ref.tokens)
    np.testing.assert_array_equal(outs[0]["owner"], ref.owner)


def test_error_paths_on_device():
    from paper_2606_28166_amd import _lib as L
    from paper_2606_28166_amd.engine import TandemEngine
    P.log("case error paths")
    wl = _tiny("f32")
    ws, wj, prompts, _ = W.make_all(wl)
    eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed,
                       max_seqs=wl.n_seqs, max_ctx=wl.prompt_len - 1 + wl.sample.max_new)
    with pytest.raises(L.TandemError) as e:
        eng.step()
    assert e.value.status == L.E_STATE
    with pytest.raises(L.TandemError) as e:
        eng.prefill([np.arange(40, dtype=np.int32)], 1)          # prompt longer than max_ctx allows
    assert e.value.status == L.E_CAPACITY
    with pytest.raises(L.TandemError) as e:
        eng.prefill(prompts, wl.group + 1)                         # more sequences than max_seqs
    assert e.value.status == L.E_CAPACITY
    # token ids are checked on the device: the prefill is queued, the id is
    # read as 0, and the next synchronising call reports the void batch
    eng.prefill([np.array([1, 2, 9999], dtype=np.int32), np.array([-3], dtype=np.int32)], 2)
    eng.step()
    with pytest.raises(L.TandemError) as e:
        eng.state()
    assert e.value.status == L.E_ARG
    with pytest.raises(L.TandemError) as e:
        eng.step()
    assert e.value.status == L.E_STATE
    # the last prompt token alone out of range (the first pending token)
    eng.prefill([np.array([4, 5, 512], dtype=np.int32)], 1)
    with pytest.raises(L.TandemError) as e:
        eng.step(want_active=True)
    assert e.value.status == L.E_ARG
    # a valid batch afterwards runs and matches a fresh handle
    eng.prefill(prompts, wl.group)
    for _ in range(4):
        eng.step()
    assert eng.step(want_active=True) == wl.n_seqs
    eng.close()


def test_step_graph_replays_match_eager_steps():
    """Free-running steps replayed from the captured step graph equal the same
    steps launched one kernel at a time, bit for bit, with host
    synchronisations and state reads between the replays."""
    from paper_2606_28166_amd import _lib as L
    from paper_2606_28166_amd.engine import TandemEngine
    P.log("case step graph vs eager launches (small shapes, 2+1 layers, ragged prompts)")
    wl = _small_reduced()
    ws, wj, prompts, bnd = W.make_all(wl)
    max_ctx = max(len(p) for p in prompts) - 1 + wl.sample.max_new
    outs, states = [], []
    for eager in (True, False):
        eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed,
                           max_seqs=wl.n_seqs, max_ctx=max_ctx, max_prefill_tokens=256)
        eng.timing(L.TIMING_EAGER if eager else 0)
        eng.prefill(prompts, wl.group)
        trace = []
        for t in range(wl.sample.max_new):
            eng.step()
            if t % 5 == 4:                      # eager work and a sync between replays
                trace.append(eng.state())
        outs.append(eng.outputs())
        states.append(trace)
        eng.close()
    for k in outs[0]:
        np.testing.assert_array_equal(outs[0][k], outs[1][k], err_msg=k)
    for a, b in zip(*states):
        for k in a:
            np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def test_eos_compaction_shrinks_the_batch():
    """EOS-terminated rows are partitioned out of the batch every 32 steps and
    the launched row count shrinks in 32-row buckets; every sequence, wherever
    compaction moves it, still matches the oracle (teacher-forced)."""
    P.log("case EOS compaction: small shapes 2+1 layers, 3 prompts x G=32 = 96 rows, ragged 40..60, strong EOS bias")
    wl = _small_reduced()
    wl.n_prompts, wl.group, wl.prompt_len = 3, 32, 60
    wl.sample.max_new = 80
    wl.sample.eos_id = wl.senior.vocab - 1
    wl.sample.eos_bias_senior = wl.sample.eos_bias_junior = 7.5
    p = P.run(wl, logits_at=(1, 40, 80), max_prefill_tokens=256)
    ended = p.ref.length < wl.sample.max_new
    assert ended.mean() > 0.5, "most sequences should end early"
    # by step 64 (the second compaction) fewer than 64 sequences are alive
    assert (p.ref.length > 64).sum() < 64
    P.check(p, P.TOL_BF16)


def test_compaction_crosses_from_separate_to_fused_sampling():
    """160 rows start above the 128 rows the LM heads' sampling epilogue takes,
    so the first steps store the logits and sample in a separate pass; EOS
    ends enough sequences that the compaction at step 32 brings the launch to
    at most 128 rows, and from there the steps sample inside the LM heads.
    Teacher-forced steps match the oracle throughout, and so do free-running
    steps replayed from the step graph (captured for each row count) up to
    each row's first in-band step."""
    P.log("case separate -> fused sampling across a compaction: small shapes 2+1 layers, 5 prompts x G=32 = 160 rows")
    wl = _small_reduced()
    wl.n_prompts, wl.group, wl.prompt_len = 5, 32, 60
    wl.sample.max_new = 72
    wl.sample.eos_id = wl.senior.vocab - 1
    wl.sample.eos_bias_senior = wl.sample.eos_bias_junior = 7.5
    seen = {}

    def free(eng, prompts, ref):
        out = P.free_run(eng, prompts, wl.group, wl.sample.max_new, eager=False)
        seen["div"] = P.first_divergence(out, ref, ref.seq_ids, wl.sample.max_new)

    p = P.run(wl, logits_at=(1, 40, 72), max_prefill_tokens=256, after=free)
    alive32 = int((p.ref.length > 32).sum())
    assert alive32 <= 128, f"{alive32} sequences still run after step 32: the launch stays above 128 rows"
    P.check(p, P.TOL_BF16)
    first, full, n = seen["div"]
    P.log(f"  {alive32} sequences alive after step 32; free-running graph replays: {full}/{wl.n_seqs} rows "
          f"identical to the oracle, {n} tokens compared, first divergence at step {first}")


@pytest.mark.parametrize("name,switch", [
    ("ALTERNATE at a 20% boundary set, no cap", W.SwitchSettings(W.ALTERNATE, 0.5, -1, "random:0.2", W.SENIOR)),
    ("ALTERNATE with a span cap of 4, junior first", W.SwitchSettings(W.ALTERNATE, 0.5, 4, "random:0.05", W.JUNIOR)),
    ("SWITCH p=0 per token (solo senior)", W.SwitchSettings(W.SWITCH, 0.0, -1, "all", W.SENIOR)),
    ("SWITCH p=1 per token (strict alternation)", W.SwitchSettings(W.SWITCH, 1.0, -1, "all", W.SENIOR)),
    ("REDRAW p=0.3, junior first, 35% boundary set, K=5", W.SwitchSettings(W.REDRAW, 0.3, 5, "random:0.351", W.JUNIOR)),
    ("REDRAW p=1 drawn first owner (solo senior)", W.SwitchSettings(W.REDRAW, 1.0, 2, "random:0.351", W.DRAW)),
    ("REDRAW p=0 drawn first owner (solo junior)", W.SwitchSettings(W.REDRAW, 0.0, 2, "random:0.351", W.DRAW)),
])
def test_handoff_branches(name, switch):
    """Every branch of the handoff block on the GPU: the ALTERNATE flip (with
    and without the span cap), the coin thresholds 0 and 2^32 (p = 0 and
    p = 1), the junior as first owner, and the drawn first owner at p in
    {0, 1}; owner masks, decision state and tokens bit-exact."""
    P.log(f"case handoff branch: {name} (tiny bf16)")
    wl = _tiny("bf16")
    wl.switch = switch
    p = P.run(wl, logits_at=(7,))
    P.check(p, P.TOL_BF16)
    own = p.ref.owner
    if switch.mode == W.SWITCH and switch.p == 0.0:
        assert own.all()
    elif switch.mode == W.SWITCH and switch.p == 1.0:
        assert (own[:, 1:] != own[:, :-1]).all()
    elif switch.mode == W.REDRAW and switch.p in (0.0, 1.0):
        assert (own == int(switch.p)).all()
    elif switch.mode == W.ALTERNATE:
        assert p.ref.decided.sum() > 0
        if switch.first_owner == W.JUNIOR:
            assert (own[:, 0] == 0).all()


@pytest.mark.parametrize("schedule", ["alternate", "stepcoin"])
def test_reasoning_step_schedules_at_qwen_shapes(schedule):
    """The evaluation schedules: the owner flips at every reasoning-step
    boundary (deterministic round-robin) or is redrawn there by a fair coin,
    with no span cap and T = 0.6, on a sparse synthetic step-boundary set
    (Qwen shapes, 2+2 layers, 64 steps)."""
    wl_ref = W.workload("qwen-eval-" + schedule)
    P.log(f"case reasoning-step schedule {schedule} at Qwen shapes, 2+2 layers, 64 steps")
    wl = _qwen_reduced()
    wl.switch, wl.sample.temperature = wl_ref.switch, wl_ref.sample.temperature
    wl.switch.boundary = "random:0.1"          # denser than the workload's, so 64 steps cross several steps
    wl.sample.max_new = 64
    p = P.run(wl, logits_at=(1, 64))
    P.check(p, P.TOL_BF16)
    assert p.ref.decided.sum() > 0 and 0 < p.ref.owner.mean() < 1


def test_graph_replays_with_compaction_match_oracle_fp32():
    """Free-running steps replayed from the step graph, with EOS ending most
    sequences so that compaction shrinks the launched rows and the graph is
    captured again: the stream equals eager launches bit for bit, and equals
    the free-running oracle (fp32 models: up to each row's first step whose
    Gumbel margin is inside the float32 band)."""
    from paper_2606_28166_amd.engine import TandemEngine
    from oracle.rollout import rollout, build_models
    P.log("case graph replays across compactions vs oracle: tiny fp32, 3 prompts x G=32, EOS")
    wl = _tiny("f32")
    wl.n_prompts, wl.group = 3, 32
    wl.sample.max_new = 80
    wl.sample.eos_id, wl.sample.eos_bias_senior, wl.sample.eos_bias_junior = 7, 3.0, 2.5
    ws, wj, prompts, bnd = W.make_all(wl)
    sen, jun = build_models(wl, ws, wj)
    ref = rollout(sen, jun, prompts, wl.group, wl.switch, wl.sample, wl.philox_seed, bnd)
    assert (ref.length < 32).sum() >= 32 and (ref.length > 64).sum() > 0, "compaction must shrink the batch"
    eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed,
                       max_seqs=wl.n_seqs, max_ctx=wl.prompt_len - 1 + wl.sample.max_new)
    graph = P.free_run(eng, prompts, wl.group, wl.sample.max_new, eager=False)
    eager = P.free_run(eng, prompts, wl.group, wl.sample.max_new, eager=True)
    eng.close()
    for k in graph:
        np.testing.assert_array_equal(graph[k], eager[k], err_msg=k)
    first, full, n = P.first_divergence(graph, ref, np.arange(wl.n_seqs), wl.sample.max_new, band=1e-4)
    P.log(f"  {full}/{wl.n_seqs} rows identical to the oracle, {n} tokens compared, first divergence {first}")
    assert full >= wl.n_seqs - 2


def test_senior_alone_matches_single_model_sampling():
    """A handle without a junior: the senior emits every token through the
    same kernels, as the oracle's tandem rollout does with SWITCH p = 0 and the
    senior first (pinned on the CPU to equal plain single-model sampling)."""
    from paper_2606_28166_amd.engine import TandemEngine
    from oracle.rollout import rollout, build_models
    P.log("case the senior alone: small shapes 2 layers, ragged prompts, 24 steps")
    wl = _small_reduced()
    wl.switch = W.SwitchSettings(W.SWITCH, 0.0, -1, "all", W.SENIOR)
    ws, wj, prompts, bnd = W.make_all(wl)
    sen, jun = build_models(wl, ws, wj)
    ref = rollout(sen, jun, prompts, wl.group, wl.switch, wl.sample, wl.philox_seed, bnd, keep_logits_at=(1, 24))
    n = wl.n_seqs
    eng = TandemEngine(wl.senior, ws, None, None, wl.switch, wl.sample, wl.philox_seed, max_seqs=n,
                       max_ctx=max(len(p) for p in prompts) - 1 + wl.sample.max_new, max_prefill_tokens=256)
    eng.prefill(prompts, wl.group)
    worst = 0.0
    for t in range(1, wl.sample.max_new + 1):
        dbg = eng.step_forced(ref.tokens[:, t - 1], logits=t in (1, 24))
        big = ref.margin[:, t - 1] > P.MARGIN
        got = dbg["sampled"][:n].cpu().numpy()
        np.testing.assert_array_equal(got[big], ref.sampled[big, t - 1])
        if t in (1, 24):
            z = dbg["logits_senior"][:n].cpu().numpy()
            worst = max(worst, float(np.abs(z - ref.logits[t]["senior"]).max()))
    out = eng.outputs()
    eng.close()
    assert worst < P.TOL_BF16
    np.testing.assert_array_equal(out["tokens"], ref.tokens)
    assert out["owner"].all() and ref.owner.all()
    np.testing.assert_allclose(out["logprob"], ref.logprob, rtol=0, atol=P.TOL_BF16)
    P.log(f"  max |dlogits| {worst:.2e}")


def test_self_paired_shapes_paper_schedule():
    """The paper's self-paired pair (two Qwen3-4B-shaped models) under its
    training schedule (REDRAW p = 0.5, K = 32, drawn first owner, T = 0.6, 35%
    boundary set), 2 + 2 layers, 40 steps."""
    P.log("case self-paired 4B/4B shapes, paper schedule, 2+2 layers, 40 steps")
    wl = W.workload("self-paired").replace(gain_jitter=0.05, n_prompts=1, group=4, prompt_len=64)
    wl.senior.n_layers, wl.junior.n_layers = 2, 2
    wl.sample.max_new = 40
    p = P.run(wl, logits_at=(1, 40))
    P.check(p, P.TOL_BF16)
    assert p.ref.decided.sum() > 0 and 0 < p.ref.owner.mean() < 1
