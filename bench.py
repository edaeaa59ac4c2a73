#!/usr/bin/env python3
"""Benchmark of the tandem co-generation rollout on one MI355X.

One bench step = one whole rollout of the batch through the hot path:
prefill of both models on every prompt, then max_new tandem decode steps
(dual forward, owner sampling, senior log-probs, handoff rule).  Inputs
(weights, prompts, KV arena) are resident in HBM before the timed region.

A rollout of the Qwen-shaped workload takes about 22 s, so the run keeps a
wall-clock budget (--budget-s, counted from process start): the warmup runs
one rollout (more only when they fit a short warm budget), the timed region
covers at least one whole rollout and at most as many as fit --timed-s, and
the optional legs (the instrumented rollouts, the CPU oracle) run only
while the budget lasts.  `steps` and `warmup` in the line are the rollouts
actually run (`steps_requested`, `warmup_requested` the flags), and
ms_per_step x steps is the timed wall time.

Prints ONE JSON line:
  value            co-generated tokens / s over the whole job (prefill + decode)
  roofline         decode attention (the dominant kernel): algorithmic K/V
                   bytes per launch / its average launch time, from HIP event
                   pairs around every launch (on the stream it runs on) in an
                   extra rollout whose two forwards run one after the other, so
                   each launch has the GPU to itself; the per-class breakdown
                   comes from the same rollout.  When the G sequences of a
                   prompt share its K/V prefix, its rows read the prefix side
                   by side (HBM delivers it about once per group) and the
                   algorithmic bytes count it once per group
  roofline_concurrent the same in the two-stream schedule of the timed region
                   (the junior's forward overlapping the senior's)
  (the timed region replays the captured step graph; graph-captured event
   records carry no launch times, so both roofline rollouts launch from the host)
  cpu_baseline     the CPU oracle (float64 NumPy) timed on a bounded sample of
                   the same workload on this host's cores
  decode_*         decode-only tokens/s and whole-decode-step HBM fraction
  tandem_over_solo the same batch with the senior alone (a handle with no
                   junior): decode ms per step of both and their ratio
  sampling         where the step samples: inside the LM-head GEMMs (no logits
                   stored), or a separate pass over stored logits (more than
                   128 rows, fp32 models, or --separate-sample)

Counter mode (HBM traffic per kernel class, rocprofv3 FETCH_SIZE and
WRITE_SIZE, each in a run of its own):
    rocprofv3 --pmc FETCH_SIZE -d <dir> -o fetch --output-format csv -- python3 bench.py --pmc-run
    rocprofv3 --pmc WRITE_SIZE -d <dir> -o write --output-format csv -- python3 bench.py --pmc-run
    python3 bench.py --pmc-analyze <fetch csv> <write csv>
(--pmc-warm N on all three: N graph-replayed steps before the measured ones,
1000 by default so that the attention reads mid-rollout contexts; 0 for the
other classes.)
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

T_START = time.perf_counter()
ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
METRIC = "co-generated tokens/sec on 1 MI355X; decode HBM GB/s as % of peak"

DESCRIPTIONS = {
    "qwen": "Qwen3-4B-shaped senior + Qwen3-0.6B-shaped junior, bf16, 16 prompts x G=8, prompt 256, 2048 new tokens, switch p=0.1",
    "small": "8-layer d=1024 senior + 4-layer d=512 junior, bf16, 8 prompts x G=8, prompt 128, 512 new tokens, switch p=0.1",
    "wide": "small shapes, 64 prompts x G=16 = 1024 sequences, prompt 256, 4096 new tokens, switch p=0.5",
    "tiny": "2-layer d=128 senior + 1-layer d=64 junior, fp32, 1 prompt x G=4, 32 new tokens",
    "longcot": "small shapes, 32 prompts x G=8 = 256 sequences, ragged prompts 64..512, up to 8192 new tokens, "
               "EOS bias for mean length 4000, ownership switch p=0.3 per 32-token chunk, finished sequences compacted",
    "paper": "small shapes, 4 prompts x G=8, prompt 64, 128 new tokens, the paper's schedule: word-level REDRAW "
             "p=0.5, span cap K=32, drawn first owner, T=0.6, 35% boundary bitmap",
    "qwen-paper": "Qwen3-4B-shaped senior + Qwen3-0.6B-shaped junior, bf16, 16 prompts x G=8, prompt 256, 2048 new "
                  "tokens, the paper's schedule: word-level REDRAW p=0.5, span cap K=32, drawn first owner, T=0.6, "
                  "35% boundary bitmap",
    "self-paired": "Qwen3-4B-shaped senior + Qwen3-4B-shaped junior, bf16, 16 prompts x G=8, prompt 256, 3000 new "
                   "tokens, the paper's schedule (REDRAW p=0.5, K=32, drawn first owner, T=0.6, 35% boundary bitmap)",
    "qwen-eval-alternate": "Qwen3-4B-shaped senior + Qwen3-0.6B-shaped junior, bf16, 16 prompts x G=8, prompt 256, "
                           "2048 new tokens, the evaluation schedule: owner flips at every reasoning-step boundary "
                           "(1/48-density synthetic boundary set), senior first, no cap, T=0.6",
    "qwen-eval-stepcoin": "Qwen3-4B-shaped senior + Qwen3-0.6B-shaped junior, bf16, 16 prompts x G=8, prompt 256, "
                          "2048 new tokens, the stochastic evaluation schedule: fair-coin redraw at every "
                          "reasoning-step boundary (1/48-density synthetic boundary set), drawn first owner, no cap, "
                          "T=0.6",
}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# ----------------------------------------------------------- algorithmic bytes
def kv_bytes_per_token(s: W.ModelShape) -> int:
    """K and V bytes of one position over all layers of one model."""
    esz = 2 if s.dtype == "bf16" else 4
    return 2 * s.n_layers * s.n_kv_heads * s.head_dim * esz


def weight_bytes(s: W.ModelShape) -> int:
    esz = 2 if s.dtype == "bf16" else 4
    d, hd = s.d_model, s.head_dim
    body = s.n_layers * (d * (s.n_q_heads + 2 * s.n_kv_heads) * hd + s.n_q_heads * hd * d + 3 * d * s.ffn_dim)
    return esz * (body + d * s.vocab)


def shares_prefix(wl: W.Workload) -> bool:
    """Whether the G sequences of a prompt share its K/V prefix (bf16 models,
    head_dim 64 or 128, at most 16 query heads per kv head, G > 1), as the
    library decides at prefill: decode attention then reads the prefix from
    the prompt's first slot for every row of the group, and the group's rows
    run side by side on one XCD, so HBM delivers the prefix about once per
    group (the rest comes from L2)."""
    def ok(s):
        g = s.n_q_heads // s.n_kv_heads
        return s.dtype == "bf16" and s.head_dim in (64, 128) and g in (1, 2, 4, 8, 16) and s.n_q_heads % s.n_kv_heads == 0
    return wl.group > 1 and ok(wl.senior) and ok(wl.junior)


def _context_positions(wl: W.Workload, plens, t: int, lengths=None):
    """(active rows, K/V positions decode step t must read per layer of a model).
    Row r of prompt j attends positions 0 .. P_j + t - 2.  With a shared prefix
    the first lo_j = (P_j - 1) rounded down to 16 positions count once per group
    with an active row, the rest once per row; otherwise every row counts its
    whole context (lengths: tokens each sequence generated; None: all run every
    step)."""
    share = shares_prefix(wl)
    n_rows, pos = 0, 0
    for j, P in enumerate(plens):
        act = wl.group if lengths is None else sum(1 for i in range(wl.group) if t <= lengths[j * wl.group + i])
        if act == 0:
            continue
        lo = (P - 1) // 16 * 16 if share else 0
        n_rows += act
        pos += lo + act * (P + t - 1 - lo)
    return n_rows, pos


def decode_step_bytes(wl: W.Workload, plens, t: int, lengths=None) -> int:
    """Bytes the decode step t must move: both models' weights once, the K/V
    context of every active row for both models (a shared prompt prefix once
    per group), the K/V append and the embedding rows."""
    n_rows, pos = _context_positions(wl, plens, t, lengths)
    if n_rows == 0:
        return 0
    kv = kv_bytes_per_token(wl.senior) + kv_bytes_per_token(wl.junior)
    esz_s = 2 if wl.senior.dtype == "bf16" else 4
    esz_j = 2 if wl.junior.dtype == "bf16" else 4
    return (weight_bytes(wl.senior) + weight_bytes(wl.junior) + pos * kv + n_rows * kv
            + n_rows * (esz_s * wl.senior.d_model + esz_j * wl.junior.d_model))


def attention_bytes(wl: W.Workload, plens, steps: int, lengths=None) -> int:
    """K/V bytes the decode attention must read over `steps` decode steps (a
    shared prompt prefix once per group)."""
    kv = kv_bytes_per_token(wl.senior) + kv_bytes_per_token(wl.junior)
    return sum(kv * _context_positions(wl, plens, t, lengths)[1] for t in range(1, steps + 1))


def prefill_flops(wl: W.Workload, plens) -> float:
    f = 0.0
    for s in (wl.senior, wl.junior):
        d, hd = s.d_model, s.head_dim
        body = s.n_layers * (d * (s.n_q_heads + 2 * s.n_kv_heads) * hd + s.n_q_heads * hd * d + 3 * d * s.ffn_dim)
        M = sum(P - 1 for P in plens)
        f += 2.0 * M * body
        f += sum(4.0 * (P - 1) * P / 2 * s.n_q_heads * hd * s.n_layers for P in plens)
    return f




# ------------------------------------------------------- HBM traffic counters
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_traffic_qwen_by_kernel.txt")
CSRC = os.path.join(ROOT, "paper_2606_28166_amd", "csrc")
PMC_COPY_BYTES = 1 << 30
PMC_WARM = 1000          # graph-replayed steps first: contexts ~1255 .. 1279 in the measured steps
PMC_STEPS = 24
# kernel classes of the decode step at the Qwen shapes (128 rows): (name,
# kernel-name substring, source file)
PMC_CLASSES = (("attention", "attn_rows_kernel", "k_attn.hip"),
               ("qkv_o", "gemm_stream_kernel<4, 4, false, 0>", "k_stream.hip"),
               ("ffn_partial", "gemm_stream_kernel<4, 4, true, 0>", "k_stream.hip"),
               ("gate_up_swiglu", "gemm_stream_kernel<4, 4, true, 2>", "k_stream.hip"),
               ("lm_heads", "gemm_stream_kernel<4, 4, true, 3>", "k_stream.hip"),
               ("resid_norm_split", "resid_norm_kernel<1>", "k_misc.hip"),
               ("resid_norm_f16", "resid_norm_kernel<2>", "k_misc.hip"),
               ("qkv_post", "qkv_post_kernel", "k_misc.hip"),
               ("swiglu_finish", "swiglu_finish_kernel", "k_misc.hip"),
               ("gumbel_noise", "gumbel_noise_kernel", "k_misc.hip"),
               ("sample_finish", "sample_finish_kernel", "k_misc.hip"),
               ("sample_partials", "sample_partials_kernel", "k_misc.hip"))
PMC_REGEX = "attn_rows|gemm_stream|resid_norm|qkv_post|swiglu_finish|gumbel_noise|sample_finish|sample_partials|copy"


def source_digest(name: str) -> str:
    import hashlib
    with open(os.path.join(CSRC, name), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic_ratio():
    """HBM bytes (FETCH_SIZE + WRITE_SIZE, calibrated on a plain copy) per
    algorithmic K/V byte of the decode attention kernel, from the committed
    rocprofv3 counter summary; None when that summary is missing or was taken
    on a different version of the kernel source."""
    try:
        txt = open(TRAFFIC_FILE).read()
        d = json.loads(txt[txt.index("\n{") + 1:])
        att = d["classes"]["attention"]
        if att["source_sha256_16"] != source_digest("k_attn.hip"):
            return None
        return float(att["traffic_over_algorithmic"])
    except (OSError, IndexError, KeyError, ValueError):
        return None


def pmc_run(warm: int = PMC_WARM) -> None:
    """The program the counter passes profile: a 1 GiB device copy (what
    FETCH_SIZE / WRITE_SIZE report for exactly that many bytes read and
    written), `warm` decode steps of the Qwen-shaped rollout replayed from
    the step graph (1000: the contexts reach the middle of the 2048-token
    rollout; 0 for the classes whose traffic does not depend on the context),
    a second, 4 MiB copy that marks where the measured steps begin, then
    PMC_STEPS decode steps launched from the host (one dispatch per kernel)."""
    import torch
    from paper_2606_28166_amd import _lib as L
    from paper_2606_28166_amd.engine import TandemEngine

    dev = torch.device("cuda:0")
    print("pmc: calibration copy", flush=True)
    x = torch.empty(PMC_COPY_BYTES // 4, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    del x, y
    wl = W.workload("qwen")
    wl.sample.max_new = warm + PMC_STEPS + 8           # every row still runs in the measured steps
    ws, wj, prompts, bnd = W.make_all(wl)
    print("pmc: weights generated", flush=True)
    eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed,
                       max_seqs=wl.n_seqs, max_ctx=max(len(p) for p in prompts) - 1 + wl.sample.max_new,
                       max_prefill_tokens=4096, boundary_words=W.boundary_bits(bnd))
    torch.cuda.synchronize()
    print("pmc: engine ready", flush=True)
    eng.prefill(prompts, wl.group)
    torch.cuda.synchronize()
    print("pmc: prefill done", flush=True)
    for t in range(warm):
        eng.step()
        if (t + 1) % 250 == 0:
            torch.cuda.synchronize()
            print(f"pmc: {t + 1} graph steps", flush=True)
    torch.cuda.synchronize()
    m = torch.empty(1 << 20, dtype=torch.float32, device=dev)
    m2 = torch.empty_like(m)
    m2.copy_(m)                                  # marker: the measured steps follow
    torch.cuda.synchronize()
    eng.timing(L.TIMING_EAGER)
    for _ in range(PMC_STEPS):
        eng.step()
    torch.cuda.synchronize()
    eng.close()
    print("pmc run done", flush=True)


def class_weight_bytes(wl: W.Workload) -> dict:
    """Weight bytes each streaming-GEMM class of one decode step reads, both
    models (bf16): split-activation QKV and O; the fp16 split-K products (the
    down projections, and the gate/up of an FFN narrower than 8192); the
    gate/up products with the SwiGLU epilogue; the two LM heads."""
    out = {"qkv_o": 0, "ffn_partial": 0, "gate_up_swiglu": 0, "lm_heads": 0}
    for s in (wl.senior, wl.junior):
        d, hd, F = s.d_model, s.head_dim, s.ffn_dim
        out["qkv_o"] += 2 * s.n_layers * (d * (s.n_q_heads + 2 * s.n_kv_heads) * hd + s.n_q_heads * hd * d)
        out["ffn_partial"] += 2 * s.n_layers * F * d
        out["ffn_partial" if F < 8192 else "gate_up_swiglu"] += 2 * s.n_layers * 2 * F * d
        out["lm_heads"] += 2 * s.vocab * d
    return out


def pmc_analyze(fetch_csv: str, write_csv: str, warm: int = PMC_WARM) -> dict:
    """Per kernel class, the HBM bytes of the measured steps' dispatches
    (counter KiB x copy bytes / copy counter KiB) against the algorithmic
    bytes of that class: the K/V context for decode attention (a shared
    prompt prefix once per group), the weights each GEMM class streams (the
    LM heads' sampling epilogue also reads one row of Gumbel noise per row,
    R x V x 4 bytes, counted apart), the noise the noise kernel writes; the
    split-K reductions and the other helpers have none of their own (their
    bytes are reported per step and as a fraction of all weight bytes)."""
    import csv
    wl = W.workload("qwen")
    plens = [wl.prompt_len] * wl.n_prompts
    res = {"copy_bytes": PMC_COPY_BYTES, "prompt_len": wl.prompt_len,
           "decode_steps": [warm + 1, warm + PMC_STEPS], "classes": {}}
    per = {}
    for name, path in (("fetch", fetch_csv), ("write", write_csv)):
        rows = sorted((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"]))
                      for r in csv.DictReader(open(path)))
        copies = [(i, v) for i, k, v in rows if "copy" in k.lower()]
        if len(copies) < 2:
            raise SystemExit(f"{path}: expected the calibration copy and the marker copy")
        cal = max(v for _, v in copies)
        marker = copies[-1][0]
        scale = PMC_COPY_BYTES / cal
        res[name] = {"copy_counter_kib": cal, "scale_bytes_per_kib": scale}
        for cname, sub, _ in PMC_CLASSES:
            vals = [v * scale for i, k, v in rows if i > marker and sub in k]
            per.setdefault(cname, {})[name] = (sum(vals), len(vals))
    kv = kv_bytes_per_token(wl.senior) + kv_bytes_per_token(wl.junior)
    t0, t1 = warm + 1, warm + PMC_STEPS
    alg = {"attention": sum(kv * _context_positions(wl, plens, t)[1] for t in range(t0, t1 + 1)),
           "gumbel_noise": PMC_STEPS * wl.n_seqs * wl.senior.vocab * 4,
           "sample_partials": PMC_STEPS * 2 * wl.n_seqs * wl.senior.vocab * 4}
    for k, v in class_weight_bytes(wl).items():
        alg[k] = PMC_STEPS * v
    wbytes = PMC_STEPS * (weight_bytes(wl.senior) + weight_bytes(wl.junior))
    for cname, sub, srcf in PMC_CLASSES:
        (fb, fn), (wb, wn) = per[cname]["fetch"], per[cname]["write"]
        if fn == 0 and wn == 0:
            continue                              # not collected in these passes
        if fn != wn:
            raise SystemExit(f"{cname}: {fn} fetch dispatches against {wn} write dispatches")
        c = {"kernel": sub, "source_sha256_16": source_digest(srcf), "steps": [t0, t1], "dispatches": fn,
             "dispatches_per_step": fn / PMC_STEPS, "fetch_bytes": fb, "write_bytes": wb,
             "bytes_per_step": (fb + wb) / PMC_STEPS, "over_weight_bytes": (fb + wb) / wbytes}
        if cname in alg:
            c["algorithmic_bytes"] = alg[cname]
            c["traffic_over_algorithmic"] = (fb + wb) / alg[cname]
        res["classes"][cname] = c
    return res


# ------------------------------------------------------------------ CPU oracle
def cpu_baseline(wl: W.Workload, ws, wj, prompts, steps: int):
    """The oracle (float64 NumPy, as it stands) on prompt 0's G rows: its
    prefill plus `steps` decode steps, timed after the float64 weight copies
    are built."""
    from oracle.rollout import rollout, build_models
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        cores = len(os.sched_getaffinity(0))
    sen, jun = build_models(wl, ws, wj)
    t0 = time.perf_counter()
    rollout(sen, jun, prompts, wl.group, wl.switch, wl.sample, wl.philox_seed, W.make_boundary(wl),
            seq_subset=list(range(wl.group)), max_steps=steps)
    dt = time.perf_counter() - t0
    return {"value": round(wl.group * steps / dt, 3), "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "precision": "f64",
            "sample": f"prompt 0 x G={wl.group} rows: prefill of {len(prompts[0]) - 1} prompt tokens + "
                      f"{steps} decode steps ({wl.group * steps} co-generated tokens) in {dt:.1f} s, "
                      f"float64 NumPy on the same bf16-valued weights",
            "host_cpus": os.cpu_count(), "affinity": len(os.sched_getaffinity(0))}


# ------------------------------------------------------------------------ main
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1, help="timed rollouts requested (capped by --timed-s)")
    ap.add_argument("--warmup", type=int, default=1, help="warmup rollouts requested (the first always runs)")
    ap.add_argument("--workload", default="qwen", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--max-new", type=int, default=None, help="shorter rollouts (development only)")
    ap.add_argument("--budget-s", type=float, default=420.0,
                    help="wall-clock budget of the whole run, counted from process start: optional legs are "
                         "skipped when what is left would not cover them")
    ap.add_argument("--timed-s", type=float, default=75.0,
                    help="the timed region runs as many requested rollouts as fit this many seconds (at least one)")
    ap.add_argument("--warm-s", type=float, default=30.0,
                    help="warmup rollouts after the first run only while they fit this many seconds")
    ap.add_argument("--cpu-steps", type=int, default=16, help="decode steps of the CPU-oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--separate-sample", action="store_true",
                    help="store the logits and sample in a separate pass instead of inside the LM-head GEMMs")
    ap.add_argument("--no-isolated", action="store_true",
                    help="skip the extra rollout that times every kernel class with the forwards serialized")
    ap.add_argument("--no-concurrent", action="store_true",
                    help="skip the extra rollout that times the attention launches in the two-stream schedule")
    ap.add_argument("--no-solo", action="store_true",
                    help="skip the single-model rollout of the senior (the tandem-over-solo step-time ratio)")
    ap.add_argument("--score", type=int, default=0, metavar="STEPS",
                    help="also time tandem_score_step after each of STEPS decode steps (reported as 'scoring')")
    ap.add_argument("--grpo", type=int, default=0, metavar="REPS",
                    help="also time tandem_grpo_loss REPS times over the last rollout's arenas (reported as 'grpo')")
    ap.add_argument("--pmc-run", action="store_true", help="counter mode: the program rocprofv3 --pmc profiles")
    ap.add_argument("--pmc-analyze", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="counter mode: per-class HBM traffic from the two counter passes (JSON)")
    ap.add_argument("--pmc-warm", type=int, default=PMC_WARM,
                    help="counter mode: graph-replayed steps before the measured ones (0: none)")
    args = ap.parse_args()

    if args.pmc_analyze:
        print(json.dumps(pmc_analyze(*args.pmc_analyze, warm=args.pmc_warm), indent=1))
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus > 1 or world > 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: the tandem rollout shards over prompt "
                                   "groups with no per-step exchange, and no multi-GPU path is built"}))
        sys.exit(2)
    if args.pmc_run:
        pmc_run(args.pmc_warm)
        return

    def left() -> float:
        return args.budget_s - (time.perf_counter() - T_START)

    log(f"[bench] {args.workload}: importing torch")
    import torch
    from paper_2606_28166_amd import _lib as LIB
    from paper_2606_28166_amd.engine import TandemEngine, grpo_loss
    log(f"[bench] torch ready ({time.perf_counter() - T_START:.0f}s since start)")

    wl = W.workload(args.workload)
    if args.max_new:
        wl.sample.max_new = args.max_new
    t0 = time.time()
    ws, wj, prompts, bnd = W.make_all(wl)
    plens = [len(p) for p in prompts]
    log(f"[bench] weights generated in {time.time() - t0:.1f}s ({time.perf_counter() - T_START:.0f}s since start)")
    max_ctx = max(plens) - 1 + wl.sample.max_new
    eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed,
                       max_seqs=wl.n_seqs, max_ctx=max_ctx, max_prefill_tokens=4096,
                       boundary_words=W.boundary_bits(bnd))
    log(f"[bench] engine ready: KV arena {eng.kv_bytes / 2**30:.1f} GiB, scratch {eng.scratch_bytes / 2**30:.2f} GiB")
    stream = eng.stream
    L = wl.sample.max_new
    n = wl.n_seqs
    skipped = []

    SEP = LIB.TIMING_SEPARATE_SAMPLE if args.separate_sample else 0

    def rollout_once(timing=0):
        """Prefill + L decode steps; timing = the library's class mask (0: step-graph replays).
        Returns (prefill ms, decode ms, per-class timing or None, wall s)."""
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        w0 = time.perf_counter()
        ev[0].record(stream)
        eng.prefill(prompts, wl.group)
        ev[1].record(stream)
        eng.timing(timing | SEP)
        for _ in range(L):
            eng.step()
        ev[2].record(stream)
        torch.cuda.synchronize()
        tr = eng.timing_read() if timing & 0b1111 else None
        eng.timing(SEP)
        return ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2]), tr, time.perf_counter() - w0

    # ---- warmup: the first rollout captures the step graph and sets the
    # estimate of one rollout's duration
    n_warm, warm_wall, est = 0, 0.0, None
    while n_warm < max(1, args.warmup):
        if n_warm > 0 and (warm_wall + est > args.warm_s or left() < 3 * est):
            break
        p_ms, d_ms, _, w = rollout_once()
        n_warm += 1
        warm_wall += w
        est = w
        log(f"[bench] warmup {n_warm - 1}: prefill {p_ms:.1f} ms, decode {d_ms:.1f} ms ({w:.1f} s)")

    # ---- timed region: whole rollouts, decode steps replayed from the step graph
    n_timed = max(1, min(args.steps, int(args.timed_s // est), int((left() - 2.0 * est) // est)))
    log(f"[bench] timing {n_timed} rollout(s) of {args.steps} requested ({left():.0f}s of budget left)")
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    pre, dec = [], []
    for i in range(n_timed):
        p_ms, d_ms, _, _ = rollout_once()
        pre.append(p_ms)
        dec.append(d_ms)
        log(f"[bench] step {i}: prefill {p_ms:.1f} ms, decode {d_ms:.1f} ms")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    est = wall / n_timed

    out = eng.outputs()
    lengths = out["length"].tolist() if wl.sample.eos_id >= 0 else None     # every run of this batch is identical
    gen = int(out["length"].sum())
    mask = np.arange(L)[None, :] < out["length"][:, None]
    senior_share = float(out["owner"][:, :L][mask].mean())
    toks = gen * n_timed
    ms_per_step = wall * 1e3 / n_timed
    value = toks / wall
    dec_s = sum(dec) / 1e3
    dec_bytes = sum(decode_step_bytes(wl, plens, t, lengths) for t in range(1, L + 1)) * n_timed
    pf = prefill_flops(wl, plens)
    pre_ms = float(np.mean(pre))

    # ---- the dominant kernel's roofline.  Event records captured into a HIP
    # graph carry no launch times, so the attention launches are timed in extra
    # rollouts whose steps are launched from the host, with a HIP event pair
    # around every launch on the stream it runs on: one with the two forwards
    # serialized (each launch alone on the GPU: the kernel's own roofline, and
    # the per-class breakdown), one in the production two-stream schedule.
    traffic_ratio = measured_traffic_ratio() if wl.name in ("qwen", "qwen-paper") else None

    def roofline_of(att, method):
        ms, nl = att
        nbytes = attention_bytes(wl, plens, L, lengths)
        gbs = nbytes / (ms / 1e3) / 1e9
        per = nbytes / max(nl, 1)
        return {"bound": "hbm", "kernel": "decode attention (both models; shared prompt prefix)" if shares_prefix(wl)
                else "decode attention (both models)", "achieved": round(gbs, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                "traffic": None if traffic_ratio is None else int(per * traffic_ratio),
                "launches": nl, "avg_launch_us": round(ms * 1e3 / max(nl, 1), 2),
                "bytes_per_launch": int(per), "method": method}

    roof, roof_conc, breakdown = None, None, None
    if args.no_isolated:
        skipped.append("serialized rollout (--no-isolated)")
    elif left() < 1.8 * est:
        skipped.append(f"serialized rollout (budget: {left():.0f}s left)")
    else:
        _, d_ser, tr, _ = rollout_once(0b1111 | LIB.TIMING_SERIAL)
        breakdown = {k: {"ms": round(v[0], 3), "launches": v[1]} for k, v in tr.items()}
        roof = roofline_of(tr["attention"], "one rollout's decode steps, the two forwards serialized and launched "
                                            "from the host, a HIP event pair around every attention launch")
        log(f"[bench] serialized rollout: decode {d_ser:.1f} ms, attention {tr['attention'][0]:.1f} ms / "
            f"{tr['attention'][1]} launches -> {roof['achieved']:.0f} GB/s ({left():.0f}s of budget left)")

    cpu = None
    if args.no_cpu_baseline:
        skipped.append("cpu baseline (--no-cpu-baseline)")
    elif left() < 120:
        skipped.append(f"cpu baseline (budget: {left():.0f}s left)")
    else:
        log("[bench] timing the CPU oracle sample")
        try:
            cpu = cpu_baseline(wl, ws, wj, prompts, args.cpu_steps)
            log(f"[bench] cpu oracle: {cpu['sample']} ({left():.0f}s of budget left)")
        except MemoryError as e:                  # the float64 copies of the weights do not fit this host
            skipped.append(f"cpu baseline ({e!r})")

    if args.no_concurrent:
        skipped.append("concurrent instrumented rollout (--no-concurrent)")
    elif args.no_isolated or left() < 1.5 * est + 20:
        skipped.append(f"concurrent instrumented rollout (budget: {left():.0f}s left)")
    else:
        _, d_con, tr, _ = rollout_once(1 << LIB.K_ATTENTION)
        roof_conc = roofline_of(tr["attention"], "one rollout's decode steps in the two-stream schedule, launched "
                                                 "from the host, a HIP event pair around every attention launch")
        log(f"[bench] concurrent instrumented rollout: decode {d_con:.1f} ms, attention -> "
            f"{roof_conc['achieved']:.0f} GB/s")

    scoring = None
    if args.score > 0:
        # the dual-distribution scores after each step of a fresh rollout:
        # HIP events on the library's stream around every scoring call (the
        # steps store their logits, as a caller scoring every step would ask)
        eng.timing(LIB.TIMING_SEPARATE_SAMPLE)
        eng.prefill(prompts, wl.group)
        sc_out = torch.empty((wl.n_seqs, 3), dtype=torch.float32, device=eng.dev)
        tot, ns = 0.0, min(args.score, L)
        for _ in range(ns):
            eng.step()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            eng.score(sc_out)
            e1.record(stream)
            torch.cuda.synchronize()
            tot += e0.elapsed_time(e1)
        eng.timing(SEP)
        ms = tot / ns
        nbytes = 4 * n * wl.senior.vocab * 4          # two passes over both models' fp32 logits
        scoring = {"steps": ns, "ms_per_step": round(ms, 4), "bytes_per_step": nbytes,
                   "achieved_gbs": round(nbytes / (ms / 1e3) / 1e9, 1),
                   "frac_of_decode_step": round(ms / (sum(dec) / (L * n_timed)), 4)}
        log(f"[bench] scoring: {ms * 1e3:.1f} us per step ({scoring['achieved_gbs']:.0f} GB/s)")

    grpo = None
    if args.grpo > 0:
        # the senior-only GRPO loss pieces over the last rollout's arenas (its
        # authorship, log-prob and length arenas as tandem_step left them),
        # seeded binary rewards and the recorded log-probs plus seeded offsets
        # as the current policy's: HIP events on the stream the call runs on
        g = torch.Generator(device="cpu").manual_seed(41)
        rewards = (torch.rand(n, generator=g) < 0.5).float().to(eng.dev)
        lp_new = eng.logprob[:n] + (0.15 * torch.randn(eng.logprob[:n].shape, generator=g)).to(eng.dev)
        grpo_ws = torch.empty(LIB.tandem_grpo_workspace_size(LIB.GrpoCfg(n // wl.group, wl.group, eng.max_new, 0.2)),
                              dtype=torch.uint8, device=eng.dev)
        args_g = (rewards, eng.owner[:n], eng.length[:n], eng.logprob[:n], lp_new, wl.group)
        ref_g = grpo_loss(*args_g, workspace=grpo_ws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.grpo):
            grpo_loss(*args_g, workspace=grpo_ws)
        e1.record(stream)
        torch.cuda.synchronize()
        ms_eager = e0.elapsed_time(e1) / args.grpo
        # the launches of one call captured in a HIP graph and replayed:
        # device time without the host's per-call marshalling
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            cap_g = grpo_loss(*args_g, workspace=grpo_ws)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.grpo):
            graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.grpo
        same = all(torch.equal(ref_g[k], cap_g[k]) for k in ("advantages", "loss", "n_masked", "grad"))
        lens = eng.length[:n].cpu().numpy().astype(np.int64)
        # per position t < length: authorship byte + two log-probs read; every
        # position of the [S][T] arena: gradient written; per rollout: reward,
        # length, advantage
        nbytes = int(9 * lens.sum() + 4 * n * eng.max_new + 12 * n)
        grpo = {"calls": args.grpo, "us_per_call": round(ms * 1e3, 2), "timing": "HIP graph replays",
                "us_per_call_eager": round(ms_eager * 1e3, 2), "replays_match_eager": same,
                "rollouts": n, "stride": eng.max_new,
                "positions": int(lens.sum()), "bytes_per_call": nbytes,
                "achieved_gbs": round(nbytes / (ms / 1e3) / 1e9, 1),
                "frac_of_8tbs": round(nbytes / (ms / 1e3) / 8e12, 4)}
        log(f"[bench] grpo loss: {ms * 1e3:.1f} us per call replayed ({ms_eager * 1e3:.1f} us eager; "
            f"{grpo['achieved_gbs']:.0f} GB/s over {grpo['positions']} positions; replays match: {same})")

    # ---- the senior alone through the same kernels (a handle without a
    # junior): the decode step-time ratio of the tandem rollout over a
    # single-model rollout of the same batch, which the paper reports as about
    # 2x latency and 0.5x throughput on its two-GPU layout
    solo = None
    tandem_dec_ms = sum(dec) / (L * n_timed)
    if args.no_solo:
        skipped.append("solo rollout (--no-solo)")
    elif left() < 1.0 * est + 30:
        skipped.append(f"solo rollout (budget: {left():.0f}s left)")
    else:
        sen_model = eng.sen
        eng.close()
        del eng.kv, eng.scratch
        torch.cuda.empty_cache()
        seng = TandemEngine(wl.senior, None, None, None, wl.switch, wl.sample, wl.philox_seed, max_seqs=n,
                            max_ctx=max_ctx, max_prefill_tokens=4096, models=(sen_model, None))
        seng.timing(SEP)
        seng.prefill(prompts, wl.group)
        seng.step()                                  # captures the single-model step graph
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev[0].record(seng.stream)
        seng.prefill(prompts, wl.group)
        ev[1].record(seng.stream)
        for _ in range(L):
            seng.step()
        ev[2].record(seng.stream)
        torch.cuda.synchronize()
        s_pre, s_dec = ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2])
        seng.close()
        solo_ms = s_dec / L
        solo = {"solo_decode_ms_per_step": round(solo_ms, 4), "tandem_decode_ms_per_step": round(tandem_dec_ms, 4),
                "step_time_ratio": round(tandem_dec_ms / solo_ms, 4),
                "throughput_ratio": round(solo_ms / tandem_dec_ms, 4),
                "solo_prefill_ms": round(s_pre, 3), "tandem_prefill_ms": round(pre_ms, 3),
                "solo_tokens_per_s": round(gen / ((s_pre + s_dec) / 1e3), 2),
                "method": "one rollout of the same batch with a handle that has no junior (the senior emits every "
                          "token, same kernels, step graph), HIP events around prefill and decode",
                "paper_context": "tandem step about 2x a single-model step and rollout throughput about 0.5x "
                                 "single-model vLLM, senior and junior on two A100 80 GB GPUs"}
        log(f"[bench] solo senior rollout: decode {s_dec:.1f} ms ({solo_ms:.3f} ms/step); tandem/solo step time "
            f"{solo['step_time_ratio']:.3f}")

    bf16 = wl.senior.dtype == "bf16"
    res = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": n_timed,
        "warmup": n_warm,
        "steps_requested": args.steps,
        "warmup_requested": args.warmup,
        "step_unit": "one whole rollout: prefill of every prompt + %d tandem decode steps over %d rows" % (L, n),
        "ms_per_step": round(ms_per_step, 3),
        "timed_wall_s": round(wall, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16+fp16" if bf16 else "f32",
        "dtype_detail": ("bf16 weights and K/V cache, fp32 accumulation and residual; QKV and O products on bf16 "
                         "hi+lo split activations (two bf16 MFMAs), FFN and LM-head products fp16 x fp16 MFMA on "
                         "fp16 copies of the bf16 weights; attention bf16 K/V with hi+lo q and P; fp32 sampling")
                        if bf16 else "fp32 weights, activations and K/V",
        "data": "synthetic",
        "sampling": ("separate pass over stored logits" if SEP or not bf16 or (n > 128 and wl.sample.eos_id < 0)
                     else "separate pass while more than 128 rows are launched, then (after compaction) inside the "
                          "LM-head GEMMs" if n > 128
                     else "inside the LM-head GEMMs (Gumbel noise beside the forwards, no logits stored)"),
        "config": {"workload": DESCRIPTIONS[wl.name], "name": wl.name, "rows": n,
                   "prompt_len": plens[0] if min(plens) == max(plens) else [min(plens), max(plens)],
                   "max_new": L, "senior_layers": wl.senior.n_layers, "junior_layers": wl.junior.n_layers,
                   "vocab": wl.senior.vocab},
        "roofline": roof,
        "roofline_concurrent": roof_conc,
        "cpu_baseline": cpu,
        "decode_tokens_per_s": round(gen * n_timed / dec_s, 2),
        "generated_tokens": gen,
        "decode_ms_per_token_step": round(sum(dec) / (L * n_timed), 4),
        "decode_hbm_gbs": round(dec_bytes / dec_s / 1e9, 1),
        "decode_hbm_frac": round(dec_bytes / dec_s / 1e9 / HBM_PEAK_GBS, 4),
        "prefill_ms": round(pre_ms, 3),
        "prefill_tflops": round(pf / (pre_ms / 1e3) / 1e12, 1),
        "prefill_mfma_frac": round(pf / (pre_ms / 1e3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
        "senior_share": round(senior_share, 4),
        "breakdown": breakdown,
        "skipped": skipped,
        "run_wall_s": round(time.perf_counter() - T_START, 1),
    }
    res["tandem_over_solo"] = solo
    if scoring is not None:
        res["scoring"] = scoring
    if grpo is not None:
        res["grpo"] = grpo
    eng.close()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
