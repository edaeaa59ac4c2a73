"""HBM traffic of the decode attention kernel, from rocprofv3 counters.

Run mode (the program rocprofv3 profiles): a plain device copy of known size
(the calibration: what FETCH_SIZE / WRITE_SIZE report for exactly N bytes
read and N bytes written), then a short tandem rollout of the Qwen-shaped
models (128 rows, prompts of PROMPT_LEN tokens so the contexts sit in the
middle of the benchmark's rollout) with eagerly launched decode steps (one
dispatch per kernel):

    cd /tmp && rocprofv3 --pmc FETCH_SIZE -d <dir> -o fetch --output-format csv -- \\
        python3 <repo>/paper_2606_28166_amd/pmc_probe.py
    cd /tmp && rocprofv3 --pmc WRITE_SIZE -d <dir> -o write --output-format csv -- \\
        python3 <repo>/paper_2606_28166_amd/pmc_probe.py

Analysis mode: per attention dispatch, counter KiB x (copy bytes / copy
counter KiB) against the algorithmic K/V bytes of that dispatch; prints a
JSON summary (the ratio traffic / algorithmic bytes is what the benchmark
applies to its own launches):

    python3 paper_2606_28166_amd/pmc_probe.py --analyze <fetch csv> <write csv>
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

COPY_BYTES = 1 << 30
STEPS = 24
PROMPT_LEN = 1280        # contexts 1279 .. 1302: the middle of the 2048-token rollout from 256-token prompts
ATTN_SRC = os.path.join(ROOT, "paper_2606_28166_amd", "csrc", "k_attn.hip")


def kernel_digest() -> str:
    with open(ATTN_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def run() -> None:
    import torch
    import workloads as W
    from paper_2606_28166_amd import _lib as L
    from paper_2606_28166_amd.engine import TandemEngine

    dev = torch.device("cuda:0")
    x = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    y.copy_(x)                                   # calibration: COPY_BYTES read, COPY_BYTES written
    torch.cuda.synchronize()
    del x, y

    wl = W.workload("qwen")
    wl.sample.max_new = STEPS
    wl.prompt_len = PROMPT_LEN
    ws, wj, prompts, bnd = W.make_all(wl)
    eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed,
                       max_seqs=wl.n_seqs, max_ctx=max(len(p) for p in prompts) - 1 + STEPS,
                       max_prefill_tokens=4096, boundary_words=W.boundary_bits(bnd))
    eng.prefill(prompts, wl.group)
    eng.timing(L.TIMING_EAGER)                   # one dispatch per kernel (no graph replay)
    for _ in range(STEPS):
        eng.step()
    torch.cuda.synchronize()
    eng.close()
    print("pmc_probe done", flush=True)


def _rows(path):
    out = []
    for r in csv.DictReader(open(path)):
        out.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
    out.sort()
    return out


def analyze(fetch_csv: str, write_csv: str) -> dict:
    import workloads as W
    wl = W.workload("qwen")
    wl.prompt_len = PROMPT_LEN
    res = {"kernel_source_sha256_16": kernel_digest(), "copy_bytes": COPY_BYTES, "prompt_len": PROMPT_LEN,
           "decode_steps": STEPS}
    for name, path in (("fetch", fetch_csv), ("write", write_csv)):
        rows = _rows(path)
        copies = [v for _, k, v in rows if "copy" in k.lower() or "elementwise" in k.lower()]
        if not copies:
            raise SystemExit(f"no copy kernel in {path}")
        cal = max(copies)                        # KiB the counter reports for COPY_BYTES
        # the decode launches are the last STEPS * (both models' layers)
        # attention dispatches (the prefill's come first)
        n_dec = STEPS * (wl.senior.n_layers + wl.junior.n_layers)
        att = [(k, v) for _, k, v in rows if "attn_mfma_kernel" in k][-n_dec:]
        res[name] = {"copy_counter_kib": cal, "scale_bytes_per_kib": COPY_BYTES / cal,
                     "attention_dispatches": len(att)}
        res[name]["attention_counter_kib"] = [v for _, v in att]
    # decode attention dispatches in launch order: per step, the junior's 28
    # layers and the senior's 36 (two streams); K/V bytes per dispatch depend
    # only on the model and the step's context
    kv = {"senior": 2 * wl.senior.n_kv_heads * wl.senior.head_dim * 2,
          "junior": 2 * wl.junior.n_kv_heads * wl.junior.head_dim * 2}   # bytes per position per layer
    rows_per = wl.n_seqs
    P = wl.prompt_len
    att_alg = []
    for t in range(1, STEPS + 1):
        ctx = P - 1 + t                           # the step's context, new position included
        att_alg += [rows_per * ctx * kv["junior"]] * wl.junior.n_layers
        att_alg += [rows_per * ctx * kv["senior"]] * wl.senior.n_layers
    fet = [v * res["fetch"]["scale_bytes_per_kib"] for v in res["fetch"]["attention_counter_kib"]]
    wri = [v * res["write"]["scale_bytes_per_kib"] for v in res["write"]["attention_counter_kib"]]
    n = min(len(fet), len(att_alg))
    res["dispatches_compared"] = n
    res["algorithmic_bytes"] = sum(att_alg[:n])
    res["fetch_bytes"] = sum(fet[:n])
    res["write_bytes"] = sum(wri[:n])
    res["traffic_over_algorithmic"] = (res["fetch_bytes"] + res["write_bytes"]) / res["algorithmic_bytes"]
    for k in ("fetch", "write"):
        del res[k]["attention_counter_kib"]
    return res


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--analyze", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"))
    a = ap.parse_args()
    if a.analyze:
        print(json.dumps(analyze(*a.analyze), indent=1))
    else:
        run()


if __name__ == "__main__":
    main()
