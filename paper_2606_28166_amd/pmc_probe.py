"""HBM traffic of the decode attention kernel, from rocprofv3 counters.

Run mode (the program rocprofv3 profiles): a plain device copy of known size
(the calibration: what FETCH_SIZE / WRITE_SIZE report for exactly N bytes
read and N bytes written), then the benchmark's Qwen-shaped rollout (16
prompts of 256 tokens x G = 8 rows): WARM decode steps replayed from the
step graph, so that the contexts reach the middle of the benchmark's
2048-token rollout, then STEPS decode steps launched eagerly (one dispatch
per kernel).  Counters are collected for the attention kernels and the copy
only:

    cd /tmp && rocprofv3 --pmc FETCH_SIZE --kernel-include-regex 'attn_shared|copy' -d <dir> -o fetch \\
        --output-format csv -- python3 <repo>/paper_2606_28166_amd/pmc_probe.py
    cd /tmp && rocprofv3 --pmc WRITE_SIZE --kernel-include-regex 'attn_shared|copy' -d <dir> -o write \\
        --output-format csv -- python3 <repo>/paper_2606_28166_amd/pmc_probe.py

Analysis mode: the counters of the last STEPS steps' attention dispatches
(both models; each reads the shared prompt prefix once per block of rows and
every row's own positions) x
(copy bytes / copy counter KiB) against the algorithmic K/V bytes of those
steps (a shared prompt prefix once per group); prints a JSON summary (the
ratio traffic / algorithmic bytes is what the benchmark applies to its own
attention calls):

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
WARM = 1000              # graph-replayed steps first: contexts ~1255 .. 1279 in the measured steps
STEPS = 24
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
    wl.sample.max_new = WARM + STEPS
    ws, wj, prompts, bnd = W.make_all(wl)
    eng = TandemEngine(wl.senior, ws, wl.junior, wj, wl.switch, wl.sample, wl.philox_seed,
                       max_seqs=wl.n_seqs, max_ctx=max(len(p) for p in prompts) - 1 + WARM + STEPS,
                       max_prefill_tokens=4096, boundary_words=W.boundary_bits(bnd))
    eng.prefill(prompts, wl.group)
    for t in range(WARM):
        eng.step()
        if (t + 1) % 250 == 0:
            torch.cuda.synchronize()
            print(f"pmc_probe: {t + 1} graph steps", flush=True)
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
    P = wl.prompt_len
    lo = (P - 1) // 16 * 16                      # the shared prefix (G > 1, bf16, head_dim 128)
    res = {"kernel_source_sha256_16": kernel_digest(), "copy_bytes": COPY_BYTES, "prompt_len": P,
           "shared_prefix": lo, "decode_steps": [WARM + 1, WARM + STEPS]}
    for name, path in (("fetch", fetch_csv), ("write", write_csv)):
        rows = _rows(path)
        copies = [v for _, k, v in rows if "copy" in k.lower() or "elementwise" in k.lower()]
        if not copies:
            raise SystemExit(f"no copy kernel in {path}")
        cal = max(copies)                        # KiB the counter reports for COPY_BYTES
        # the measured launches are the last STEPS * (both models' layers)
        # attention dispatches
        n_dec = STEPS * (wl.senior.n_layers + wl.junior.n_layers)
        att = [(k, v) for _, k, v in rows if "attn_shared_kernel" in k][-n_dec:]
        res[name] = {"copy_counter_kib": cal, "scale_bytes_per_kib": COPY_BYTES / cal,
                     "attention_dispatches": len(att)}
        res[name]["attention_counter_kib"] = [v for _, v in att]
    # algorithmic K/V bytes of those steps: per layer of a model, the shared
    # prefix once per prompt and each row's positions lo .. its context end
    kv = (2 * wl.senior.n_kv_heads * wl.senior.head_dim * 2 * wl.senior.n_layers
          + 2 * wl.junior.n_kv_heads * wl.junior.head_dim * 2 * wl.junior.n_layers)   # bytes per position
    alg = 0
    for t in range(WARM + 1, WARM + STEPS + 1):
        ctx = P - 1 + t                           # the step's context, new position included
        alg += kv * (wl.n_prompts * lo + wl.n_seqs * (ctx - lo))
    fet = [v * res["fetch"]["scale_bytes_per_kib"] for v in res["fetch"]["attention_counter_kib"]]
    wri = [v * res["write"]["scale_bytes_per_kib"] for v in res["write"]["attention_counter_kib"]]
    if len(fet) != n_dec or len(wri) != n_dec:
        raise SystemExit(f"expected {n_dec} attention dispatches, found {len(fet)} / {len(wri)}")
    res["dispatches_compared"] = n_dec
    res["algorithmic_bytes"] = alg
    res["fetch_bytes"] = sum(fet)
    res["write_bytes"] = sum(wri)
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
