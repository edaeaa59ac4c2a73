"""The benchmark's host-side accounting, checked on the CPU: the algorithmic
byte counts against the generated weights and a row-by-row count of the K/V
context, and the counter analysis against synthetic counter files."""
import csv
import os
import sys

import numpy as np
import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench as B  # noqa: E402


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_weight_bytes_count_the_generated_projection_and_head_matrices(name):
    wl = W.workload(name)
    ws, wj, _, _ = W.make_all(wl)
    for shape, w in ((wl.senior, ws), (wl.junior, wj)):
        esz = 2 if shape.dtype == "bf16" else 4
        mats = [k for k in w if any(t in k for t in ("w_qkv", "w_o", "w_gate_up", "w_down", "lm_head"))]
        n = sum(int(np.prod(w[k].shape)) for k in mats)
        if "lm_head" not in w:            # a tied head reads the embedding matrix
            n += int(np.prod(w["embed"].shape))
        assert B.weight_bytes(shape) == esz * n


def test_class_weight_bytes_partition_the_weights():
    for name in ("qwen", "small", "self-paired"):
        wl = W.workload(name)
        c = B.class_weight_bytes(wl)
        assert sum(c.values()) == B.weight_bytes(wl.senior) + B.weight_bytes(wl.junior)


@pytest.mark.parametrize("t", [1, 7, 300])
def test_context_positions_against_a_row_by_row_count(t):
    wl = W.workload("longcot")
    plens = [64 + 37 * j for j in range(wl.n_prompts)]
    rng = np.random.default_rng(5)
    lengths = rng.integers(1, 400, size=wl.n_seqs)
    n_rows, pos = B._context_positions(wl, plens, t, lengths.tolist())
    share = B.shares_prefix(wl)
    want_rows, want_pos = 0, 0
    for j, P in enumerate(plens):
        lo = (P - 1) // 16 * 16 if share else 0
        rows = [j * wl.group + i for i in range(wl.group) if t <= lengths[j * wl.group + i]]
        if rows:
            want_pos += lo                       # the shared prefix once per group with a running row
        for _ in rows:
            want_rows += 1
            want_pos += P + t - 1 - lo           # positions 0 .. P + t - 2, minus the shared prefix
    assert (n_rows, pos) == (want_rows, want_pos)


def _write(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Value"])
        w.writerows(rows)


def test_pmc_analyze_scales_by_the_calibration_copy_and_counts_after_the_marker(tmp_path):
    # the 1 GiB calibration copy reads as 2^19 KiB (x2.0 bytes per KiB), the
    # marker copy separates the warm-up from the measured steps; dispatches
    # before the marker are not counted
    steps = B.PMC_STEPS
    fetch = [(1, "copyBuffer", 524288.0), (2, "gemm_stream_kernel<4, 4, true, 3>(x)", 999.0),
             (3, "copyBuffer", 4096.0)]
    write = [(1, "copyBuffer", 1048576.0), (2, "gemm_stream_kernel<4, 4, true, 3>(x)", 999.0),
             (3, "copyBuffer", 4096.0)]
    for i in range(steps):
        fetch.append((10 + i, "gemm_stream_kernel<4, 4, true, 3>(x)", 100.0))
        write.append((10 + i, "gemm_stream_kernel<4, 4, true, 3>(x)", 10.0))
    _write(tmp_path / "f.csv", fetch)
    _write(tmp_path / "w.csv", write)
    r = B.pmc_analyze(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), warm=0)
    c = r["classes"]["lm_heads"]
    assert c["dispatches"] == steps
    assert c["fetch_bytes"] == pytest.approx(steps * 100.0 * 2048.0)
    assert c["write_bytes"] == pytest.approx(steps * 10.0 * 1024.0)
    wl = W.workload("qwen")
    alg = steps * 2 * wl.senior.vocab * (wl.senior.d_model + wl.junior.d_model)
    assert c["algorithmic_bytes"] == alg
    assert c["traffic_over_algorithmic"] == pytest.approx(steps * (100.0 * 2048 + 10.0 * 1024) / alg)
    assert set(r["classes"]) == {"lm_heads"}
