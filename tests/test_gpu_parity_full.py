"""GPU parity at the workloads' full sizes, in the benchmark's launch configuration.

The oracle follows a subset of the batch's sequences (each sequence depends
only on the weights, its prompt, the seed and its id, so a subset is exact);
the library runs the whole batch with the benchmark's capacity, the other
sequences sampling freely next to the checked ones.
"""
import numpy as np
import pytest

import workloads as W
from tests import parity as P

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def test_qwen_full_size_prompt0_first_64_steps():
    """Teacher-forced steps at the full Qwen shapes, then, on the same handle,
    64 free-running steps replayed from the captured step graph: bit-equal to
    the same steps launched eagerly, and equal to the free-running oracle on
    prompt 0's rows up to each row's first in-band step (the first free-running
    divergence is reported)."""
    wl = W.workload("qwen")
    P.log("case qwen full size: 36 + 28 layers, V 151936, 128 rows, capacity 2303 positions; "
          "prompt 0's 8 rows, 64 steps")
    rows = list(range(wl.group))
    seen = {}

    def free(eng, prompts, ref):
        graph = P.free_run(eng, prompts, wl.group, 64, eager=False)
        eager = P.free_run(eng, prompts, wl.group, 64, eager=True)
        for k in graph:
            np.testing.assert_array_equal(graph[k], eager[k], err_msg=k)
        seen["div"] = P.first_divergence(graph, ref, np.array(rows), 64)

    p = P.run(wl, steps=64, logits_at=(1, 32, 64), seq_subset=rows, after=free)
    P.check(p, P.TOL_BF16)
    first, full, n = seen["div"]
    P.log(f"  free-running graph replays: {full}/{len(rows)} rows identical to the oracle over 64 steps, "
          f"{n} tokens compared, first divergence at step {first}")


def test_small_full_size_prompt0_all_512_steps():
    """The small pair at its full shape (8 + 4 layers, V 32000) over the whole
    64-row batch and all 512 steps; the oracle follows prompt 0's 8 rows."""
    wl = W.workload("small")
    P.log("case small full size: 8 + 4 layers, V 32000, 64 rows, 512 steps; prompt 0's 8 rows")
    p = P.run(wl, logits_at=(1, 256, 512), seq_subset=list(range(wl.group)))
    P.check(p, P.TOL_BF16)


def test_qwen_shapes_context_beyond_2048_positions():
    """Contexts past 2048 positions: one 2040-token prompt x G = 4 at the Qwen
    shapes (2+2 layers), 24 decode steps (positions 2039 .. 2062), logits
    checked at the first and the last step."""
    wl = W.workload("qwen").replace(n_prompts=1, group=4, prompt_len=2040, gain_jitter=0.05)
    wl.senior.n_layers, wl.junior.n_layers = 2, 2
    wl.sample.max_new = 24
    P.log("case long context: Qwen shapes 2+2 layers, prompt 2040 tokens, G=4, 24 steps")
    p = P.run(wl, logits_at=(1, 24))
    P.check(p, P.TOL_BF16)


def test_longcot_one_group_256_steps():
    wl = W.workload("longcot")
    P.log("case long-CoT: ragged prompts 64..512, EOS on, 32-token chunk handoffs, 256 rows; "
          "prompt 5's 8 rows, 256 steps")
    rows = [5 * wl.group + i for i in range(wl.group)]
    p = P.run(wl, steps=256, logits_at=(1, 128, 256), seq_subset=rows)
    P.check(p, P.TOL_BF16)


def test_wide_batch_16_rows_128_steps():
    wl = W.workload("wide")
    P.log("case wide: 1024 rows, p = 0.5 per token; 16 rows spread over the batch, 128 steps")
    rows = sorted({(97 * k + 13 * (k % 3)) % wl.n_seqs for k in range(16)})
    assert len(rows) == 16
    p = P.run(wl, steps=128, logits_at=(1, 64, 128), seq_subset=rows)
    P.check(p, P.TOL_BF16)
