"""GPU parity at the workloads' full sizes, in the benchmark's launch configuration.

The oracle follows a subset of the batch's sequences (each sequence depends
only on the weights, its prompt, the seed and its id, so a subset is exact);
the library runs the whole batch with the benchmark's capacity, the other
sequences sampling freely next to the checked ones.
"""
import pytest

import workloads as W
from tests import parity as P

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def test_qwen_full_size_prompt0_first_64_steps():
    wl = W.workload("qwen")
    P.log("case qwen full size: 36 + 28 layers, V 151936, 128 rows, capacity 2303 positions; "
          "prompt 0's 8 rows, 64 steps")
    p = P.run(wl, steps=64, logits_at=(1, 32, 64), seq_subset=list(range(wl.group)))
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
