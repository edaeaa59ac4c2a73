"""CPU oracle of the tandem co-generation rollout — TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously-correct NumPy (float64) implementation of what the GPU
hot path computes.  Only the test suite, the smoke check and the CPU-baseline
leg of the benchmark may import it; the product path never does.  It shares no
code with the HIP library: the only common module is ``workloads`` (seeded
input generators, no arithmetic of the method).

Paper passages followed (Tandem RL with Verifiable Rewards):
  * Section 3.3 (tandem rollout): both models read x . y_<t, the active model
    samples y_t, y_t is appended to both contexts; the owner is redrawn at
    word boundaries with probability p of choosing the senior.
  * Algorithm 1 (rollout half): first-owner draw, dual forward, owner's
    sample, authorship mask, EOS break, boundary-or-cap handoff block.
  * Section 3.4, the L_TRL equation: senior log-probabilities of the emitted
    tokens, used only at senior-owned positions by the loss.
  * Reproducibility appendix (dual-decoder backend; word-level handoff
    details): shared history, lockstep caches, span cap K, seeded draws.

Parity pins: see tests/test_oracle_*.py.  Functions without an independent
pin are marked "parity unpinned" in their docstrings.

Precision: the model forward runs in float64 on weights that are exactly the
bf16 (or fp32) values the GPU receives.  The sampling decision (Gumbel-max
argmax) is taken in float32 on both sides, the GPU kernel's precision.
"""
from .philox import philox4x32, philox_generic, philox_words, coin_threshold
from .model import OracleModel, KVCache
from .sampler import gumbel_noise, gumbel_argmax, senior_logprob, scores, handoff
from .rollout import rollout, RolloutResult

__all__ = [
    "philox4x32", "philox_generic", "philox_words", "coin_threshold",
    "OracleModel", "KVCache",
    "gumbel_noise", "gumbel_argmax", "senior_logprob", "scores", "handoff",
    "rollout", "RolloutResult",
]
