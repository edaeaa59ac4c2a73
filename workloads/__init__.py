"""Seeded synthetic workloads for the tandem co-generation rollout.

This module is shared by the CPU oracle and by the GPU path, and it holds none
of the method's arithmetic: it only describes model shapes, rollout settings
and produces seeded random weights, prompts and boundary bitmaps.

The paper trains Qwen3-4B-Instruct on DeepScaleR prompts (Section 4.1 and the
reproducibility appendix).  Neither the trained weights nor the dataset are
available here, so every workload below is synthetic: matrices are drawn from
N(0, 0.02), norm gains are 1 (optionally jittered for tests), prompts are
uniform-random token ids.  Bf16 workloads round every weight to bf16 once
(round-to-nearest-even), and the SAME rounded values feed both the oracle and
the GPU.

Shapes are the five workloads of the hot-path scope:
  tiny    2-layer d=128 senior + 1-layer d=64 junior, fp32, V=512
  small   8-layer d=1024 senior + 4-layer d=512 junior, bf16, V=32000
  qwen    Qwen3-4B-shaped senior + Qwen3-0.6B-shaped junior, bf16, V=151936
  longcot small shapes, ragged prompts, EOS, 32-token ownership chunks
  wide    small shapes, 1024 concurrent sequences
plus the paper's own schedules on these shapes: its training schedule
(paper, qwen-paper, self-paired) and its evaluation schedules at
reasoning-step boundaries (qwen-eval-alternate, qwen-eval-stepcoin).
"""
from __future__ import annotations

import copy
import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional

import numpy as np

# --------------------------------------------------------------------------
# shapes and settings
# --------------------------------------------------------------------------

REDRAW, SWITCH, ALTERNATE = 0, 1, 2          # handoff rule variants
JUNIOR, SENIOR, DRAW = 0, 1, 2               # first-owner choices


@dataclasses.dataclass
class ModelShape:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rope_theta: float = 1.0e6
    rms_eps: float = 1.0e-6
    qk_norm: bool = False
    dtype: str = "bf16"            # "bf16" or "f32"

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim


@dataclasses.dataclass
class SwitchSettings:
    mode: int = SWITCH
    p: float = 0.1
    cap_k: int = -1                 # < 0: no span cap
    boundary: str = "all"           # "all", "none" or "random:<density>"
    first_owner: int = SENIOR


@dataclasses.dataclass
class SampleSettings:
    temperature: float = 1.0
    eos_id: int = -1                # < 0: no end-of-sequence token
    eos_bias_senior: float = 0.0
    eos_bias_junior: float = 0.0
    max_new: int = 32


@dataclasses.dataclass
class Workload:
    name: str
    senior: ModelShape
    junior: ModelShape
    n_prompts: int
    group: int                      # G rollouts per prompt
    prompt_len: int                 # fixed length, or the max of a ragged range
    prompt_len_min: Optional[int]   # not None: lengths uniform in [min, prompt_len]
    switch: SwitchSettings
    sample: SampleSettings
    seed_base: int                  # weights 1000+k / 2000+k, prompts 3000+k, Philox 4000+k
    gain_jitter: float = 0.0        # 0: all norm gains are exactly 1

    @property
    def n_seqs(self) -> int:
        return self.n_prompts * self.group

    @property
    def philox_seed(self) -> int:
        return 4000 + self.seed_base

    def max_ctx(self) -> int:
        return self.prompt_len + self.sample.max_new

    def replace(self, **kw) -> "Workload":
        w = copy.deepcopy(self)
        for k, v in kw.items():
            setattr(w, k, v)
        return w


def _small_pair(vocab=32000):
    sen = ModelShape(8, 1024, 16, 4, 64, 4096, vocab)
    jun = ModelShape(4, 512, 8, 2, 64, 2048, vocab)
    return sen, jun


def workload(name: str) -> Workload:
    """The synthetic workloads by name (model shapes, batch, schedule)."""
    if name == "tiny":
        sen = ModelShape(2, 128, 4, 2, 32, 512, 512, dtype="f32")
        jun = ModelShape(1, 64, 2, 1, 32, 256, 512, dtype="f32")
        return Workload("tiny", sen, jun, 1, 4, 16, None,
                        SwitchSettings(SWITCH, 0.2, -1, "all", SENIOR),
                        SampleSettings(1.0, -1, 0.0, 0.0, 32), 1)
    if name == "small":
        sen, jun = _small_pair()
        return Workload("small", sen, jun, 8, 8, 128, None,
                        SwitchSettings(SWITCH, 0.1, -1, "all", SENIOR),
                        SampleSettings(1.0, -1, 0.0, 0.0, 512), 2)
    if name == "qwen":
        sen = ModelShape(36, 2560, 32, 8, 128, 9728, 151936, qk_norm=True)
        jun = ModelShape(28, 1024, 16, 8, 128, 3072, 151936, qk_norm=True)
        return Workload("qwen", sen, jun, 16, 8, 256, None,
                        SwitchSettings(SWITCH, 0.1, -1, "all", SENIOR),
                        SampleSettings(1.0, -1, 0.0, 0.0, 2048), 3)
    if name == "longcot":
        # EOS biases: per-model logit bias giving a mean EOS probability of
        # 1/4000 per step (geometric stop lengths of mean 4000), from
        # oracle/calibrate_eos.py (senior 2.2608, junior 2.0414)
        sen, jun = _small_pair()
        return Workload("longcot", sen, jun, 32, 8, 512, 64,
                        SwitchSettings(SWITCH, 0.3, 31, "none", SENIOR),
                        SampleSettings(1.0, 31999, 2.2608, 2.0414, 8192), 4)
    if name == "wide":
        sen, jun = _small_pair()
        return Workload("wide", sen, jun, 64, 16, 256, None,
                        SwitchSettings(SWITCH, 0.5, -1, "all", SENIOR),
                        SampleSettings(1.0, -1, 0.0, 0.0, 4096), 5)
    if name == "paper":
        # The paper's own training schedule: word-level REDRAW, p=0.5, K=32,
        # drawn first owner, T=0.6, on a 35%-dense synthetic boundary set.
        sen, jun = _small_pair()
        return Workload("paper", sen, jun, 4, 8, 64, None,
                        SwitchSettings(REDRAW, 0.5, 32, "random:0.351", DRAW),
                        SampleSettings(0.6, -1, 0.0, 0.0, 128), 6)
    if name == "qwen-paper":
        # The Qwen-shaped batch of "qwen" under the paper's training schedule.
        w = workload("qwen")
        return w.replace(name="qwen-paper", switch=SwitchSettings(REDRAW, 0.5, 32, "random:0.351", DRAW),
                         sample=SampleSettings(0.6, -1, 0.0, 0.0, 2048), seed_base=7)
    if name == "self-paired":
        # Two Qwen3-4B-shaped models (the paper's self-paired training pair),
        # 16 prompts x G=8, 3000 new tokens, the paper's schedule.
        w = workload("qwen-paper")
        return w.replace(name="self-paired", junior=copy.deepcopy(w.senior),
                         sample=SampleSettings(0.6, -1, 0.0, 0.0, 3000), seed_base=8)
    if name in ("qwen-eval-alternate", "qwen-eval-stepcoin"):
        # The paper's evaluation schedules at inference (T = 0.6): the owner
        # flips at every reasoning-step boundary (deterministic round-robin,
        # senior first), or a fair coin redraws it there (drawn first owner);
        # no span cap.  The step boundary is a sparse synthetic token set of
        # density 1/48 (reasoning steps of about 48 tokens on average).
        w = workload("qwen")
        if name.endswith("alternate"):
            sw = SwitchSettings(ALTERNATE, 0.5, -1, "random:0.0208", SENIOR)
        else:
            sw = SwitchSettings(REDRAW, 0.5, -1, "random:0.0208", DRAW)
        return w.replace(name=name, switch=sw, sample=SampleSettings(0.6, -1, 0.0, 0.0, 2048),
                         seed_base=9 if name.endswith("alternate") else 10)
    raise KeyError(name)


NAMES = ("tiny", "small", "qwen", "longcot", "wide", "paper", "qwen-paper", "self-paired", "qwen-eval-alternate",
         "qwen-eval-stepcoin")


def scaled(shape: ModelShape, **kw) -> ModelShape:
    s = copy.deepcopy(shape)
    for k, v in kw.items():
        setattr(s, k, v)
    return s


# --------------------------------------------------------------------------
# seeded generators
# --------------------------------------------------------------------------

def _threads() -> int:
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:  # pragma: no cover
        return max(1, min(16, os.cpu_count() or 1))


def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


LAYER_KEYS = ("attn_norm", "w_qkv", "q_norm", "k_norm", "w_o", "ffn_norm", "w_gate_up", "w_down")


def _tensor_list(shape: ModelShape):
    """(name, shape, kind) for every tensor of a model; kind is 'mat' or 'gain'."""
    d, hd = shape.d_model, shape.head_dim
    out = [("embed", (shape.vocab, d), "mat")]
    for i in range(shape.n_layers):
        out.append((f"layers.{i}.attn_norm", (d,), "gain"))
        out.append((f"layers.{i}.w_qkv", (shape.qkv_dim, d), "mat"))
        if shape.qk_norm:
            out.append((f"layers.{i}.q_norm", (hd,), "gain"))
            out.append((f"layers.{i}.k_norm", (hd,), "gain"))
        out.append((f"layers.{i}.w_o", (d, shape.n_q_heads * hd), "mat"))
        out.append((f"layers.{i}.ffn_norm", (d,), "gain"))
        out.append((f"layers.{i}.w_gate_up", (2 * shape.ffn_dim, d), "mat"))
        out.append((f"layers.{i}.w_down", (d, shape.ffn_dim), "mat"))
    out.append(("final_norm", (d,), "gain"))
    out.append(("lm_head", (shape.vocab, d), "mat"))
    return out


def make_weights(shape: ModelShape, seed: int, gain_jitter: float = 0.0,
                 std: float = 0.02) -> Dict[str, np.ndarray]:
    """Seeded weights for one model.

    Matrices are row-major [out][in].  For bf16 models the values are returned
    as uint16 bf16 bit patterns; for f32 models as float32.  Norm gains are
    always float32 (1.0, or 1 + gain_jitter * N(0,1) for tests).
    Each tensor draws from its own stream, SeedSequence(seed, spawn_key=(i,)),
    so generation can run on several threads and stays reproducible.
    """
    items = _tensor_list(shape)

    def gen(idx_item):
        idx, (name, shp, kind) = idx_item
        rng = np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(idx,)))
        if kind == "gain":
            g = np.ones(shp, dtype=np.float32)
            if gain_jitter:
                g += np.float32(gain_jitter) * rng.standard_normal(shp, dtype=np.float32)
            return name, g
        w = rng.standard_normal(shp, dtype=np.float32)
        w *= np.float32(std)
        if shape.dtype == "bf16":
            return name, round_to_bf16_bits(w)
        return name, w

    with ThreadPoolExecutor(_threads()) as ex:
        return dict(ex.map(gen, list(enumerate(items))))


def weights_as_float(shape: ModelShape, w: Dict[str, np.ndarray], dtype=np.float64) -> Dict[str, np.ndarray]:
    """Convert generated weights to a float dtype (exact for bf16 inputs),
    one tensor per thread (NumPy's conversions release the GIL)."""
    def conv(kv):
        k, v = kv
        if v.dtype == np.uint16:
            return k, bf16_bits_to_f32(v).astype(dtype)
        return k, v.astype(dtype)

    with ThreadPoolExecutor(_threads()) as ex:
        return dict(ex.map(conv, list(w.items())))


def make_prompts(wl: Workload) -> List[np.ndarray]:
    """Uniform-random prompt token ids (seed 3000+k); EOS never appears in a prompt."""
    rng = np.random.default_rng(3000 + wl.seed_base)
    V = wl.senior.vocab
    eos = wl.sample.eos_id
    prompts = []
    for _ in range(wl.n_prompts):
        if wl.prompt_len_min is None:
            n = wl.prompt_len
        else:
            n = int(rng.integers(wl.prompt_len_min, wl.prompt_len + 1))
        hi = V - 1 if 0 <= eos == V - 1 else V
        p = rng.integers(0, hi, size=n).astype(np.int32)
        if eos >= 0 and eos != V - 1:
            p[p == eos] = (eos + 1) % V
        prompts.append(p)
    return prompts


def make_boundary(wl: Workload) -> Optional[np.ndarray]:
    """Boundary set as a bool[V] array, or None when every token is a boundary."""
    spec = wl.switch.boundary
    V = wl.senior.vocab
    if spec == "all":
        return None
    if spec == "none":
        return np.zeros(V, dtype=bool)
    if spec.startswith("random:"):
        dens = float(spec.split(":", 1)[1])
        rng = np.random.default_rng(5000 + wl.seed_base)
        return rng.random(V) < dens
    raise ValueError(spec)


def boundary_bits(bnd: Optional[np.ndarray]) -> Optional[np.ndarray]:
    """Pack a bool[V] boundary set into uint32 words, bit (v & 31) of word v >> 5."""
    if bnd is None:
        return None
    V = bnd.shape[0]
    nw = (V + 31) // 32
    padded = np.zeros(nw * 32, dtype=np.uint64)
    padded[:V] = bnd.astype(np.uint64)
    shifts = np.arange(32, dtype=np.uint64)
    words = (padded.reshape(nw, 32) << shifts).sum(axis=1)
    return words.astype(np.uint32)


def make_all(wl: Workload):
    """Weights for both models, prompts and the boundary set of a workload."""
    ws = make_weights(wl.senior, 1000 + wl.seed_base, wl.gain_jitter)
    wj = make_weights(wl.junior, 2000 + wl.seed_base, wl.gain_jitter)
    return ws, wj, make_prompts(wl), make_boundary(wl)


def make_grpo_batch(n_groups: int, G: int, T: int, seed: int, noise: float = 0.15,
                    senior_share: float = 0.5):
    """Seeded synthetic inputs of the senior-only GRPO loss over n_groups
    prompts x G rollouts with arenas of row stride T (the paper's batch is 16
    prompts x G = 8 with responses of at most 3000 tokens).  The verifier and
    the dataset are not available, so rewards are binary draws whose success
    rate is itself drawn per group (uniform), which yields solved, unsolved and
    mixed groups alike; group 0 is forced all-correct and group 1 (when there
    is one) all-wrong.  Lengths are uniform in [0, T] with the first rollout at
    0 and the second at T; authorship is Bernoulli(senior_share) per position;
    the rollout-time log-probs are -Exponential(1); the current policy's
    log-probs add N(0, noise) to them, so the ratios fall on both sides of
    the clip band.  Returns (rewards f32 [S], owner u8 [S][T], length i32 [S],
    logp_old f32 [S][T], logp_new f32 [S][T]), S = n_groups * G."""
    rng = np.random.default_rng(seed)
    S = n_groups * G
    rate = rng.random(n_groups)
    rate[0] = 1.0
    if n_groups > 1:
        rate[1] = 0.0
    rewards = (rng.random(S) < np.repeat(rate, G)).astype(np.float32)
    length = rng.integers(0, T + 1, size=S).astype(np.int32)
    length[0] = 0
    if S > 1:
        length[1] = T
    owner = (rng.random((S, T)) < senior_share).astype(np.uint8)
    logp_old = (-rng.exponential(1.0, size=(S, T))).astype(np.float32)
    logp_new = (logp_old + rng.normal(0.0, noise, size=(S, T))).astype(np.float32)
    return rewards, owner, length, logp_old, logp_new
