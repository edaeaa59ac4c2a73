"""Device-memory plumbing around the C ABI (PyTorch allocates, the library computes).

TandemEngine uploads two models' weights as torch tensors, allocates the KV
arena, the scratch buffer and the output arenas with the sizes the library
asks for, and forwards prefill/step calls to libtandem on the current torch
stream.  Nothing here computes any part of the rollout.
"""
from __future__ import annotations

import ctypes as C
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import _lib as L

LAYER_KEYS = ("attn_norm", "w_qkv", "q_norm", "k_norm", "w_o", "ffn_norm", "w_gate_up", "w_down")


def _to_device(arr: np.ndarray, dev) -> torch.Tensor:
    if arr.dtype == np.uint16:          # bf16 bit patterns
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr)).to(dev)


def model_cfg(shape) -> L.ModelCfg:
    return L.ModelCfg(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                      shape.ffn_dim, shape.vocab, float(shape.rope_theta), float(shape.rms_eps),
                      1 if shape.qk_norm else 0, L.BF16 if shape.dtype == "bf16" else L.F32)


class DeviceModel:
    """One model's weights on the device plus its tandem_model descriptor."""

    def __init__(self, shape, weights: Dict[str, np.ndarray], dev):
        self.shape = shape
        self.t = {k: _to_device(v, dev) for k, v in weights.items()}
        ptrs = []
        for i in range(shape.n_layers):
            for k in LAYER_KEYS:
                t = self.t.get(f"layers.{i}.{k}")
                ptrs.append(t.data_ptr() if t is not None else 0)
        self.layer_ptrs = (C.c_void_p * len(ptrs))(*ptrs)
        self.desc = L.Model(model_cfg(shape), self.t["embed"].data_ptr(),
                            C.cast(self.layer_ptrs, C.POINTER(C.c_void_p)),
                            self.t["final_norm"].data_ptr(), self.t["lm_head"].data_ptr())


class TandemEngine:
    """junior_shape None (or models[1] None): the senior alone, through the
    same kernels (every token the senior's; switch is ignored)."""

    def __init__(self, senior_shape, senior_w, junior_shape, junior_w, switch, sample, seed: int,
                 max_seqs: int, max_ctx: int, max_prefill_tokens: int = 4096,
                 boundary_words: Optional[np.ndarray] = None, device: str = "cuda:0",
                 models: Optional[Sequence[Optional[DeviceModel]]] = None):
        if not torch.cuda.is_available():
            raise RuntimeError("TandemEngine needs a ROCm GPU (torch.cuda.is_available() is False)")
        self.dev = torch.device(device)
        torch.cuda.set_device(self.dev)
        if models is None:
            self.sen = DeviceModel(senior_shape, senior_w, self.dev)
            self.jun = DeviceModel(junior_shape, junior_w, self.dev) if junior_shape is not None else None
        else:
            self.sen, self.jun = models
        self.sample = sample
        self.max_seqs, self.max_new = max_seqs, sample.max_new
        self.V = self.sen.shape.vocab
        self.cap = L.Capacity(max_seqs, max_ctx, max_prefill_tokens)
        kvb, scb = L.tandem_workspace_size(self.sen.desc.cfg, self.jun.desc.cfg if self.jun else None, self.cap)
        self.kv_bytes, self.scratch_bytes = kvb, scb
        self.kv = torch.empty(kvb, dtype=torch.uint8, device=self.dev)
        self.scratch = torch.empty(scb, dtype=torch.uint8, device=self.dev)
        self.tokens = torch.full((max_seqs, self.max_new), -1, dtype=torch.int32, device=self.dev)
        self.owner = torch.zeros((max_seqs, self.max_new), dtype=torch.uint8, device=self.dev)
        self.logprob = torch.zeros((max_seqs, self.max_new), dtype=torch.float32, device=self.dev)
        self.length = torch.zeros(max_seqs, dtype=torch.int32, device=self.dev)
        self.bnd = None
        if boundary_words is not None:
            self.bnd = torch.from_numpy(np.ascontiguousarray(boundary_words).view(np.int32)).to(self.dev)
        self.sw = L.SwitchCfg(int(switch.mode), float(switch.p), int(switch.cap_k),
                              self.bnd.data_ptr() if self.bnd is not None else None, int(switch.first_owner))
        self.smp = L.SampleCfg(float(sample.temperature), int(sample.eos_id), float(sample.eos_bias_senior),
                               float(sample.eos_bias_junior), int(sample.max_new), int(seed))
        self.out = L.Outputs(self.tokens.data_ptr(), self.owner.data_ptr(), self.logprob.data_ptr(),
                             self.length.data_ptr())
        self.stream = torch.cuda.current_stream(self.dev)
        self.h = L.tandem_init(self.sen.desc, self.jun.desc if self.jun else None, self.sw, self.smp, self.cap,
                               self.kv.data_ptr(), kvb, self.scratch.data_ptr(), scb, self.out,
                               self.stream.cuda_stream)
        self.n_seq = 0
        self._forced = torch.full((max_seqs,), -1, dtype=torch.int32, device=self.dev)

    # ------------------------------------------------------------- calls
    def prefill(self, prompts: Sequence[np.ndarray], G: int) -> None:
        flat = np.concatenate([np.asarray(p, dtype=np.int32) for p in prompts])
        offs = np.concatenate([[0], np.cumsum([len(p) for p in prompts])]).astype(np.int64)
        self._prompt_dev = torch.from_numpy(flat).to(self.dev)
        L.tandem_prefill(self.h, self._prompt_dev.data_ptr(), offs.tolist(), len(prompts), G)
        self.n_seq = len(prompts) * G

    def step(self, want_active: bool = False):
        return L.tandem_step(self.h, want_active)

    def step_forced(self, forced, debug: bool = True, logits: bool = False, want_active: bool = False):
        """Append forced[s] (entries < 0: own sample); returns the debug tensors."""
        f = torch.as_tensor(np.asarray(forced, dtype=np.int32)).to(self.dev)
        self._forced[: len(f)].copy_(f)
        dbg = None
        res = {}
        if debug:
            res["sampled"] = torch.full((self.max_seqs,), -1, dtype=torch.int32, device=self.dev)
            res["margin"] = torch.zeros(self.max_seqs, dtype=torch.float32, device=self.dev)
            if logits:
                res["logits_senior"] = torch.zeros((self.max_seqs, self.V), dtype=torch.float32, device=self.dev)
                res["logits_junior"] = torch.zeros((self.max_seqs, self.V), dtype=torch.float32, device=self.dev)
            dbg = L.Debug(res["sampled"].data_ptr(), res["margin"].data_ptr(),
                          res["logits_senior"].data_ptr() if logits else None,
                          res["logits_junior"].data_ptr() if logits else None)
        n = L.tandem_step_forced(self.h, self._forced.data_ptr(), dbg, want_active)
        if want_active:
            res["n_active"] = n
        return res

    def timing(self, class_mask: int) -> None:
        """Time launches of the classes in class_mask (bit k = class k); 0 switches timing off."""
        L.tandem_timing_enable(self.h, class_mask)

    def timing_read(self):
        """{class name: (device ms, launches)} since the last timing() call."""
        names = {L.K_ATTENTION: "attention", L.K_GEMM: "gemm", L.K_SAMPLE: "sample", L.K_OTHER: "other"}
        return {v: L.tandem_timing_read(self.h, k) for k, v in names.items()}

    def score(self, out=None):
        """Dual-distribution scores of the step just taken: a device float32
        tensor [max_seqs][3] of (junior cross-entropy of the appended token,
        overlap, KL(senior || junior)) by sequence id; rows of sequences that
        were done before the step keep their previous contents."""
        if out is None:
            out = torch.full((self.max_seqs, 3), float("nan"), dtype=torch.float32, device=self.dev)
        L.tandem_score_step(self.h, out.data_ptr())
        return out

    def state(self):
        owner, c, t, pos, done = L.tandem_get_state(self.h, self.n_seq)
        return dict(owner=np.array(owner), c=np.array(c), t=np.array(t), pos=np.array(pos), done=np.array(done))

    def outputs(self):
        torch.cuda.synchronize(self.dev)
        n = self.n_seq
        return dict(tokens=self.tokens[:n].cpu().numpy(), owner=self.owner[:n].cpu().numpy(),
                    logprob=self.logprob[:n].cpu().numpy(), length=self.length[:n].cpu().numpy())

    def close(self) -> None:
        if getattr(self, "h", None):
            torch.cuda.synchronize(self.dev)
            L.tandem_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def grpo_loss(rewards: torch.Tensor, owner: torch.Tensor, length: torch.Tensor, logp_old: torch.Tensor,
              logp_new: Optional[torch.Tensor], G: int, clip_eps: float = 0.2, want_grad: bool = True,
              workspace: Optional[torch.Tensor] = None, noalloc: bool = False):
    """Senior-only GRPO loss pieces (tandem_grpo_loss) of S = len(rewards)
    rollouts in groups of G, on the current torch stream.  rewards float32
    [S]; owner uint8 [S][T]; length int32 [S]; logp_old / logp_new float32
    [S][T] (logp_new None: ratio 1).  Returns device tensors: advantages [S],
    loss [1], n_masked [1] and grad [S][T] (None unless want_grad).
    noalloc: call tandem_grpo_loss_noalloc (the library's own device
    workspace; the output tensors are still allocated here)."""
    S, T = owner.shape
    dev = owner.device
    for name, t, dt, shape in (("rewards", rewards, torch.float32, (S,)), ("owner", owner, torch.uint8, (S, T)),
                               ("length", length, torch.int32, (S,)), ("logp_old", logp_old, torch.float32, (S, T)),
                               ("logp_new", logp_new, torch.float32, (S, T))):
        if t is None:
            continue
        if t.dtype != dt or tuple(t.shape) != shape or t.device != dev or not t.is_contiguous():
            raise ValueError(f"grpo_loss: {name} must be a contiguous {dt} tensor of shape {shape} on {dev}")
    if S % G != 0:
        raise ValueError(f"grpo_loss: {S} rollouts do not form groups of {G}")
    cfg = L.GrpoCfg(S // G, G, T, float(clip_eps))
    adv = torch.empty(S, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    n = torch.empty(1, dtype=torch.int32, device=dev)
    grad = torch.empty((S, T), dtype=torch.float32, device=dev) if want_grad else None
    if noalloc:
        L.tandem_grpo_loss_noalloc(cfg, rewards.data_ptr(), owner.data_ptr(), length.data_ptr(), logp_old.data_ptr(),
                                   logp_new.data_ptr() if logp_new is not None else None, adv.data_ptr(),
                                   grad.data_ptr() if grad is not None else None, loss.data_ptr(), n.data_ptr(),
                                   torch.cuda.current_stream(dev).cuda_stream)
        return dict(advantages=adv, loss=loss, n_masked=n, grad=grad)
    wsb = L.tandem_grpo_workspace_size(cfg)
    if workspace is None or workspace.numel() < wsb:
        workspace = torch.empty(wsb, dtype=torch.uint8, device=dev)
    L.tandem_grpo_loss(cfg, rewards.data_ptr(), owner.data_ptr(), length.data_ptr(), logp_old.data_ptr(),
                       logp_new.data_ptr() if logp_new is not None else None, adv.data_ptr(),
                       grad.data_ptr() if grad is not None else None, loss.data_ptr(), n.data_ptr(),
                       workspace.data_ptr(), wsb, torch.cuda.current_stream(dev).cuda_stream)
    return dict(advantages=adv, loss=loss, n_masked=n, grad=grad)
