"""Oracle decoder forward (float64), with per-sequence KV caches.

The paper's models are Qwen3 causal LMs (Section 4.1); the synthetic stand-ins
keep their block structure: pre-norm decoder layers with RMSNorm, grouped-query
attention with rotary position embedding (NeoX half-split pairing), optional
per-head RMSNorm of q and k (Qwen3), and a SwiGLU feed-forward, followed by a
final RMSNorm and an untied LM head.  Each model keeps its own cache and both
consume every token of the shared history x . y_<t (Section 3.3; the
dual-decoder backend of the reproducibility appendix keeps the two caches in
lockstep).  A bf16 model keeps its cache in bf16 (its storage format; the
paper does not state the rollout precision).

One function, ``forward``, serves prefill and decode: it takes a list of
tokens, each with its own cache and position.  Within a layer every token's
key and value are written before any token attends, and a token at position
p attends to cache positions 0..p.  A prompt run (one cache, positions
0..n-1) is therefore causal attention, and a decode batch (one token per
sequence) is the cached single-step forward.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np


def rmsnorm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gain over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotary embedding, NeoX half-split: pair (i, i + hd/2) rotated by pos * theta^(-2i/hd).

    x: [n, heads, hd]; pos: [n] integer positions.
    """
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-(np.arange(half, dtype=np.float64) * 2.0) / hd)
    ang = pos.astype(np.float64)[:, None] * inv[None, :]          # [n, half]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 (ties to even), returned as float64.

    Correct single rounding: first round to float32 by round-to-odd (truncate,
    then set the last bit if anything was dropped), which keeps the second
    rounding to bf16 (round to nearest even on the top 16 bits) exact.
    """
    x = np.asarray(x, dtype=np.float64)
    t = x.astype(np.float32)
    away = np.abs(t.astype(np.float64)) > np.abs(x)
    t = np.where(away, np.nextafter(t, np.float32(0)), t)        # truncation toward zero
    u = t.view(np.uint32).copy()
    inexact = t.astype(np.float64) != x
    u |= inexact.astype(np.uint32)                                # sticky bit
    u = u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    u &= np.uint32(0xFFFF0000)
    return u.view(np.float32).astype(np.float64)


class KVCache:
    """One sequence's cache for one model: K and V as [layer, kv_head, ctx, hd]."""

    def __init__(self, n_layers: int, n_kv: int, max_ctx: int, hd: int):
        self.k = np.zeros((n_layers, n_kv, max_ctx, hd), dtype=np.float64)
        self.v = np.zeros((n_layers, n_kv, max_ctx, hd), dtype=np.float64)

    def copy(self) -> "KVCache":
        c = KVCache.__new__(KVCache)
        c.k = self.k.copy()
        c.v = self.v.copy()
        return c


class OracleModel:
    def __init__(self, shape, weights: Dict[str, np.ndarray]):
        """shape: workloads.ModelShape; weights: float64 arrays keyed as in workloads.

        A bf16 model stores its weights AND its KV cache in bf16: keys and
        values are rounded to bf16 when they are appended (the storage format
        of the model, as for the weights); everything else is float64.
        """
        self.s = shape
        self.w = weights
        self.kv_round = round_bf16 if getattr(shape, "dtype", "f32") == "bf16" else (lambda a: a)

    def new_cache(self, max_ctx: int) -> KVCache:
        s = self.s
        return KVCache(s.n_layers, s.n_kv_heads, max_ctx, s.head_dim)

    def _attend(self, cache: KVCache, layer: int, q: np.ndarray, ctx: int) -> np.ndarray:
        """Softmax attention of q [nq, hd] over cache positions 0..ctx-1.

        Query head h reads kv head floor(h * n_kv / n_q) (grouped-query).
        """
        s = self.s
        grp = s.n_q_heads // s.n_kv_heads
        K = cache.k[layer, :, :ctx, :]                               # [nkv, ctx, hd]
        V = cache.v[layer, :, :ctx, :]
        qg = q.reshape(s.n_kv_heads, grp, s.head_dim)                # head h -> (h // grp, h % grp)
        sc = np.einsum("kgd,kcd->kgc", qg, K) / np.sqrt(s.head_dim)
        sc = sc - sc.max(axis=-1, keepdims=True)
        p = np.exp(sc)
        p = p / p.sum(axis=-1, keepdims=True)
        o = np.einsum("kgc,kcd->kgd", p, V)
        return o.reshape(s.n_q_heads * s.head_dim)

    def forward(self, caches: Sequence[KVCache], tokens: Sequence[int],
                positions: Sequence[int], logits: bool = True) -> np.ndarray:
        """Forward n tokens; token i is at positions[i] of caches[i].

        Appends every token's k, v to its cache and returns logits [n, V]
        (or the final normed hidden states [n, d] if logits is False).
        """
        s, w = self.s, self.w
        tok = np.asarray(tokens, dtype=np.int64)
        pos = np.asarray(positions, dtype=np.int64)
        n = tok.shape[0]
        nq, nkv, hd = s.n_q_heads, s.n_kv_heads, s.head_dim
        h = w["embed"][tok].copy()                                   # [n, d]
        for li in range(s.n_layers):
            p = f"layers.{li}."
            x = rmsnorm(h, w[p + "attn_norm"], s.rms_eps)
            qkv = x @ w[p + "w_qkv"].T
            q = qkv[:, : nq * hd].reshape(n, nq, hd)
            k = qkv[:, nq * hd:(nq + nkv) * hd].reshape(n, nkv, hd)
            v = qkv[:, (nq + nkv) * hd:].reshape(n, nkv, hd)
            if s.qk_norm:
                q = rmsnorm(q, w[p + "q_norm"], s.rms_eps)
                k = rmsnorm(k, w[p + "k_norm"], s.rms_eps)
            q = rope(q, pos, s.rope_theta)
            k = rope(k, pos, s.rope_theta)
            k = self.kv_round(k)
            v = self.kv_round(v)
            for i in range(n):
                caches[i].k[li, :, pos[i], :] = k[i]
                caches[i].v[li, :, pos[i], :] = v[i]
            att = np.stack([self._attend(caches[i], li, q[i], int(pos[i]) + 1) for i in range(n)])
            h = h + att @ w[p + "w_o"].T
            x = rmsnorm(h, w[p + "ffn_norm"], s.rms_eps)
            gu = x @ w[p + "w_gate_up"].T
            a = silu(gu[:, : s.ffn_dim]) * gu[:, s.ffn_dim:]
            h = h + a @ w[p + "w_down"].T
        hf = rmsnorm(h, w["final_norm"], s.rms_eps)
        if not logits:
            return hf
        return hf @ w["lm_head"].T

    def prefill(self, cache: KVCache, tokens: Sequence[int], start: int = 0) -> np.ndarray:
        """Causal forward of a token run at positions start.. into one cache; logits [n, V]."""
        n = len(tokens)
        return self.forward([cache] * n, tokens, range(start, start + n))
