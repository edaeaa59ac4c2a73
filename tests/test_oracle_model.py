"""Pins of the oracle's decoder forward (CPU only).

Each pin reaches the forward through something other than the oracle's own
formula: library routines (torch CPU functional ops, SciPy), textbook
identities (complex rotation, norm preservation), or a structural reduction
(cached decode vs one causal pass; GQA vs duplicated-head MHA).
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy.special import expit

import workloads as W
from oracle.model import OracleModel, rmsnorm, rope, silu, KVCache, round_bf16
from oracle.rollout import build_models


def _tiny(gain_jitter=0.1, qk_norm=False, **kw):
    wl = W.workload("tiny").replace(gain_jitter=gain_jitter)
    if qk_norm:
        wl.senior.qk_norm = True
        wl.junior.qk_norm = True
    for k, v in kw.items():
        setattr(wl.senior, k, v)
    ws, wj, prompts, _ = W.make_all(wl)
    sen, jun = build_models(wl, ws, wj)
    return wl, sen, jun, prompts


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 96))
    g = 1 + 0.1 * rng.standard_normal(96)
    ref = F.rms_norm(torch.from_numpy(x), (96,), weight=torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(rmsnorm(x, g, 1e-6), ref, rtol=1e-12, atol=1e-12)


def test_silu_matches_scipy():
    x = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(silu(x), x * expit(x), rtol=1e-12, atol=1e-300)


def test_rope_is_complex_rotation():
    rng = np.random.default_rng(1)
    hd, theta = 32, 1.0e6
    x = rng.standard_normal((7, 3, hd))
    pos = np.array([0, 1, 2, 5, 100, 1000, 40000])
    out = rope(x, pos, theta)
    half = hd // 2
    z = x[..., :half] + 1j * x[..., half:]
    freq = theta ** (-np.arange(0, hd, 2) / hd)
    rot = z * np.exp(1j * pos[:, None, None] * freq[None, None, :])
    np.testing.assert_allclose(out[..., :half], rot.real, atol=1e-12)
    np.testing.assert_allclose(out[..., half:], rot.imag, atol=1e-12)
    # position 0 is the identity, and rotation preserves norms
    np.testing.assert_allclose(out[0], x[0], atol=0)
    np.testing.assert_allclose(np.linalg.norm(out, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)


def test_rope_scores_depend_on_relative_position_only():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 1, 64))
    k = rng.standard_normal((1, 1, 64))
    def score(m, n):
        return float(np.sum(rope(q, np.array([m]), 1e4) * rope(k, np.array([n]), 1e4)))
    for d in (0, 3, 17):
        np.testing.assert_allclose(score(5 + d, 5), score(300 + d, 300), rtol=1e-10)


@pytest.mark.parametrize("nq,nkv", [(4, 1), (4, 2), (8, 8), (6, 3)])
def test_attention_matches_torch_sdpa(nq, nkv):
    rng = np.random.default_rng(nq * 10 + nkv)
    hd, ctx = 32, 13
    shape = W.ModelShape(1, 64, nq, nkv, hd, 64, 16, dtype="f32")
    m = OracleModel(shape, {})
    cache = KVCache(1, nkv, 20, hd)
    cache.k[0, :, :ctx] = rng.standard_normal((nkv, ctx, hd))
    cache.v[0, :, :ctx] = rng.standard_normal((nkv, ctx, hd))
    q = rng.standard_normal((nq, hd))
    got = m._attend(cache, 0, q, ctx).reshape(nq, hd)
    ref = F.scaled_dot_product_attention(
        torch.from_numpy(q)[None, :, None, :],
        torch.from_numpy(cache.k[0, :, :ctx])[None],
        torch.from_numpy(cache.v[0, :, :ctx])[None],
        enable_gqa=True)[0, :, 0, :].numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-12)


def test_attention_special_cases():
    shape = W.ModelShape(1, 64, 2, 1, 16, 64, 16, dtype="f32")
    m = OracleModel(shape, {})
    cache = KVCache(1, 1, 8, 16)
    rng = np.random.default_rng(4)
    cache.v[0, 0, :5] = rng.standard_normal((5, 16))
    q = rng.standard_normal((2, 16))
    # a single position returns its value vector exactly
    np.testing.assert_allclose(m._attend(cache, 0, q, 1).reshape(2, 16)[1], cache.v[0, 0, 0], atol=0)
    # identical keys give the plain mean of the values
    cache.k[0, 0, :5] = rng.standard_normal(16)
    np.testing.assert_allclose(m._attend(cache, 0, q, 5).reshape(2, 16)[0],
                               cache.v[0, 0, :5].mean(axis=0), atol=1e-12)


@pytest.mark.parametrize("qk_norm", [False, True])
def test_cached_decode_equals_causal_recompute(qk_norm):
    wl, sen, jun, prompts = _tiny(qk_norm=qk_norm)
    toks = np.concatenate([prompts[0], np.arange(9) * 37 % wl.senior.vocab]).astype(np.int64)
    for model in (sen, jun):
        full = model.prefill(model.new_cache(64), toks)          # one causal pass
        cache = model.new_cache(64)
        inc = np.stack([model.forward([cache], [int(t)], [i])[0] for i, t in enumerate(toks)])
        np.testing.assert_allclose(inc, full, rtol=0, atol=1e-10)


def test_gqa_equals_mha_with_duplicated_kv_heads():
    wl, sen, _, prompts = _tiny()
    s = sen.s
    grp = s.n_q_heads // s.n_kv_heads
    mha_shape = W.scaled(s, n_kv_heads=s.n_q_heads)
    w = {k: v.copy() for k, v in sen.w.items()}
    hd, nq, nkv = s.head_dim, s.n_q_heads, s.n_kv_heads
    for li in range(s.n_layers):
        qkv = sen.w[f"layers.{li}.w_qkv"]
        q = qkv[: nq * hd]
        k = qkv[nq * hd:(nq + nkv) * hd].reshape(nkv, hd, -1)
        v = qkv[(nq + nkv) * hd:].reshape(nkv, hd, -1)
        k2 = np.repeat(k, grp, axis=0).reshape(nq * hd, -1)
        v2 = np.repeat(v, grp, axis=0).reshape(nq * hd, -1)
        w[f"layers.{li}.w_qkv"] = np.concatenate([q, k2, v2])
    mha = OracleModel(mha_shape, w)
    toks = prompts[0]
    np.testing.assert_allclose(mha.prefill(mha.new_cache(32), toks),
                               sen.prefill(sen.new_cache(32), toks), atol=1e-10)


def _torch_forward(shape, w, toks):
    """Independent composition of torch CPU library ops (float64)."""
    t = lambda a: torch.from_numpy(np.asarray(a))
    n = len(toks)
    nq, nkv, hd, d = shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.d_model
    h = t(w["embed"])[torch.as_tensor(toks)]
    half = hd // 2
    freq = torch.tensor(shape.rope_theta, dtype=torch.float64) ** (-torch.arange(0, hd, 2, dtype=torch.float64) / hd)
    rot = torch.polar(torch.ones(n, half, dtype=torch.float64), torch.arange(n, dtype=torch.float64)[:, None] * freq)
    def apply_rope(x):  # x [n, heads, hd]
        z = torch.complex(x[..., :half], x[..., half:]) * rot[:, None, :]
        return torch.cat([z.real, z.imag], dim=-1)
    for li in range(shape.n_layers):
        p = f"layers.{li}."
        x = F.rms_norm(h, (d,), weight=t(w[p + "attn_norm"]), eps=shape.rms_eps)
        qkv = F.linear(x, t(w[p + "w_qkv"]))
        q, k, v = torch.split(qkv, [nq * hd, nkv * hd, nkv * hd], dim=-1)
        q, k, v = q.view(n, nq, hd), k.view(n, nkv, hd), v.view(n, nkv, hd)
        if shape.qk_norm:
            q = F.rms_norm(q, (hd,), weight=t(w[p + "q_norm"]), eps=shape.rms_eps)
            k = F.rms_norm(k, (hd,), weight=t(w[p + "k_norm"]), eps=shape.rms_eps)
        q, k = apply_rope(q), apply_rope(k)
        o = F.scaled_dot_product_attention(q.transpose(0, 1)[None], k.transpose(0, 1)[None],
                                           v.transpose(0, 1)[None], is_causal=True, enable_gqa=True)
        h = h + F.linear(o[0].transpose(0, 1).reshape(n, nq * hd), t(w[p + "w_o"]))
        x = F.rms_norm(h, (d,), weight=t(w[p + "ffn_norm"]), eps=shape.rms_eps)
        g, u = torch.split(F.linear(x, t(w[p + "w_gate_up"])), shape.ffn_dim, dim=-1)
        h = h + F.linear(F.silu(g) * u, t(w[p + "w_down"]))
    return F.linear(F.rms_norm(h, (d,), weight=t(w["final_norm"]), eps=shape.rms_eps), t(w["lm_head"])).numpy()


@pytest.mark.parametrize("qk_norm", [False, True])
def test_forward_matches_torch_library_composition(qk_norm):
    wl, sen, jun, prompts = _tiny(qk_norm=qk_norm)
    toks = prompts[0]
    for model in (sen, jun):
        ref = _torch_forward(model.s, model.w, toks)
        got = model.prefill(model.new_cache(32), toks)
        np.testing.assert_allclose(got, ref, rtol=1e-9, atol=1e-10)


def test_zero_blocks_reduce_to_embedding_head():
    wl, sen, _, prompts = _tiny()
    w = dict(sen.w)
    for li in range(sen.s.n_layers):
        w[f"layers.{li}.w_o"] = np.zeros_like(w[f"layers.{li}.w_o"])
        w[f"layers.{li}.w_down"] = np.zeros_like(w[f"layers.{li}.w_down"])
    m = OracleModel(sen.s, w)
    toks = prompts[0][:5]
    e = w["embed"][toks]
    ref = (e / np.sqrt((e * e).mean(-1, keepdims=True) + sen.s.rms_eps) * w["final_norm"]) @ w["lm_head"].T
    np.testing.assert_allclose(m.prefill(m.new_cache(8), toks), ref, atol=1e-12)


def test_bf16_weights_are_exact_in_float64():
    wl = W.workload("small")
    shape = W.scaled(wl.senior, n_layers=1, vocab=64, d_model=128, ffn_dim=128, n_q_heads=2, n_kv_heads=1)
    w = W.make_weights(shape, 11)
    f = W.weights_as_float(shape, w)
    bits = w["w_qkv" if "w_qkv" in w else "layers.0.w_qkv"]
    back = W.round_to_bf16_bits(f["layers.0.w_qkv"].astype(np.float32))
    np.testing.assert_array_equal(back, bits)
    assert abs(f["layers.0.w_qkv"].std() - 0.02) < 0.002


def _bf16_exact(x: float) -> float:
    """Nearest bf16 by exhaustive search over the two neighbours, with exact Fractions."""
    from fractions import Fraction
    import struct
    f = Fraction(x)
    b = struct.unpack("<I", struct.pack("<f", np.float32(x)))[0] & 0xFFFF0000
    cands = set()
    for d in (-0x20000, -0x10000, 0, 0x10000, 0x20000):
        u = (b + d) & 0xFFFFFFFF
        v = struct.unpack("<f", struct.pack("<I", u))[0]
        if np.isfinite(v):
            cands.add((v, u))
    best = min(cands, key=lambda c: (abs(Fraction(c[0]) - f), (c[1] >> 16) & 1))
    return best[0]


def test_round_bf16_is_correctly_rounded():
    rng = np.random.default_rng(5)
    xs = list(rng.standard_normal(400) * 10.0 ** rng.integers(-6, 6, 400))
    # exact ties and near-ties between bf16 neighbours, which double rounding gets wrong
    base = np.float32(1.0 + 2 ** -7)
    xs += [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 1.0 + 2 ** -8 + 2 ** -40,
           1.0 + 2 ** -8 - 2 ** -40, float(base) + 2 ** -9 + 2 ** -30, 1.0 + 2 ** -8 + 2 ** -24 + 2 ** -40]
    got = round_bf16(np.array(xs))
    for x, g in zip(xs, got):
        assert g == _bf16_exact(x), x
    np.testing.assert_array_equal(round_bf16(np.array([0.0, -0.0, 1.0, -2.5])), [0.0, -0.0, 1.0, -2.5])


def test_bf16_model_stores_its_cache_in_bf16():
    wl = W.workload("small")
    shape = W.scaled(wl.senior, n_layers=1, vocab=64, d_model=128, ffn_dim=128, n_q_heads=2, n_kv_heads=1)
    f = W.weights_as_float(shape, W.make_weights(shape, 3))
    m = OracleModel(shape, f)
    c = m.new_cache(8)
    m.prefill(c, [1, 2, 3])
    np.testing.assert_array_equal(round_bf16(c.k[:, :, :3]), c.k[:, :, :3])
    np.testing.assert_array_equal(round_bf16(c.v[:, :, :3]), c.v[:, :, :3])
    assert np.any(c.k[:, :, :3] != 0)
