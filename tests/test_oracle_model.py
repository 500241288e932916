"""Pins for the oracle decoder (CPU only).

* A second implementation assembled from torch library routines (F.linear,
  F.rms_norm, F.scaled_dot_product_attention with grouped-query heads, F.silu)
  and complex-number rotation for RoPE must give the same logits.
* RoPE closed forms: identity at position 0; a unit vector on dim i is turned by
  angle pos*theta^(-2i/hd) into dims (i, i + hd/2); norms are kept; dot
  products depend only on the position difference.
* KV-cached decode equals a full causal recompute; a one-token context returns
  V exactly; batched decode equals single-sequence decode.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from workload import get_config, make_weights, ModelShape
from oracle.model import OracleModel

TINY = get_config("tiny").shape
GQA = ModelShape(2, 64, 6, 2, 16, 96, 97, 1e4, dtype="f32")     # 3 q heads per kv head


def _model(shape, seed=0):
    return OracleModel(shape, make_weights(shape, seed), kv_storage="exact")


def torch_forward(shape, w, tokens):
    """Independent decoder forward from torch functional ops (float64)."""
    f64 = lambda a: torch.tensor(np.asarray(a, np.float64))
    T = len(tokens)
    hd, half = shape.head_dim, shape.head_dim // 2
    pos = torch.arange(T, dtype=torch.float64)
    inv = torch.tensor([shape.rope_theta ** (-(2.0 * i) / hd) for i in range(half)], dtype=torch.float64)
    rot = torch.polar(torch.ones(T, half, dtype=torch.float64), pos[:, None] * inv[None, :])   # e^{i*angle}

    def rope(x):  # x [T, H, hd]: pair (i, i+half) as the complex number x_i + j x_{i+half}
        c = torch.complex(x[..., :half], x[..., half:]) * rot[:, None, :]
        return torch.cat([c.real, c.imag], dim=-1)

    x = f64(w.embed)[torch.tensor(tokens)]
    for lw in w.layers:
        h = F.rms_norm(x, (shape.d_model,), f64(lw["attn_norm"]), eps=shape.rms_eps)
        q = rope(F.linear(h, f64(lw["wq"])).view(T, shape.n_q_heads, hd))
        k = rope(F.linear(h, f64(lw["wk"])).view(T, shape.n_kv_heads, hd))
        v = F.linear(h, f64(lw["wv"])).view(T, shape.n_kv_heads, hd)
        o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                           is_causal=True, enable_gqa=True)
        x = x + F.linear(o.transpose(0, 1).reshape(T, -1), f64(lw["wo"]))
        h2 = F.rms_norm(x, (shape.d_model,), f64(lw["ffn_norm"]), eps=shape.rms_eps)
        x = x + F.linear(F.silu(F.linear(h2, f64(lw["w_gate"]))) * F.linear(h2, f64(lw["w_up"])), f64(lw["w_down"]))
    x = F.rms_norm(x, (shape.d_model,), f64(w.final_norm), eps=shape.rms_eps)
    return F.linear(x, f64(w.lm_head)).numpy()


@pytest.mark.parametrize("shape", [TINY, GQA], ids=["tiny", "gqa"])
def test_forward_matches_torch_functional(shape):
    w = make_weights(shape, 1)
    m = OracleModel(shape, w, kv_storage="exact")
    toks = np.random.default_rng(2).integers(0, shape.vocab - 1, size=21)
    ours = m.forward(toks, np.arange(len(toks)), m.new_cache())
    ref = torch_forward(shape, w, toks)
    np.testing.assert_allclose(ours, ref, rtol=0, atol=1e-12)


def test_rope_closed_forms():
    m = _model(GQA)
    hd, half = GQA.head_dim, GQA.head_dim // 2
    # identity at position 0
    x = np.random.default_rng(0).normal(size=(1, 3, hd))
    np.testing.assert_array_equal(m.rope(x, np.array([0])), x)
    # unit vector on dim i, position p: (cos a) e_i + (sin a) e_{i+half}, a = p theta^(-2i/hd)
    for i in [0, 1, half - 1]:
        for p in [1, 7, 1000]:
            e = np.zeros((1, 1, hd)); e[0, 0, i] = 1.0
            a = p * GQA.rope_theta ** (-2.0 * i / hd)
            r = m.rope(e, np.array([p]))[0, 0]
            exp = np.zeros(hd); exp[i] = math.cos(a); exp[i + half] = math.sin(a)
            np.testing.assert_allclose(r, exp, atol=1e-12)
    # norm preserved, dot product depends on the offset only
    q = np.random.default_rng(1).normal(size=(1, 1, hd)); k = np.random.default_rng(2).normal(size=(1, 1, hd))
    rq = lambda p: m.rope(q, np.array([p]))[0, 0]
    rk = lambda p: m.rope(k, np.array([p]))[0, 0]
    assert abs(np.linalg.norm(rq(123)) - np.linalg.norm(q)) < 1e-12
    assert abs(rq(10) @ rk(3) - rq(107) @ rk(100)) < 1e-10


def test_one_token_attention_returns_v():
    m = _model(GQA)
    rng = np.random.default_rng(3)
    q = rng.normal(size=(1, 6, 16)); k = rng.normal(size=(1, 2, 16)); v = rng.normal(size=(1, 2, 16))
    o = m.attention(q, k, v, np.array([5]), np.array([5]))
    for h in range(6):
        np.testing.assert_array_equal(o[0, h], v[0, h // 3])


@pytest.mark.parametrize("shape", [TINY, GQA], ids=["tiny", "gqa"])
def test_kv_cached_decode_equals_full_recompute(shape):
    m = _model(shape, 4)
    toks = np.random.default_rng(5).integers(0, shape.vocab - 1, size=19)
    full = m.forward(toks, np.arange(19), m.new_cache())
    cache = m.new_cache()
    pre = m.forward(toks[:11], np.arange(11), cache)
    np.testing.assert_allclose(pre, full[:11], rtol=0, atol=1e-12)
    for i in range(11, 19):
        z = m.forward(toks[i:i + 1], np.array([i]), cache)[0]
        np.testing.assert_allclose(z, full[i], rtol=0, atol=1e-11)


def test_decode_batch_equals_single():
    shape = GQA
    m = _model(shape, 6)
    rng = np.random.default_rng(7)
    prompts = [rng.integers(0, shape.vocab - 1, size=n) for n in (5, 9, 3)]
    caches_a, caches_b = [], []
    for p in prompts:
        c = m.new_cache(); m.forward(p, np.arange(len(p)), c)
        caches_a.append(c); caches_b.append(m.copy_cache(c))
    toks = np.array([1, 2, 3]); pos = np.array([5, 9, 3])
    zb = m.decode_batch(toks, pos, caches_a)
    for i in range(3):
        zi = m.forward(toks[i:i + 1], pos[i:i + 1], caches_b[i])[0]
        np.testing.assert_allclose(zb[i], zi, rtol=0, atol=1e-12)


def test_round_bf16_matches_torch_and_ties_to_even():
    x = np.random.default_rng(0).normal(size=100000).astype(np.float32).astype(np.float64)
    ours = OracleModel.round_bf16(x)
    ref = torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)
    # halfway cases go to the even neighbour; anything above half rounds up
    np.testing.assert_array_equal(OracleModel.round_bf16(np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8),
                                                                     1 + 2 ** -8 + 2 ** -30])),
                                  [1.0, 1 + 2 ** -6, -1.0, 1 + 2 ** -7])


def test_kv_storage_modes():
    bshape = ModelShape(2, 64, 4, 2, 16, 96, 97, 1e4, dtype="bf16")
    w = make_weights(bshape, 2)
    toks = np.random.default_rng(3).integers(0, 96, size=12)
    m = OracleModel(bshape, w)                       # bf16 cache
    c = m.new_cache()
    full = m.forward(toks, np.arange(12), c)
    for layer in c:                                  # every cached value is a bf16 number
        np.testing.assert_array_equal(layer["k"], OracleModel.round_bf16(layer["k"]))
        np.testing.assert_array_equal(layer["v"], OracleModel.round_bf16(layer["v"]))
    # KV-cached decode still equals full recompute with the same storage rule
    c2 = m.new_cache()
    m.forward(toks[:7], np.arange(7), c2)
    for i in range(7, 12):
        np.testing.assert_allclose(m.forward(toks[i:i + 1], np.array([i]), c2)[0], full[i], rtol=0, atol=1e-11)
    ex = OracleModel(bshape, w, kv_storage="exact")
    d = np.abs(ex.forward(toks, np.arange(12), ex.new_cache()) - full).max()
    assert 0 < d < 5e-2                              # storage rounding moves logits a little
