"""Float64 reference decoder: the policy whose rollouts the library generates.

Architecture (a reading of the Llama/Qwen-style decoder the workloads name):
pre-norm blocks x += Attn(RMSNorm(x)); x += MLP(RMSNorm(x)); a final RMSNorm
and an untied lm_head; no biases, no embedding scale.

* RMSNorm(x) = x / sqrt(mean(x^2) + eps) * g.
* RoPE, rotate-half pairing: dims (i, i + hd/2) for i < hd/2 are rotated by
  angle pos * theta^(-2i/hd).  Prompt tokens sit at positions 0..Lp-1, the
  t-th generated token (t counted from 0) at position Lp + t.
* Causal attention softmax(q k^T / sqrt(hd)) v; query head h reads key/value
  head floor(h * n_kv / n_q) (grouped-query attention).
* MLP = W_down (silu(W_gate x) * (W_up x)), silu(a) = a / (1 + e^-a).

Weight matrices are stored [out, in] (a linear map is x @ W^T).  All arithmetic
is float64; the bf16 weights of bf16 models are exactly representable.

Storage precision.  A model's matrices and its key/value cache are stored in
the model's dtype (fp32 or bf16); every other value -- activations entering a
matrix product, residual stream, norms, RoPE, queries, attention scores,
softmax and every accumulation -- is exact here (float64).  So a bf16 model
computes with bf16 weights (exactly representable) and reads back keys and
values rounded to nearest-even in the storage type (keys after RoPE).
``kv_storage="exact"`` keeps the cache in float64 (the pure definition).
"""
from __future__ import annotations

from typing import List

import numpy as np


class OracleModel:
    def __init__(self, shape, weights, cache_f64: bool = True, kv_storage: str = "model"):
        if kv_storage == "model":
            kv_storage = shape.dtype
        if kv_storage not in ("exact", "f32", "bf16"):
            raise ValueError(kv_storage)
        self.s = shape
        self.kv_storage = kv_storage
        cv = (lambda a: np.asarray(a, np.float64)) if cache_f64 else (lambda a: a)
        self.embed = cv(weights.embed)
        self.final_norm = np.asarray(weights.final_norm, np.float64)
        self.lm_head = cv(weights.lm_head)
        self.layers = [{k: (np.asarray(v, np.float64) if k.endswith("norm") else cv(v))
                        for k, v in lw.items()} for lw in weights.layers]
        hd = shape.head_dim
        i = np.arange(hd // 2, dtype=np.float64)
        self.inv_freq = float(shape.rope_theta) ** (-(2.0 * i) / hd)

    # ---- building blocks ------------------------------------------------
    def rmsnorm(self, x: np.ndarray, g: np.ndarray) -> np.ndarray:
        ms = np.mean(x * x, axis=-1, keepdims=True)
        return x / np.sqrt(ms + self.s.rms_eps) * g

    @staticmethod
    def round_bf16(x: np.ndarray) -> np.ndarray:
        """Round to the nearest bfloat16 value (8 significant bits), ties to
        even; finite normal inputs."""
        m, e = np.frexp(np.asarray(x, np.float64))          # x = m * 2**e, 0.5 <= |m| < 1
        return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)

    @staticmethod
    def linear(x: np.ndarray, w: np.ndarray) -> np.ndarray:
        return np.asarray(x, np.float64) @ np.asarray(w, np.float64).T

    def kv_store(self, a: np.ndarray) -> np.ndarray:
        """The value the cache holds for a freshly computed key or value."""
        if self.kv_storage == "bf16":
            return self.round_bf16(a)
        if self.kv_storage == "f32":
            return np.asarray(a, np.float32).astype(np.float64)
        return a

    def rope(self, x: np.ndarray, pos: np.ndarray) -> np.ndarray:
        """x: [T, H, hd]; pos: [T] integer positions."""
        half = self.s.head_dim // 2
        ang = np.asarray(pos, np.float64)[:, None] * self.inv_freq[None, :]   # [T, half]
        c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
        x1, x2 = x[..., :half], x[..., half:]
        return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)

    def attention(self, q, k, v, q_pos, k_pos) -> np.ndarray:
        """q: [Tq, nq, hd]; k, v: [Tk, nkv, hd]; causal on positions."""
        s = self.s
        rep = s.n_q_heads // s.n_kv_heads
        out = np.empty_like(q)
        mask = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]          # [Tq, Tk]
        scale = 1.0 / np.sqrt(float(s.head_dim))
        for h in range(s.n_q_heads):
            kv = h // rep
            sc = (q[:, h, :] @ k[:, kv, :].T) * scale
            sc = np.where(mask, sc, -np.inf)
            sc = sc - sc.max(axis=1, keepdims=True)
            p = np.exp(sc)
            p /= p.sum(axis=1, keepdims=True)
            out[:, h, :] = p @ v[:, kv, :]
        return out

    @staticmethod
    def silu(a: np.ndarray) -> np.ndarray:
        return a / (1.0 + np.exp(-a))

    # ---- caches ---------------------------------------------------------
    def new_cache(self) -> List[dict]:
        s = self.s
        return [{"k": np.zeros((0, s.n_kv_heads, s.head_dim)), "v": np.zeros((0, s.n_kv_heads, s.head_dim)),
                 "pos": np.zeros(0, np.int64)} for _ in range(s.n_layers)]

    @staticmethod
    def copy_cache(cache: List[dict]) -> List[dict]:
        return [{k: v.copy() for k, v in c.items()} for c in cache]

    # ---- forward --------------------------------------------------------
    def forward(self, tokens, positions, cache: List[dict]) -> np.ndarray:
        """Run tokens [T] at positions [T] of ONE sequence, appending their keys
        and values to ``cache``; returns logits [T, V] (float64)."""
        s = self.s
        tokens = np.asarray(tokens, np.int64)
        positions = np.asarray(positions, np.int64)
        T = len(tokens)
        x = np.asarray(self.embed[tokens], np.float64)
        for lw, c in zip(self.layers, cache):
            h = self.rmsnorm(x, lw["attn_norm"])
            q = self.linear(h, lw["wq"]).reshape(T, s.n_q_heads, s.head_dim)
            k = self.linear(h, lw["wk"]).reshape(T, s.n_kv_heads, s.head_dim)
            v = self.linear(h, lw["wv"]).reshape(T, s.n_kv_heads, s.head_dim)
            q, k = self.rope(q, positions), self.kv_store(self.rope(k, positions))
            v = self.kv_store(v)
            c["k"] = np.concatenate([c["k"], k]); c["v"] = np.concatenate([c["v"], v])
            c["pos"] = np.concatenate([c["pos"], positions])
            o = self.attention(q, c["k"], c["v"], positions, c["pos"])
            x = x + self.linear(o.reshape(T, s.q_dim), lw["wo"])
            h2 = self.rmsnorm(x, lw["ffn_norm"])
            x = x + self.linear(self.silu(self.linear(h2, lw["w_gate"])) * self.linear(h2, lw["w_up"]), lw["w_down"])
        return self.linear(self.rmsnorm(x, self.final_norm), self.lm_head)

    def decode_batch(self, tokens, positions, caches: List[List[dict]]) -> np.ndarray:
        """One token for each of B independent sequences (row b uses caches[b]).
        Row-wise identical to ``forward`` with T = 1; the projections of the B
        rows are done as one matrix product.  Returns logits [B, V]."""
        s = self.s
        tokens = np.asarray(tokens, np.int64)
        positions = np.asarray(positions, np.int64)
        B = len(tokens)
        x = np.asarray(self.embed[tokens], np.float64)
        for li, lw in enumerate(self.layers):
            h = self.rmsnorm(x, lw["attn_norm"])
            q = self.rope(self.linear(h, lw["wq"]).reshape(B, s.n_q_heads, s.head_dim), positions)
            k = self.kv_store(self.rope(self.linear(h, lw["wk"]).reshape(B, s.n_kv_heads, s.head_dim), positions))
            v = self.kv_store(self.linear(h, lw["wv"]).reshape(B, s.n_kv_heads, s.head_dim))
            o = np.empty_like(q)
            for b in range(B):
                c = caches[b][li]
                c["k"] = np.concatenate([c["k"], k[b:b + 1]]); c["v"] = np.concatenate([c["v"], v[b:b + 1]])
                c["pos"] = np.concatenate([c["pos"], positions[b:b + 1]])
                o[b] = self.attention(q[b:b + 1], c["k"], c["v"], positions[b:b + 1], c["pos"])[0]
            x = x + self.linear(o.reshape(B, s.q_dim), lw["wo"])
            h2 = self.rmsnorm(x, lw["ffn_norm"])
            x = x + self.linear(self.silu(self.linear(h2, lw["w_gate"])) * self.linear(h2, lw["w_up"]), lw["w_down"])
        return self.linear(self.rmsnorm(x, self.final_norm), self.lm_head)
