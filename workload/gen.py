"""Seeded generators for the synthetic rollout workloads.

Everything here is an *input*: weights ~ N(0, 0.02) (rounded to bfloat16 with
round-to-nearest-even for bf16 models; RMSNorm gains are 1), prompt ids uniform
on [0, V-1) (the last id is EOS and never appears in a prompt), per-prompt group
sizes, forced completion lengths and Bernoulli rewards.  Each stream is seeded
from ``numpy.random.SeedSequence([seed, stream_id, ...])`` so the same seed
gives the same bytes on every machine.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import Dict, List, Optional

import numpy as np

from .configs import ModelShape, Workload

# stream ids: keep stable, they are part of the workload definition
_S_WEIGHT, _S_PROMPT, _S_GROUP, _S_LEN, _S_REWARD_P, _S_REWARD = 11, 12, 13, 14, 15, 16
_S_STEP_LEN, _S_STEP_REWARD, _S_DRIFT = 17, 18, 19

LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")


def _rng(*ids: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(i) for i in ids])))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bfloat16 (nearest-even) and return the 16-bit patterns.
    Inputs must be finite."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((b >> 16) & 1) + np.uint32(0x7FFF)
    return ((b + rounding) >> 16).astype(np.uint16)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    return (h.astype(np.uint32) << 16).view(np.float32)


def bf16_round_f32(x: np.ndarray) -> np.ndarray:
    """fp32 array whose values are the bf16 nearest-even roundings of x."""
    return bf16_bits_to_f32(f32_to_bf16_bits(x))


def layer_tensor_shapes(s: ModelShape) -> Dict[str, tuple]:
    d, f = s.d_model, s.ffn_dim
    return {
        "attn_norm": (d,), "wq": (s.q_dim, d), "wk": (s.kv_dim, d), "wv": (s.kv_dim, d),
        "wo": (d, s.q_dim), "ffn_norm": (d,), "w_gate": (f, d), "w_up": (f, d), "w_down": (d, f),
    }


@dataclass
class Weights:
    """fp32 host copies of every tensor.  For bf16 models the values are already
    bf16-representable, so converting to bf16 on upload is exact."""
    shape: ModelShape
    embed: np.ndarray            # [V, d]
    final_norm: np.ndarray       # [d]   (fp32 always)
    lm_head: np.ndarray          # [V, d]
    layers: List[Dict[str, np.ndarray]]

    def nbytes(self) -> int:
        n = self.embed.nbytes + self.final_norm.nbytes + self.lm_head.nbytes
        return n + sum(a.nbytes for lw in self.layers for a in lw.values())


def _normal_tensor(seed: int, tid: int, shape: tuple, round_bf16: bool) -> np.ndarray:
    a = _rng(seed, _S_WEIGHT, tid).standard_normal(size=shape, dtype=np.float32)
    a *= np.float32(0.02)
    if round_bf16:
        a = bf16_round_f32(a).reshape(shape)
    return a


def make_weights(shape: ModelShape, seed: int, threads: int = 8) -> Weights:
    """Random-init decoder weights: matrices ~ N(0, 0.02), norm gains = 1."""
    rb = shape.dtype == "bf16"
    d, V = shape.d_model, shape.vocab
    jobs = [("embed", 900001, (V, d)), ("lm_head", 900002, (V, d))]
    shp = layer_tensor_shapes(shape)
    for li in range(shape.n_layers):
        for j, name in enumerate(LAYER_TENSORS):
            if not name.endswith("norm"):
                jobs.append((f"{li}.{name}", 1000 * li + j, shp[name]))
    with ThreadPoolExecutor(max_workers=threads) as ex:
        outs = list(ex.map(lambda jb: _normal_tensor(seed, jb[1], jb[2], rb), jobs))
    got = {jb[0]: o for jb, o in zip(jobs, outs)}
    layers = []
    for li in range(shape.n_layers):
        lw = {}
        for name in LAYER_TENSORS:
            lw[name] = np.ones(d, np.float32) if name.endswith("norm") else got[f"{li}.{name}"]
        layers.append(lw)
    return Weights(shape, got["embed"], np.ones(d, np.float32), got["lm_head"], layers)


def make_prompts(wl: Workload, seed: int) -> np.ndarray:
    """int32 [P, Lp], uniform on [0, V-1): EOS (= V-1) never occurs in a prompt."""
    V = wl.shape.vocab
    return _rng(seed, _S_PROMPT).integers(0, V - 1, size=(wl.n_prompts, wl.prompt_len), dtype=np.int64).astype(np.int32)


def make_group_sizes(wl: Workload, seed: int) -> np.ndarray:
    """int32 [P]: the fixed G, or a per-prompt draw from the admissible sizes."""
    if wl.group_size is not None:
        return np.full(wl.n_prompts, wl.group_size, np.int32)
    ch = np.asarray(wl.group_choices, np.int32)
    return ch[_rng(seed, _S_GROUP).integers(0, len(ch), size=wl.n_prompts)].astype(np.int32)


def make_forced_lengths(wl: Workload, n_seq: int, seed: int) -> np.ndarray:
    """int32 [N] completion lengths (generated tokens including the final EOS),
    in [1, max_new]."""
    rng = _rng(seed, _S_LEN)
    kind = wl.length_dist[0]
    if kind == "uniform":
        a, b = int(wl.length_dist[1]), int(wl.length_dist[2])
        L = rng.integers(a, b + 1, size=n_seq, dtype=np.int64)
    elif kind == "lognormal":
        mu, sigma = float(wl.length_dist[1]), float(wl.length_dist[2])
        z = rng.standard_normal(size=n_seq)
        L = np.floor(np.exp(mu + sigma * z) + 0.5).astype(np.int64)
    else:
        raise ValueError(kind)
    return np.clip(L, 1, wl.max_new).astype(np.int32)


def make_rewards(wl: Workload, G: np.ndarray, seed: int) -> np.ndarray:
    """fp32 [N] Bernoulli rewards, success probability drawn per prompt."""
    kind = wl.reward_dist[0]
    if kind == "const_p":
        p = np.full(len(G), float(wl.reward_dist[1]))
    else:
        lo, hi = float(wl.reward_dist[1]), float(wl.reward_dist[2])
        p = lo + (hi - lo) * _rng(seed, _S_REWARD_P).random(len(G))
    pr = np.repeat(p, G)
    return (_rng(seed, _S_REWARD).random(int(G.sum())) < pr).astype(np.float32)


@dataclass
class Inputs:
    workload: Workload
    seed: int
    prompts: np.ndarray          # int32 [P, Lp]
    G: np.ndarray                # int32 [P]
    forced_len: np.ndarray       # int32 [N]
    rewards: np.ndarray          # fp32 [N]

    @property
    def n_seq(self) -> int:
        return int(self.G.sum())


def make_inputs(wl: Workload, seed: int, n_prompts: Optional[int] = None) -> Inputs:
    """All per-run inputs except weights.  ``n_prompts`` truncates the prompt
    set (for small test slices of a large workload)."""
    prompts = make_prompts(wl, seed)
    G = make_group_sizes(wl, seed)
    if n_prompts is not None:
        prompts, G = prompts[:n_prompts], G[:n_prompts]
    N = int(G.sum())
    L = make_forced_lengths(wl, N, seed)
    r = make_rewards(wl, G, seed)
    return Inputs(wl, seed, prompts, G, L, r)


def lognormal_cap_fraction(mu: float, sigma: float, cap: int) -> float:
    """P(exp(mu + sigma Z) + 0.5 >= cap): analytic fraction of capped lengths."""
    x = (math.log(cap - 0.5) - mu) / sigma
    return 0.5 * math.erfc(x / math.sqrt(2.0))


def step_group_lengths(P: int, G: int, max_new: int, seed: int, step: int, sigma_w: float,
                       mu: float = math.log(1200.0), sigma_p: float = 0.3) -> np.ndarray:
    """Forced lengths [P*G] (prompt-major) of one training step of the
    group-size sweep: prompt p has a typical length m_p = exp(mu + sigma_p z_p)
    and its G completions floor(exp(log m_p + sigma_w z_pi) + 0.5), clipped to
    [1, max_new].  sigma_w (within-group spread) sets the straggler rate."""
    r = _rng(seed, _S_STEP_LEN, step)
    zp = r.standard_normal(P)
    zi = r.standard_normal((P, G))
    L = np.floor(np.exp(mu + sigma_p * zp[:, None] + sigma_w * zi) + 0.5)
    return np.clip(L, 1, max_new).astype(np.int32).reshape(-1)


def step_rewards(n: int, seed: int, step: int, p: float = 0.5) -> np.ndarray:
    """Bernoulli(p) rewards [n] of one training step of the group-size sweep."""
    return (_rng(seed, _S_STEP_REWARD, step).random(n) < p).astype(np.float32)


def drifted_logprobs(logprobs: np.ndarray, lengths: np.ndarray, seed: int, scale: float = 0.1) -> np.ndarray:
    """float32 [N, max_new]: a stand-in for the log-probabilities of an older
    policy snapshot -- the given ones plus N(0, scale) noise at every valid
    position (t < lengths[s]), zero elsewhere."""
    lp = np.asarray(logprobs, np.float64)
    N, T = lp.shape
    noise = _rng(seed, _S_DRIFT).standard_normal((N, T)) * scale
    valid = np.arange(T)[None, :] < np.asarray(lengths)[:, None]
    return np.where(valid, lp + noise, 0.0).astype(np.float32)
