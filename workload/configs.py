"""Model shapes and workload recipes for the five synthetic rollout workloads.

The shapes are random-init decoders standing in for the 3B policies trained in
the paper's experiments (Sec. 5.1): the paper's models and dataset are not
available, so every workload is synthetic and seeded.  Completion lengths are
forced by a seeded draw (EOS is masked before the drawn length and forced at
it) so that the ragged, heavy-tailed length mix that makes stragglers
(Sec. 3.1, Eq. ratio) is reproducible.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rope_theta: float
    rms_eps: float = 1e-6
    dtype: str = "bf16"          # "f32" or "bf16": storage type of matrices and KV

    @property
    def eos_id(self) -> int:
        return self.vocab - 1

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def matrix_params_per_layer(self) -> int:
        d, f = self.d_model, self.ffn_dim
        return d * (self.q_dim + 2 * self.kv_dim) + self.q_dim * d + 3 * d * f

    def decode_weight_bytes(self) -> int:
        """Bytes of weights one decode step must stream: every layer's matrices
        and norm gains (norm gains are fp32), the final norm and the lm_head.
        The embedding is gathered per token and is not streamed."""
        per_layer = self.matrix_params_per_layer() * self.elem_bytes + 2 * self.d_model * 4
        return self.n_layers * per_layer + self.d_model * 4 + self.vocab * self.d_model * self.elem_bytes

    def kv_bytes_per_token(self) -> int:
        return self.n_layers * 2 * self.kv_dim * self.elem_bytes


@dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    n_prompts: int
    prompt_len: int
    max_new: int
    group_size: Optional[int]                 # fixed G, or None for per-prompt draws
    group_choices: Tuple[int, ...] = ()       # admissible sizes when group_size is None
    length_dist: Tuple = ("uniform", 8, 32)   # ("uniform", a, b) | ("lognormal", mu, sigma)
    reward_dist: Tuple = ("const_p", 0.5)     # ("const_p", p) | ("uniform_p", lo, hi)
    note: str = ""


_TINY = ModelShape(2, 128, 4, 4, 32, 512, 512, 1e4, dtype="f32")
_GPT2S = ModelShape(12, 768, 12, 12, 64, 3072, 32000, 1e4, dtype="bf16")
_Q15 = ModelShape(28, 1536, 12, 2, 128, 8960, 151936, 1e6, dtype="bf16")
_Q7 = ModelShape(28, 3584, 28, 4, 128, 18944, 152064, 1e6, dtype="bf16")

import math as _m

CONFIGS = {
    "tiny": Workload("tiny", _TINY, 1, 16, 32, 4, length_dist=("uniform", 8, 32),
                     reward_dist=("const_p", 0.5)),
    "gpt2s": Workload("gpt2s", _GPT2S, 8, 256, 1024, 8, length_dist=("lognormal", _m.log(300.0), 0.6),
                      reward_dist=("uniform_p", 0.1, 0.9)),
    "1.5b": Workload("1.5b", _Q15, 32, 512, 4096, 16, length_dist=("lognormal", _m.log(1200.0), 0.8),
                     reward_dist=("uniform_p", 0.1, 0.9)),
    "1.5b-dyn": Workload("1.5b-dyn", _Q15, 32, 512, 4096, None, group_choices=(4, 8, 16, 32),
                         length_dist=("lognormal", _m.log(1200.0), 0.8),
                         reward_dist=("uniform_p", 0.1, 0.9)),
    "7b": Workload("7b", _Q7, 16, 1024, 8192, 16, length_dist=("lognormal", _m.log(2500.0), 0.9),
                   reward_dist=("uniform_p", 0.1, 0.9)),
}


def get_config(name: str) -> Workload:
    try:
        return CONFIGS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; choose one of {sorted(CONFIGS)}") from None
