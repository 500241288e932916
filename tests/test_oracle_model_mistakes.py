"""Planted mistakes in the oracle decoder must fail its independent pin (the
torch-functional forward of test_oracle_model.py).  Each case swaps one
building block of the oracle for a plausible wrong version on the CPU (a sign,
a pairing, a dropped term or factor, a wrong index, an off-by-one mask) and
checks that the logits then differ from the pin by far more than its
tolerance.  This shows the pin can catch such slips."""
import numpy as np
import pytest

from oracle.model import OracleModel
from test_oracle_model import GQA, torch_forward
from workload import make_weights


def _rope_sign(self, x, pos):
    half = self.s.head_dim // 2
    ang = np.asarray(pos, np.float64)[:, None] * self.inv_freq[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c + x2 * s, x2 * c - x1 * s], axis=-1)       # rotated the wrong way


def _rope_interleaved(self, x, pos):
    ang = np.asarray(pos, np.float64)[:, None] * self.inv_freq[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., 0::2], x[..., 1::2]                                     # pairs (2i, 2i+1)
    out = np.empty_like(x)
    out[..., 0::2], out[..., 1::2] = x1 * c - x2 * s, x2 * c + x1 * s
    return out


def _rmsnorm_no_eps(self, x, g):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) * g


def _rmsnorm_variance(self, x, g):
    return x / np.sqrt(np.var(x, axis=-1, keepdims=True) + self.s.rms_eps) * g


def _attention_variant(kind):
    def att(self, q, k, v, q_pos, k_pos):
        s = self.s
        rep = s.n_q_heads // s.n_kv_heads
        out = np.empty_like(q)
        if kind == "mask_excludes_self":
            mask = np.asarray(k_pos)[None, :] < np.asarray(q_pos)[:, None]
            mask[:, 0] = True                                               # keep a row non-empty
        else:
            mask = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]
        scale = 1.0 if kind == "no_scale" else 1.0 / np.sqrt(float(s.head_dim))
        for h in range(s.n_q_heads):
            kv = h % s.n_kv_heads if kind == "gqa_modulo" else h // rep
            sc = np.where(mask, (q[:, h, :] @ k[:, kv, :].T) * scale, -np.inf)
            p = np.exp(sc - sc.max(axis=1, keepdims=True))
            out[:, h, :] = (p / p.sum(axis=1, keepdims=True)) @ v[:, kv, :]
        return out
    return att


def _silu_sigmoid(a):
    return 1.0 / (1.0 + np.exp(-a))                                         # dropped the factor a



MISTAKES = {
    "rope_sign": ("rope", _rope_sign),
    "rope_interleaved_pairs": ("rope", _rope_interleaved),
    "rmsnorm_without_eps": ("rmsnorm", _rmsnorm_no_eps),
    "rmsnorm_mean_subtracted": ("rmsnorm", _rmsnorm_variance),
    "attention_unscaled": ("attention", _attention_variant("no_scale")),
    "attention_gqa_head_modulo": ("attention", _attention_variant("gqa_modulo")),
    "attention_mask_excludes_self": ("attention", _attention_variant("mask_excludes_self")),
    "silu_without_input_factor": ("silu", staticmethod(_silu_sigmoid)),
}


@pytest.mark.parametrize("name", sorted(MISTAKES))
def test_planted_mistake_fails_the_pin(name, monkeypatch):
    w = make_weights(GQA, 1)
    toks = np.random.default_rng(2).integers(0, GQA.vocab - 1, size=21)
    ref = torch_forward(GQA, w, toks)
    good = OracleModel(GQA, w, kv_storage="exact")
    ok = good.forward(toks, np.arange(len(toks)), good.new_cache())
    assert np.max(np.abs(ok - ref)) <= 1e-12              # the unplanted oracle meets the pin
    attr, fn = MISTAKES[name]
    monkeypatch.setattr(OracleModel, attr, fn)
    bad = OracleModel(GQA, w, kv_storage="exact")
    got = bad.forward(toks, np.arange(len(toks)), bad.new_cache())
    gap = float(np.max(np.abs(got - ref)))
    assert gap > 1e-8, (name, gap)                         # far outside the pin's 1e-12
