"""Pins for the oracle rollout and group advantage (CPU only)."""
import json
import math
import os

import numpy as np
import pytest

from workload import get_config, make_weights, make_inputs, ModelShape, Workload
from oracle.model import OracleModel
from oracle.rollout import rollout, group_offsets
from oracle.advantage import group_advantage

HERE = os.path.dirname(os.path.abspath(__file__))
TINY = get_config("tiny")


@pytest.fixture(scope="module")
def tiny():
    w = make_weights(TINY.shape, 0)
    return OracleModel(TINY.shape, w), make_inputs(TINY, 0)


def test_lengths_tokens_and_padding(tiny):
    m, inp = tiny
    out = rollout(m, inp.prompts, inp.G, TINY.max_new, 0, inp.forced_len)
    eos = TINY.shape.eos_id
    np.testing.assert_array_equal(out["lengths"], inp.forced_len)
    for s, L in enumerate(inp.forced_len):
        row = out["tokens"][s]
        assert row[L - 1] == eos and np.all(row[:L - 1] != eos) and np.all(row[:L - 1] >= 0)
        assert np.all(row[L:] == -1) and np.all(out["logprobs"][s, L:] == 0)
        assert np.all(out["logprobs"][s, :L] <= 0)


def test_logprobs_normalised_and_match_recorded_logits(tiny):
    m, inp = tiny
    out = rollout(m, inp.prompts, inp.G, TINY.max_new, 0, inp.forced_len, record_steps=TINY.max_new)
    for (s, t), z in out["logits"].items():
        ls = z - (np.log(np.sum(np.exp(z - z.max()))) + z.max())
        assert abs(np.sum(np.exp(ls)) - 1) < 1e-12
        assert abs(out["logprobs"][s, t] - ls[out["tokens"][s, t]]) < 1e-12


def test_cached_rollout_logits_equal_full_recompute(tiny):
    m, inp = tiny
    out = rollout(m, inp.prompts, inp.G, TINY.max_new, 0, inp.forced_len, record_steps=TINY.max_new)
    prompt = inp.prompts[0]
    for s in range(int(inp.G[0])):
        L = int(out["lengths"][s])
        seq = np.concatenate([prompt, out["tokens"][s, :L - 1]])
        full = m.forward(seq, np.arange(len(seq)), m.new_cache())
        for t in range(L):
            np.testing.assert_allclose(out["logits"][(s, t)], full[len(prompt) - 1 + t], rtol=0, atol=1e-11)


def test_shared_prefix_equals_unshared(tiny):
    """G siblings of one prompt == G copies of the prompt with G = 1 each (the
    sequence ids coincide, so the noise streams do too)."""
    m, inp = tiny
    G = int(inp.G[0])
    a = rollout(m, inp.prompts[:1], [G], TINY.max_new, 9, inp.forced_len)
    b = rollout(m, np.repeat(inp.prompts[:1], G, axis=0), [1] * G, TINY.max_new, 9, inp.forced_len)
    for k in ("tokens", "lengths"):
        np.testing.assert_array_equal(a[k], b[k])
    # batched BLAS rows may round differently in the last bit
    np.testing.assert_allclose(a["logprobs"], b["logprobs"], rtol=0, atol=1e-12)


def test_natural_eos_mode_retires_on_eos():
    shape = ModelShape(1, 32, 2, 2, 16, 64, 8, 1e4, dtype="f32")   # tiny vocab: EOS comes early
    m = OracleModel(shape, make_weights(shape, 3))
    out = rollout(m, [np.array([1, 2, 3])] * 3, [4, 4, 4], 40, 5, None)
    for s in range(12):
        L = out["lengths"][s]
        row = out["tokens"][s]
        assert 1 <= L <= 40
        assert row[L - 1] == shape.eos_id or L == 40
        assert np.all(row[:L - 1] != shape.eos_id) and np.all(row[L:] == -1)


def test_step_zero_siblings_share_logits_but_not_noise(tiny):
    m, inp = tiny
    out = rollout(m, inp.prompts, inp.G, TINY.max_new, 0, inp.forced_len, record_steps=1)
    z0 = [out["logits"][(s, 0)] for s in range(int(inp.G[0]))]
    for z in z0[1:]:
        np.testing.assert_array_equal(z, z0[0])
    assert len(set(out["tokens"][:, 0].tolist())) > 1


def test_group_offsets():
    np.testing.assert_array_equal(group_offsets([4, 8, 1]), [0, 4, 12, 13])


# ---------------------------------------------------------------- advantage
def test_advantage_worked_examples():
    with open(os.path.join(HERE, "golden", "advantage_worked.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        a = group_advantage(np.array(c["rewards"], np.float32), c["G"], 1e-6, c["ddof"])
        np.testing.assert_allclose(a, np.array(c["advantages"], np.float32), rtol=2e-7, atol=0)


@pytest.mark.parametrize("ddof", [0, 1])
def test_advantage_invariants(ddof):
    rng = np.random.default_rng(0)
    G = np.array([4, 8, 16, 32, 3, 2])
    r = rng.normal(size=int(G.sum())).astype(np.float32)
    a = group_advantage(r, G, 1e-6, ddof).astype(np.float64)
    off = group_offsets(G)
    for p in range(len(G)):
        seg, ra = a[off[p]:off[p + 1]], r[off[p]:off[p + 1]].astype(np.float64)
        sigma = np.std(ra, ddof=ddof)
        assert abs(seg.sum()) <= 1e-6 * len(seg)
        assert abs(np.std(seg, ddof=ddof) - sigma / (sigma + 1e-6)) < 1e-6
        np.testing.assert_allclose(seg, (ra - np.mean(ra)) / (sigma + 1e-6), rtol=1e-6, atol=1e-7)


def test_advantage_constant_groups_and_bernoulli():
    G = np.array([4, 4, 1, 16])
    r = np.array([1, 1, 1, 1, 0, 0, 0, 0, 1] + [1, 0] * 8, np.float32)
    a = group_advantage(r, G)
    assert np.all(a[:9] == 0)
    # a balanced Bernoulli group: +-(0.5 / (std + eps)) with std = sqrt(16/4/15)
    sd = math.sqrt(16 * 0.25 / 15)
    np.testing.assert_allclose(a[9:], np.where(r[9:] > 0, 0.5, -0.5) / (sd + 1e-6), rtol=1e-6)


def test_advantage_permutation_equivariant():
    rng = np.random.default_rng(4)
    r = rng.random(16).astype(np.float32)
    perm = rng.permutation(16)
    np.testing.assert_array_equal(group_advantage(r, [16])[perm], group_advantage(r[perm], [16]))
