"""Pins of the GRPO loss-forward oracle (CPU only).

* Teacher-forced log-probabilities (one causal forward per sequence, no cache
  sharing) reproduce the log-probabilities the oracle rollout reported while
  decoding incrementally -- two independent routes to the same numbers.
* The clipped surrogate matches its piecewise closed form, the hand-worked
  quadrants of the PPO clip, the ratio-1 closed forms (-mean advantage; zero
  for standardised groups under the sequence mean) and the keep mask as a
  subset."""
import math

import numpy as np
import pytest

from workload import get_config, make_weights, make_inputs, drifted_logprobs
from oracle.model import OracleModel
from oracle.rollout import rollout
from oracle.advantage import group_advantage
from oracle.grpo import teacher_forced_logprobs, clipped_surrogate

TINY = get_config("tiny")


@pytest.fixture(scope="module")
def tiny():
    return OracleModel(TINY.shape, make_weights(TINY.shape, 0)), make_inputs(TINY, 0)


@pytest.mark.parametrize("T", [1.0, 0.7])
def test_recompute_equals_rollout_logprobs(tiny, T):
    m, inp = tiny
    out = rollout(m, inp.prompts, inp.G, TINY.max_new, 3, inp.forced_len, temperature=T)
    lp = teacher_forced_logprobs(m, inp.prompts, inp.G, out["tokens"], out["lengths"], T)
    np.testing.assert_allclose(lp, out["logprobs"], rtol=0, atol=1e-10)
    assert np.all(lp[np.arange(TINY.max_new)[None, :] >= out["lengths"][:, None]] == 0)


def test_recompute_bf16_model_matches_rollout():
    wl = get_config("tiny")
    shape = wl.shape.__class__(**{**wl.shape.__dict__, "dtype": "bf16"})
    m = OracleModel(shape, make_weights(shape, 1))
    inp = make_inputs(wl, 1)
    out = rollout(m, inp.prompts, inp.G, wl.max_new, 5, inp.forced_len)
    lp = teacher_forced_logprobs(m, inp.prompts, inp.G, out["tokens"], out["lengths"])
    np.testing.assert_allclose(lp, out["logprobs"], rtol=0, atol=1e-10)


def test_recompute_rejects_bad_lengths(tiny):
    m, inp = tiny
    tok = np.zeros((inp.n_seq, TINY.max_new), np.int32)
    for bad in (0, TINY.max_new + 1):
        L = np.full(inp.n_seq, 3, np.int32)
        L[-1] = bad
        with pytest.raises(ValueError):
            teacher_forced_logprobs(m, inp.prompts, inp.G, tok, L)


def test_clip_quadrants_by_hand():
    # one token per sequence; eps = 0.2
    rho = np.array([1.5, 0.5, 0.5, 1.5, 1.1, 0.9])
    A = np.array([1.0, -1.0, 1.0, -1.0, 2.0, -2.0])
    want = np.array([1.2, -0.8, 0.5, -1.5, 2.2, -1.8])   # clip, clip, keep, keep, inside, inside
    old = np.zeros((6, 1))
    new = np.log(rho)[:, None]
    for k in range(6):
        loss, frac, nt, ns = clipped_surrogate(new[k:k + 1], old[k:k + 1], A[k:k + 1], [1], [1])
        assert abs(loss + want[k]) < 1e-12 and nt == 1 and ns == 1
        assert frac == (1.0 if k < 2 else 0.0)
    loss, frac, nt, ns = clipped_surrogate(new, old, A, np.ones(6, int), [6])
    assert abs(loss + want.mean()) < 1e-12 and frac == pytest.approx(2 / 6)


def test_decoupled_clip_upper_bound():
    # DAPO clip-higher: eps_hi = 0.28 lets a positive-advantage token reach 1.28
    new, old = np.log([[1.5]]), np.zeros((1, 1))
    assert clipped_surrogate(new, old, [1.0], [1], [1], 0.2, 0.28)[0] == pytest.approx(-1.28, abs=1e-12)
    assert clipped_surrogate(np.log([[0.5]]), old, [-1.0], [1], [1], 0.2, 0.28)[0] == pytest.approx(0.8, abs=1e-12)


def _piecewise(new, old, adv, lengths, eps_lo, eps_hi):
    """The same objective written as cases of the sign of A."""
    terms, clips = [], 0
    for s in range(len(adv)):
        for t in range(int(lengths[s])):
            rho = math.exp(float(new[s, t]) - float(old[s, t]))
            a = float(adv[s])
            if a > 0 and rho > 1 + eps_hi:
                terms.append((1 + eps_hi) * a); clips += 1
            elif a < 0 and rho < 1 - eps_lo:
                terms.append((1 - eps_lo) * a); clips += 1
            else:
                terms.append(rho * a)
    return terms, clips


@pytest.mark.parametrize("eps", [(0.2, 0.2), (0.2, 0.28), (0.1, 0.5)])
def test_matches_piecewise_form(eps):
    rng = np.random.default_rng(7)
    G = [4, 8, 3, 16]
    N, T = sum(G), 24
    L = rng.integers(1, T + 1, size=N)
    old = rng.normal(-2, 1, size=(N, T))
    new = old + rng.normal(0, 0.3, size=(N, T))
    adv = rng.normal(size=N)
    terms, clips = _piecewise(new, old, adv, L, *eps)
    loss, frac, nt, ns = clipped_surrogate(new, old, adv, L, G, *eps, mode="token")
    assert nt == L.sum() and ns == N and 0 < clips < nt
    assert loss == pytest.approx(-sum(terms) / nt, rel=1e-12)
    assert frac == pytest.approx(clips / nt, rel=1e-12)
    o = np.concatenate([[0], np.cumsum(L)])
    seq_means = [sum(terms[o[s]:o[s + 1]]) / L[s] for s in range(N)]
    assert clipped_surrogate(new, old, adv, L, G, *eps, mode="seq")[0] == pytest.approx(-np.mean(seq_means), rel=1e-12)


def test_ratio_one_closed_forms():
    rng = np.random.default_rng(8)
    G = [8, 8, 4, 16]
    N, T = sum(G), 30
    L = rng.integers(1, T + 1, size=N)
    lp = rng.normal(-2, 1, size=(N, T))
    r = (rng.random(N) < 0.5).astype(np.float32)
    adv = group_advantage(r, G, 1e-6, 0).astype(np.float64)
    tok = clipped_surrogate(lp, lp, adv, L, G, mode="token")
    assert tok[0] == pytest.approx(-np.sum(L * adv) / L.sum(), rel=1e-12, abs=1e-15) and tok[1] == 0
    seq = clipped_surrogate(lp, lp, adv, L, G, mode="seq")
    assert seq[0] == pytest.approx(-np.mean(adv), abs=1e-12)
    assert abs(seq[0]) < 1e-6     # ddof 0 standardised groups sum to zero


def test_equal_lengths_make_modes_agree():
    rng = np.random.default_rng(9)
    G = [4, 4]
    new, old = rng.normal(size=(8, 5)), rng.normal(size=(8, 5))
    adv, L = rng.normal(size=8), np.full(8, 5)
    assert clipped_surrogate(new, old, adv, L, G, mode="token")[0] == pytest.approx(
        clipped_surrogate(new, old, adv, L, G, mode="seq")[0], rel=1e-12)


def test_keep_mask_is_the_subset():
    rng = np.random.default_rng(10)
    G = [4, 2, 8, 3]
    N, T = sum(G), 12
    L = rng.integers(1, T + 1, size=N)
    new, old, adv = rng.normal(size=(N, T)), rng.normal(size=(N, T)), rng.normal(size=N)
    keep = [1, 0, 1, 0]
    sel = np.r_[0:4, 6:14]
    for mode in ("token", "seq"):
        a = clipped_surrogate(new, old, adv, L, G, mode=mode, keep=keep)
        b = clipped_surrogate(new[sel], old[sel], adv[sel], L[sel], [4, 8], mode=mode)
        assert a == pytest.approx(b, rel=1e-12)
    assert clipped_surrogate(new, old, adv, L, G, keep=[0, 0, 0, 0]) == (0.0, 0.0, 0, 0)


def test_drifted_logprobs_only_touch_valid_positions(tiny):
    m, inp = tiny
    out = rollout(m, inp.prompts, inp.G, TINY.max_new, 0, inp.forced_len)
    old = drifted_logprobs(out["logprobs"], out["lengths"], 0, 0.1)
    valid = np.arange(TINY.max_new)[None, :] < out["lengths"][:, None]
    assert np.all(old[~valid] == 0)
    d = (old - out["logprobs"])[valid]
    assert 0.05 < np.std(d) < 0.2
