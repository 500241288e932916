"""Pins for the oracle's Philox4x64-10 and Gumbel noise (CPU only).

The oracle's generator is checked bit-for-bit against numpy's independent
Philox4x64-10 implementation (numpy increments its counter before producing a
block, so its first block for state counter c is the Philox image of c + 1).
"""
import math

import numpy as np
import pytest
from scipy import stats

from oracle.philox import (philox4x64_10, gumbel_uniform_bits, gumbel_uniform_bits_batch,
                           uniforms_from_bits, gumbel_noise, TAG_GUMBEL)
from oracle.sampling import sample_token



def numpy_block(ctr, key):
    """The Philox block at counter ``ctr`` as produced by numpy.random.Philox."""
    c = [int(x) for x in ctr]
    # numpy adds one (with carry) before generating: hand it ctr - 1.
    v = sum(x << (64 * i) for i, x in enumerate(c))
    v = (v - 1) % (1 << 256)
    c = [(v >> (64 * i)) & ((1 << 64) - 1) for i in range(4)]
    bg = np.random.Philox(key=np.array(key, np.uint64), counter=np.array(c, np.uint64))
    return bg.random_raw(4)


@pytest.mark.parametrize("ctr,key", [
    ((0, 0, 0, 0), (0, 0)),
    ((1, 0, 0, 0), (0, 1)),
    ((5, 3, 17, 0), (12345, TAG_GUMBEL)),
    ((18991, 4095, 511, 0), (2 ** 63 + 5, TAG_GUMBEL)),
    ((2 ** 64 - 1, 2 ** 64 - 1, 2 ** 64 - 1, 2 ** 64 - 1), (2 ** 64 - 1, 2 ** 64 - 1)),
    ((0, 7, 0, 9), (0xDEADBEEF, 3)),
])
def test_philox_matches_numpy(ctr, key):
    ours = philox4x64_10(np.array([ctr], np.uint64), key)[0]
    np.testing.assert_array_equal(ours, numpy_block(ctr, key))


def test_philox_many_counters_match_numpy_stream():
    key = (987654321, TAG_GUMBEL)
    bg = np.random.Philox(key=np.array(key, np.uint64), counter=np.array([0, 3, 11, 0], np.uint64))
    ref = bg.random_raw(4 * 300).reshape(300, 4)          # blocks at counters (1..300, 3, 11, 0)
    ctr = np.zeros((300, 4), np.uint64)
    ctr[:, 0] = np.arange(1, 301, dtype=np.uint64)
    ctr[:, 1], ctr[:, 2] = 3, 11
    np.testing.assert_array_equal(philox4x64_10(ctr, key), ref)


def test_gumbel_bits_layout():
    seed, t, s, V = 42, 9, 5, 37
    bits = gumbel_uniform_bits(seed, t, s, V)
    for v in [0, 1, 7, 8, 15, 36]:
        w = numpy_block((v >> 3, t, s, 0), (seed, TAG_GUMBEL))
        j = v & 7
        word = int(w[j >> 1])
        expect = (word >> (32 * (j & 1))) & 0xFFFFFFFF
        assert int(bits[v]) == expect
    batch = gumbel_uniform_bits_batch(seed, t, np.array([5, 6]), V)
    np.testing.assert_array_equal(batch[0], bits)
    np.testing.assert_array_equal(batch[1], gumbel_uniform_bits(seed, t, 6, V))


def test_uniform_mapping_endpoints_and_exactness():
    x = np.array([0, 1, 511, 512, 0xFFFFFFFF, 0x80000000], np.uint32)
    u = uniforms_from_bits(x)
    assert u[0] == np.float32(2.0 ** -24) and u[1] == u[0] and u[2] == u[0]
    assert u[3] == np.float32(3 * 2.0 ** -24)
    assert u[4] == np.float32(1 - 2.0 ** -24)
    assert u[5] == np.float32(0.5 + 2.0 ** -24)
    assert np.all((u > 0) & (u < 1))
    # exactly representable: converting back through float64 changes nothing
    assert np.all(u.astype(np.float64).astype(np.float32) == u)


def test_uniforms_are_uniform():
    bits = gumbel_uniform_bits_batch(7, 0, np.arange(64), 4096).ravel()
    u = uniforms_from_bits(bits).astype(np.float64)
    assert stats.kstest(u, "uniform").pvalue > 1e-3
    g = -np.log(-np.log(u))
    assert stats.kstest(g, "gumbel_r").pvalue > 1e-3


def _gumbel_max_counts(z, n_draws, seed=3, T=1.0):
    V = len(z)
    counts = np.zeros(V, np.int64)
    chunk = 100_000
    zs = (np.asarray(z, np.float32) / np.float32(T)).astype(np.float32)
    for c0 in range(0, n_draws, chunk):
        s = np.arange(c0, min(n_draws, c0 + chunk))
        g = gumbel_noise(seed, 0, s, V)            # the oracle's own noise, one row per draw
        y = np.argmax(zs[None, :] + g, axis=1)
        counts += np.bincount(y, minlength=V)
    return counts


@pytest.mark.parametrize("T", [1.0, 0.7])
def test_gumbel_max_frequencies_match_softmax(T):
    rng = np.random.default_rng(0)
    z = rng.normal(0, 1.5, size=16)
    n = 1_000_000
    counts = _gumbel_max_counts(z, n, T=T)
    p = np.exp(z / T - np.max(z / T)); p /= p.sum()
    assert stats.chisquare(counts, n * p).pvalue > 1e-3


@pytest.mark.parametrize("T", [1.0, 0.7])
def test_sample_token_frequencies_match_softmax(T):
    # the oracle's full sampling decision (scaling by T, noise, argmax), one
    # call per draw: 20,000 draws on 6 tokens against softmax(z/T)
    z = np.array([0.3, -1.1, 1.4, 0.0, -0.4, 0.9])
    n = 20_000
    counts = np.bincount([sample_token(z, 9, 0, s, len(z) - 1, T)[0] for s in range(n)], minlength=len(z))
    p = np.exp(z / T - np.max(z / T)); p /= p.sum()
    assert stats.chisquare(counts, n * p).pvalue > 1e-3


def test_gumbel_max_flat_is_uniform_and_gap_wins():
    n = 200_000
    counts = _gumbel_max_counts(np.zeros(8), n)
    assert stats.chisquare(counts, np.full(8, n / 8)).pvalue > 1e-3
    z = np.zeros(16); z[11] = 30.0
    counts = _gumbel_max_counts(z, 50_000)
    assert counts[11] == 50_000


def test_sample_token_forced_eos_and_logprob():
    rng = np.random.default_rng(1)
    V, eos = 64, 63
    z = rng.normal(0, 1, V); z[eos] = 50.0           # EOS would always win if not masked
    for t in range(5):
        y, lp, mg = sample_token(z, 11, t, 2, eos, 1.0, forced_len=6)
        assert y != eos and mg >= 0
        lse = math.log(np.sum(np.exp(z - z.max()))) + z.max()
        assert abs(lp - (z[y] - lse)) < 1e-12
    y, lp, mg = sample_token(z, 11, 5, 2, eos, 1.0, forced_len=6)
    assert y == eos and mg == math.inf
    assert abs(lp - (z[eos] - (math.log(np.sum(np.exp(z - z.max()))) + z.max()))) < 1e-12
    # natural mode: EOS is a normal token and wins here
    y, _, _ = sample_token(z, 11, 0, 2, eos, 1.0, forced_len=None)
    assert y == eos


def test_sample_token_tie_goes_to_lowest_id():
    # identical logits + the same noise at two ids cannot happen by accident,
    # so construct the decision directly: equal scores -> np.argmax picks first.
    V = 16
    g = gumbel_noise(5, 0, 0, V)
    z = -g.astype(np.float64)             # every fp32 score is (nearly) 0
    z32 = z.astype(np.float32)
    score = z32 + g
    y, _, _ = sample_token(z, 5, 0, 0, V - 1, 1.0, forced_len=None)
    best = np.flatnonzero(score == score.max())
    assert y == best[0]
