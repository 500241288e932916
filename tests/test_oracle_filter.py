"""Pins of the zero-variance group filter oracle: a group is dropped exactly
when its rewards are all equal, checked against the variance, against the
advantage (a dropped group has A = 0 for every member), and on hand cases."""
import numpy as np
import pytest

from oracle.advantage import group_advantage, zero_variance_filter


def _offsets(G):
    return np.concatenate([[0], np.cumsum(G)]).astype(np.int64)


def test_binary_rewards_hand_case():
    # all correct, all wrong, mixed, single member, mixed
    G = [4, 4, 4, 1, 2]
    r = np.array([1, 1, 1, 1, 0, 0, 0, 0, 1, 0, 1, 1, 0, 0, 1], np.float32)
    keep, ids = zero_variance_filter(r, G)
    np.testing.assert_array_equal(keep, [0, 0, 1, 0, 1])
    np.testing.assert_array_equal(ids, [2, 4])


def test_agrees_with_variance_on_finite_rewards():
    rng = np.random.default_rng(3)
    G = rng.integers(1, 20, size=400)
    N = int(G.sum())
    r = rng.integers(0, 3, size=N).astype(np.float32)
    off = _offsets(G)
    for p in range(0, len(G), 3):   # plant constant groups
        r[off[p]:off[p + 1]] = r[off[p]]
    keep, ids = zero_variance_filter(r, G)
    var = np.array([np.var(r[off[p]:off[p + 1]].astype(np.float64)) for p in range(len(G))])
    np.testing.assert_array_equal(keep, (var > 0).astype(np.int32))
    np.testing.assert_array_equal(ids, np.nonzero(var > 0)[0])
    assert 0 < len(ids) < len(G)


def test_dropped_groups_have_zero_advantage():
    rng = np.random.default_rng(5)
    G = rng.integers(2, 17, size=200)
    N = int(G.sum())
    r = (rng.random(N) < rng.random(N)).astype(np.float32)
    keep, _ = zero_variance_filter(r, G)
    a = group_advantage(r, G)
    off = _offsets(G)
    for p in range(len(G)):
        seg = a[off[p]:off[p + 1]]
        assert np.all(seg == 0) == (keep[p] == 0)


def test_signed_zero_nan_and_tiny_differences():
    G = [2, 2, 2, 1, 2]
    r = np.array([0.0, -0.0, 1.0, np.nextafter(np.float32(1), np.float32(2)), np.nan, np.nan, np.nan, 5.0, 5.0],
                 np.float32)
    keep, ids = zero_variance_filter(r, G)
    # -0 == +0; one ulp apart differs; NaN never equals itself; a lone NaN has nothing to differ from
    np.testing.assert_array_equal(keep, [0, 1, 1, 0, 0])
    np.testing.assert_array_equal(ids, [1, 2])


def test_rejects_bad_partitions():
    for G in ([4, 3], [4, 0, 4], [4, 5], [-1, 9]):
        with pytest.raises(ValueError):
            zero_variance_filter(np.ones(8, np.float32), G)
