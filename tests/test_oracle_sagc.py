"""Pins of the oracle's group-size controller (Sec. 3.1 Eq. ratio / Eq. event,
Sec. 4.2-4.3, Algorithm 1).

* Gamma / Beta draws: Kolmogorov-Smirnov against scipy's distributions and
  the Beta mean a / (a + b).
* Straggler statistics: hand-worked groups, numpy's median, the strict
  inequality at R = tau.
* Dual ascent and posterior update: worked numbers.
* Selection: zero lambda picks the largest neighbour (u is increasing), an
  exact tie goes to the smaller size, moves never leave the neighbourhood.
* Closed loop on synthetic lengths: the posterior straggler risk separates as
  p16 > p8 > p4 (the ordering the paper's Fig. 4 reports) by step 30.
"""
import math

import numpy as np
import pytest
import scipy.stats as ss

from oracle import sagc as O


@pytest.mark.parametrize("a", [0.3, 1.0, 2.5, 12.0])
def test_gamma_draws_follow_gamma(a):
    x = [O.gamma_draw(11, s, 3, a) for s in range(3000)]
    assert ss.kstest(x, "gamma", args=(a,)).pvalue > 1e-3
    assert min(x) > 0.0


@pytest.mark.parametrize("a,b", [(1.0, 1.0), (1.95, 0.95), (0.4, 3.0), (20.0, 5.0)])
def test_beta_draws_follow_beta(a, b):
    x = np.array([O.beta_draw(5, s, 1, a, b) for s in range(3000)])
    assert ss.kstest(x, "beta", args=(a, b)).pvalue > 1e-3
    sd = math.sqrt(a * b / ((a + b) ** 2 * (a + b + 1)) / len(x))
    assert abs(x.mean() - a / (a + b)) < 4 * sd
    assert np.all((x > 0) & (x < 1))


def test_draws_depend_on_every_counter_field():
    base = O.beta_draw(1, 2, 0, 2.0, 3.0)
    assert base == O.beta_draw(1, 2, 0, 2.0, 3.0)
    for other in (O.beta_draw(2, 2, 0, 2.0, 3.0), O.beta_draw(1, 3, 0, 2.0, 3.0), O.beta_draw(1, 2, 1, 2.0, 3.0)):
        assert other != base


def test_u53_range():
    assert O.u53(0) == 0.5 * 2.0 ** -53
    assert O.u53(2 ** 64 - 1) == 1.0 - 0.5 * 2.0 ** -53


def test_group_stats_worked_examples():
    st = O.group_stats([1, 2, 3, 4, 5, 5, 5, 9, 1, 7], [4, 5, 1], 1.25)
    assert st[0] == (4.0, 2.5, 1.6, 1.0)            # even group: mean of the middle pair
    assert st[1] == (9.0, 5.0, 1.8, 1.0)            # odd group: the middle value
    assert st[2] == (7.0, 7.0, 1.0, 0.0)            # single completion: R = 1
    # R exactly tau is not a straggler (strict inequality)
    assert O.group_stats([4, 4, 5, 3], [4], 1.25)[0][3] == 0.0   # median 4, max 5: R = 1.25
    assert O.group_stats([4, 4, 6, 3], [4], 1.25)[0][3] == 1.0


def test_group_stats_match_numpy():
    rng = np.random.default_rng(0)
    G = [1, 2, 3, 4, 7, 8, 16, 33]
    L = rng.integers(1, 100, size=sum(G))
    off = 0
    for g, (lmax, lmed, R, S) in zip(G, O.group_stats(L, G, 1.3)):
        seg = L[off:off + g]
        off += g
        assert lmax == seg.max() and lmed == np.median(seg)
        assert R == seg.max() / np.median(seg) and S == float(R > 1.3)


def test_dual_and_posterior_worked_example():
    cfg = O.SagcConfig(sizes=(4, 8, 16), delta=0.1, eta=0.5, gamma=0.95, seed=0)
    st = O.sagc_init(cfg)
    i0 = st.g_index
    O.sagc_step(cfg, st, [1.0, 1.0])                 # S_bar = 1
    assert st.lam == 0.5 * (1.0 - 0.1)
    assert st.alpha[i0] == 0.95 + 1.0 and st.beta[i0] == 0.95
    assert all(st.alpha[j] == 1.0 and st.beta[j] == 1.0 for j in range(3) if j != i0)
    i1 = st.g_index
    O.sagc_step(cfg, st, [0.0, 1.0, 0.0, 0.0])      # S_bar = 0.25
    assert st.lam == max(0.0, 0.45 + 0.5 * (0.25 - 0.1))
    for _ in range(40):                               # no stragglers: lambda decays to 0 and stays there
        O.sagc_step(cfg, st, [0.0])
        assert st.lam >= 0.0
    assert st.lam == 0.0
    assert st.step == 42 and i1 in (0, 1, 2)


def test_choice_rules():
    cfg = O.SagcConfig(sizes=(4, 8, 16))
    # lambda = 0: the utility alone, so the largest size of the neighbourhood
    assert O.sagc_choose(cfg, 0.0, [0.9, 0.9, 0.9], 0)[0] == 1
    assert O.sagc_choose(cfg, 0.0, [0.9, 0.9, 0.9], 1)[0] == 2
    # exact tie between 4 (2 - 4*0.25) and 8 (3 - 4*0.5), 16 scoring 4 - 4*0.875: the smaller size wins
    best, scores = O.sagc_choose(cfg, 4.0, [0.25, 0.5, 0.875], 1)
    assert scores == [1.0, 1.0, 0.5] and best == 0
    # a strong penalty on large sizes moves down one step at a time
    assert O.sagc_choose(cfg, 100.0, [0.1, 0.5, 0.9], 2)[0] == 1


def _closed_loop(seed, steps, s0=0.2, s1=0.1, eb=64):
    """Synthetic rollouts at a fixed effective batch of eb sequences: lengths
    lognormal around 1200 tokens with a spread that narrows over training."""
    cfg = O.SagcConfig(sizes=(4, 8, 16), seed=seed)
    st = O.sagc_init(cfg)
    rng = np.random.default_rng(1000 + seed)
    seq, risk = [], []
    for t in range(steps):
        G = cfg.sizes[st.g_index]
        sigma = s0 + (s1 - s0) * t / steps
        L = np.floor(np.exp(rng.normal(math.log(1200.0), sigma, size=eb)) + 0.5).astype(int)
        S = [s[3] for s in O.group_stats(L, [G] * (eb // G), cfg.tau)]
        nxt = O.sagc_step(cfg, st, S)
        seq.append((G, nxt))
        risk.append([a / (a + b) for a, b in zip(st.alpha, st.beta)])
    return seq, risk, st


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_closed_loop_separates_arms(seed):
    seq, risk, st = _closed_loop(seed, 120)
    sizes = (4, 8, 16)
    for g, nxt in seq:                                # local moves only
        assert abs(sizes.index(g) - sizes.index(nxt)) <= 1
    assert risk[29][2] > risk[29][1] > risk[29][0]     # p16 > p8 > p4 by step 30
    assert risk[-1][2] > risk[-1][1] > risk[-1][0]
    assert st.lam >= 0.0


@pytest.mark.parametrize("sizes", [(4, 8, 16), (2, 4), (4, 8, 16, 32, 64)])
def test_initial_size_is_uniform_over_the_admitted_sizes(sizes):
    """Algorithm 1 starts from a size drawn at random from the admitted list:
    over 3,000 seeds every size is drawn, and the counts pass a chi-square
    test against the uniform distribution."""
    n = 3000
    idx = [O.sagc_init(O.SagcConfig(sizes=sizes, seed=s)).g_index for s in range(n)]
    assert min(idx) >= 0 and max(idx) < len(sizes)
    counts = np.bincount(idx, minlength=len(sizes))
    assert np.all(counts > 0), counts
    assert ss.chisquare(counts).pvalue > 1e-3, counts


def test_initial_size_state():
    st = O.sagc_init(O.SagcConfig(sizes=(4, 8, 16), seed=3))
    assert st.lam == 0.0 and st.step == 0
    assert st.alpha == [1.0] * 3 and st.beta == [1.0] * 3
