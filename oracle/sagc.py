"""Straggler-aware group-size control: the reference controller.

Test infrastructure (this package is the oracle): plain Python scalars, one
step of Algorithm 1 (SAGC) per call, written from the paper's method section.

* Straggler statistics (Eq. ratio, Eq. event): for a group's completion
  lengths l_1..l_G, R = max_i l_i / median_i l_i and S = 1[R > tau].  The
  median of an even-sized group is the mean of the two middle order statistics
  (reading: the paper does not say which median; this is numpy's).
* Dual ascent (Eq. lambda_update): lambda <- max(0, lambda + eta (S_bar - delta))
  with S_bar the mean straggler event over the step's completed groups.
* Discounted Beta posterior of the current arm only: alpha_G <- gamma alpha_G +
  S_bar, beta_G <- gamma beta_G + (1 - S_bar); every arm starts at (1, 1).
* Thompson sampling: p~_G ~ Beta(alpha_G, beta_G) for every arm; score
  u(G) - lambda p~_G with u(G) = log2(G) (Eq. lagrangian_score).
* Local move (Eq. choose_G restricted to the neighbourhood of Algorithm 1):
  the next G maximises the score over {G, prev(G), next(G)} within the
  admissible sizes; ties go to the smaller G.
* G_0 is drawn at random from the admissible sizes.

Random numbers (a reading: the paper does not fix a generator).  Every draw
comes from Philox4x64-10 with key (seed, TAG_SAGC) and counter
(step, stream, attempt, 0); a 64-bit word w becomes the double
((w >> 11) + 0.5) * 2**-53 in (0, 1).  Gamma(a) variates follow Marsaglia and
Tsang (2000): d = a - 1/3, c = 1/sqrt(9d); per attempt a normal x from the
Box-Muller transform of words 0 and 1, v = (1 + c x)^3, accept when v > 0 and
log(u) < x^2/2 + d - d v + d log v with u from word 2, returning d v; shapes
below one use Gamma(a + 1) * U^(1/a) with U from word 3 of attempt 0.
Beta(a, b) = X / (X + Y) with X ~ Gamma(a) on stream 2k and Y ~ Gamma(b) on
stream 2k + 1 for arm k.  G_0 uses word 0 of counter (2**63, 0, 0, 0).
The arithmetic is plain double precision in the order written here.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from .philox import philox4x64_10

TAG_SAGC = 2


def _words(seed: int, ctr) -> list[int]:
    w = philox4x64_10(np.array([ctr], dtype=np.uint64), (seed, TAG_SAGC))[0]
    return [int(x) for x in w]


def u53(word: int) -> float:
    """64-bit word -> double ((w >> 11) + 0.5) * 2**-53, strictly inside (0, 1)."""
    return ((word >> 11) + 0.5) * 2.0 ** -53


def gamma_draw(seed: int, step: int, stream: int, a: float) -> float:
    """Gamma(a, 1) by Marsaglia-Tsang on the stream (step, stream)."""
    if not a > 0.0:
        raise ValueError("gamma shape must be > 0")
    boost = a < 1.0
    shape = a + 1.0 if boost else a
    d = shape - 1.0 / 3.0
    c = 1.0 / math.sqrt(9.0 * d)
    attempt = 0
    first = None
    while True:
        w = _words(seed, (step, stream, attempt, 0))
        if first is None:
            first = w
        x = math.sqrt(-2.0 * math.log(u53(w[0]))) * math.cos(2.0 * math.pi * u53(w[1]))
        t = 1.0 + c * x
        attempt += 1
        if t <= 0.0:
            continue
        v = t * t * t
        if math.log(u53(w[2])) < 0.5 * x * x + d - d * v + d * math.log(v):
            g = d * v
            break
    if boost:
        g = g * math.pow(u53(first[3]), 1.0 / a)
    return g


def beta_draw(seed: int, step: int, arm: int, a: float, b: float) -> float:
    x = gamma_draw(seed, step, 2 * arm, a)
    y = gamma_draw(seed, step, 2 * arm + 1, b)
    return x / (x + y)


def group_stats(lengths, G, tau: float):
    """Per group: (l_max, l_median, R, S) for prompt-major lengths [sum(G)]."""
    out = []
    off = 0
    for g in G:
        seg = sorted(int(v) for v in lengths[off:off + g])
        off += g
        lmax = seg[-1]
        if g % 2:
            lmed = float(seg[g // 2])
        else:
            lmed = (seg[g // 2 - 1] + seg[g // 2]) / 2.0
        R = lmax / lmed
        out.append((float(lmax), lmed, R, 1.0 if R > tau else 0.0))
    return out


@dataclass
class SagcConfig:
    sizes: tuple = (4, 8, 16)
    tau: float = 1.25
    delta: float = 0.1
    eta: float = 0.5
    gamma: float = 0.95
    seed: int = 0


@dataclass
class SagcState:
    lam: float
    alpha: list
    beta: list
    g_index: int
    step: int = 0
    last_rate: float = 0.0
    last_sample: list = field(default_factory=list)
    last_score: list = field(default_factory=list)


def sagc_init(cfg: SagcConfig) -> SagcState:
    k = len(cfg.sizes)
    w = _words(cfg.seed, (1 << 63, 0, 0, 0))
    g0 = int(u53(w[0]) * k)            # uniform index in [0, k)
    return SagcState(lam=0.0, alpha=[1.0] * k, beta=[1.0] * k, g_index=min(g0, k - 1))


def sagc_choose(cfg: SagcConfig, lam: float, samples, g_index: int) -> tuple[int, list]:
    """Neighbourhood argmax of log2(G) - lam * p~_G; ties to the smaller G."""
    k = len(cfg.sizes)
    scores = [math.log2(cfg.sizes[i]) - lam * samples[i] for i in range(k)]
    best = None
    for i in (g_index - 1, g_index, g_index + 1):     # ascending G
        if 0 <= i < k and (best is None or scores[i] > scores[best]):
            best = i
    return best, scores


def sagc_step(cfg: SagcConfig, st: SagcState, S_values) -> int:
    """One controller step after a rollout with group size sizes[st.g_index]
    whose completed groups had straggler events S_values.  Returns the next G."""
    k = len(cfg.sizes)
    s_bar = sum(float(s) for s in S_values) / len(S_values)
    st.lam = max(0.0, st.lam + cfg.eta * (s_bar - cfg.delta))
    i = st.g_index
    st.alpha[i] = cfg.gamma * st.alpha[i] + s_bar
    st.beta[i] = cfg.gamma * st.beta[i] + (1.0 - s_bar)
    samples = [beta_draw(cfg.seed, st.step, a, st.alpha[a], st.beta[a]) for a in range(k)]
    st.g_index, scores = sagc_choose(cfg, st.lam, samples, i)
    st.step += 1
    st.last_rate = s_bar
    st.last_sample = samples
    st.last_score = scores
    return cfg.sizes[st.g_index]
