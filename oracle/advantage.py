"""Group-relative advantage (Sec. 3.1: each prompt's G completions are scored
against the group's mean/standardized reward; Sec. 4 requirement (iii)).

A_i = (r_i - mean(r)) / (std(r) + eps) within each group, mean and std in
float64, result rounded to float32.  Readings: eps is added to the standard
deviation (not to the variance); std uses ``ddof`` (default 1, Bessel); a group
whose rewards are all equal, or whose size does not exceed ddof, has A = 0.
"""
from __future__ import annotations

import math

import numpy as np


def group_advantage(rewards, G, eps: float = 1e-6, ddof: int = 1) -> np.ndarray:
    r_all = np.asarray(rewards, np.float64)
    G = np.asarray(G, np.int64)
    out = np.zeros(len(r_all), np.float32)
    o = 0
    for g in G:
        g = int(g)
        r = r_all[o:o + g]
        if g - ddof > 0 and not np.all(r == r[0]):
            mu = sum(float(v) for v in r) / g
            var = sum((float(v) - mu) ** 2 for v in r) / (g - ddof)
            sigma = math.sqrt(var)
            out[o:o + g] = np.array([(float(v) - mu) / (sigma + eps) for v in r], np.float32)
        o += g
    return out


def zero_variance_filter(rewards, G):
    """Which groups carry a learning signal.  Sec. 2 cites DAPO's dynamic
    sampling, used again in Sec. 5.1: a group whose rewards are all equal has
    A = 0 for every member, so the trainer drops it and draws more prompts.

    keep[p] = 1 when some reward of group p differs (IEEE float32 comparison)
    from the group's first one, else 0; kept_ids = the p with keep[p] = 1,
    ascending.  Raises ValueError unless every G[p] >= 1 and sum(G) == len(rewards).
    """
    r_all = np.asarray(rewards, np.float32)
    G = [int(g) for g in G]
    if any(g < 1 for g in G) or sum(G) != len(r_all):
        raise ValueError("group sizes do not partition the rewards")
    keep = np.zeros(len(G), np.int32)
    o = 0
    for p, g in enumerate(G):
        first = r_all[o]
        keep[p] = int(any(r_all[o + i] != first for i in range(1, g)))
        o += g
    return keep, np.flatnonzero(keep).astype(np.int32)
