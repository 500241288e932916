"""Exact Gumbel-max sampling of one token, with forced-length EOS handling.

Sampling from softmax(z/T) is done by the Gumbel-max identity: argmax_v of
z_v/T + g_v with g_v i.i.d. standard Gumbel is distributed as softmax(z/T).
The argmax is an integer decided by floating point, so it is taken in fp32
(the precision the kernel uses): score_v = fp32(fp32(z_v) / T) + g_v.  Ties go to
the lowest id.

Forced lengths (the synthetic stand-in for a policy's natural EOS): while
t < L_s - 1 the EOS score is -inf; at t = L_s - 1 the token is EOS regardless of
the scores.  Without a forced length EOS is an ordinary token.

The reported log-probability is that of the emitted token under the full,
unmasked distribution: z_y/T - logsumexp(z/T), in float64.
"""
from __future__ import annotations

import math

import numpy as np

from .philox import gumbel_noise


def logsumexp(a: np.ndarray) -> float:
    m = float(np.max(a))
    return m + math.log(float(np.sum(np.exp(a - m))))


def sample_token(z: np.ndarray, seed: int, t: int, s: int, eos_id: int,
                 temperature: float = 1.0, forced_len=None):
    """Returns (token, logprob, margin).  ``margin`` is the gap between the best
    and second-best fp32 score (inf where the token was forced)."""
    z = np.asarray(z, np.float64)
    zt = z / float(temperature)
    lse = logsumexp(zt)
    if forced_len is not None and t == int(forced_len) - 1:
        y, margin = eos_id, math.inf
    else:
        zs = (z.astype(np.float32) / np.float32(temperature)).astype(np.float32)
        score = zs + gumbel_noise(seed, t, s, len(z))
        if forced_len is not None:
            score[eos_id] = -np.inf
        y = int(np.argmax(score))
        rest = np.delete(score, y)
        margin = float(score[y]) - float(np.max(rest)) if len(rest) else math.inf
    return y, float(zt[y] - lse), margin
