"""Philox4x64-10 counter-based generator and the Gumbel noise drawn from it.

Philox4x64 follows Salmon, Moraes, Dror and Shaw, "Parallel Random Numbers:
As Easy as 1, 2, 3" (SC'11): a 4-word counter and a 2-word key; each round
multiplies counter words 0 and 2 by two fixed odd constants, takes the 128-bit
products' halves, and XORs the high halves with the other two counter words and
the key; the key is advanced by two Weyl increments between rounds; ten rounds.

Stream layout used for sampling (a reading, fixed here and in the library
header): key = (seed, TAG_GUMBEL), counter = (v >> 3, t, s, 0) for vocabulary
id v, decode step t and sequence id s; the block's four 64-bit words give eight
32-bit values, value j = v & 7 being the (j & 1)-th 32-bit half (low half first)
of word j >> 1.  The 32-bit value x becomes u = (2*(x >> 9) + 1) * 2**-24, an
fp32 number strictly inside (0, 1), and the Gumbel variate is -log(-log(u))
evaluated in fp32.
"""
from __future__ import annotations

import numpy as np

PHILOX_M0 = np.uint64(0xD2E7470EE14C6C93)
PHILOX_M1 = np.uint64(0xCA5A826395121157)
PHILOX_W0 = np.uint64(0x9E3779B97F4A7C15)   # golden ratio
PHILOX_W1 = np.uint64(0xBB67AE8584CAA73B)   # sqrt(3) - 1
TAG_GUMBEL = 1

_M32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo64(a: np.ndarray, b: np.uint64):
    """(hi, lo) 64-bit halves of the 128-bit product a*b, via 32-bit limbs."""
    a = a.astype(np.uint64)
    a0, a1 = a & _M32, a >> _S32
    b0, b1 = b & _M32, b >> _S32
    p00, p01, p10, p11 = a0 * b0, a0 * b1, a1 * b0, a1 * b1
    mid = (p00 >> _S32) + (p01 & _M32) + (p10 & _M32)
    hi = p11 + (p01 >> _S32) + (p10 >> _S32) + (mid >> _S32)
    lo = a * b  # wraps modulo 2**64
    return hi, lo


def philox4x64_10(ctr: np.ndarray, key) -> np.ndarray:
    """Apply Philox4x64-10 to counters ``ctr`` (uint64 [..., 4]) under
    ``key = (k0, k1)``; returns uint64 [..., 4]."""
    c = np.asarray(ctr, dtype=np.uint64)
    c0, c1, c2, c3 = (c[..., i].copy() for i in range(4))
    k0, k1 = np.uint64(key[0]), np.uint64(key[1])
    with np.errstate(over="ignore"):
        for r in range(10):
            if r > 0:
                k0 = np.uint64(k0 + PHILOX_W0)
                k1 = np.uint64(k1 + PHILOX_W1)
            hi0, lo0 = _mulhilo64(c0, PHILOX_M0)
            hi1, lo1 = _mulhilo64(c2, PHILOX_M1)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1)


def gumbel_uniform_bits(seed: int, t: int, s: int, vocab: int) -> np.ndarray:
    """uint32 [vocab]: the 32-bit value drawn for every vocabulary id at decode
    step t of sequence s."""
    nb = (vocab + 7) // 8
    ctr = np.zeros((nb, 4), np.uint64)
    ctr[:, 0] = np.arange(nb, dtype=np.uint64)
    ctr[:, 1] = np.uint64(t)
    ctr[:, 2] = np.uint64(s)
    w = philox4x64_10(ctr, (seed, TAG_GUMBEL))            # [nb, 4]
    halves = np.empty((nb, 8), np.uint64)
    halves[:, 0::2] = w & _M32                             # low half first
    halves[:, 1::2] = w >> _S32
    return halves.reshape(-1)[:vocab].astype(np.uint32)


def uniforms_from_bits(x: np.ndarray) -> np.ndarray:
    """fp32 uniforms (2*(x>>9)+1) * 2**-24: 2**23 equally spaced odd multiples
    of 2**-24, exact in fp32, never 0 or 1."""
    k = (np.asarray(x, np.uint32) >> np.uint32(9)).astype(np.float64)
    return ((2.0 * k + 1.0) * 2.0 ** -24).astype(np.float32)


def gumbel_noise(seed: int, t: int, s, vocab: int) -> np.ndarray:
    """fp32 [vocab] standard Gumbel variates g = -log(-log(u)), in fp32, for
    sequence s at decode step t; an array of sequence ids gives
    [len(s), vocab], row i for sequence s[i]."""
    if np.ndim(s) == 0:
        u = uniforms_from_bits(gumbel_uniform_bits(seed, t, int(s), vocab))
    else:
        u = uniforms_from_bits(gumbel_uniform_bits_batch(seed, t, s, vocab))
    return -np.log(-np.log(u))


def gumbel_uniform_bits_batch(seed: int, t: int, s: np.ndarray, vocab: int) -> np.ndarray:
    """uint32 [len(s), vocab]: ``gumbel_uniform_bits`` for many sequence ids at
    once (same layout, vectorised over s)."""
    s = np.asarray(s, np.uint64)
    nb = (vocab + 7) // 8
    ctr = np.zeros((len(s), nb, 4), np.uint64)
    ctr[:, :, 0] = np.arange(nb, dtype=np.uint64)[None, :]
    ctr[:, :, 1] = np.uint64(t)
    ctr[:, :, 2] = s[:, None]
    w = philox4x64_10(ctr, (seed, TAG_GUMBEL))
    halves = np.empty((len(s), nb, 8), np.uint64)
    halves[:, :, 0::2] = w & _M32
    halves[:, :, 1::2] = w >> _S32
    return halves.reshape(len(s), -1)[:, :vocab].astype(np.uint32)
