"""Seeded stochastic drafting: t~ drawn from p_theta by Gumbel-max.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 3.3 writes the draft as a sample t~ ~ p_theta(. | h_k); the default path reads it as
the argmax (greedy drafting).  This module defines the sampled variant:

  t~ = argmax_v ( z_v / tau + g_v ),   g_v = -log(-log(u_v))

which draws t~ from softmax(z / tau) (the Gumbel-max property).  The uniforms u_v come from
the counter-based generator Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
numbers: as easy as 1, 2, 3", SC 2011), written here from its published definition:

  * state: four 64-bit counter words c0..c3 and two 64-bit key words k0, k1;
  * one round: (hi0, lo0) = M0 * c0 and (hi1, lo1) = M1 * c2 as 128-bit products, then
    c = (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0);
  * ten rounds, the key advanced by the Weyl increments (W0, W1) before each round after
    the first.

Counter layout of one draft: c0 = v // 4 (output word v % 4), c1 = row = sequence * 16 +
draft index j, c2 = decode step (0 for the first step after the prefill), c3 = 0; key =
(seed, 0).  u = (2 * (x >> 41) + 1) / 2^24 lies strictly inside (0, 1).

Pins (tests/test_oracle_sampling.py): the generator equals numpy's Philox bit generator (which
advances its counter before each block) on several counters and keys; sampled tokens follow
softmax(z / tau) (chi-square); the DVI rollout stays lossless with sampled drafts.
"""
from __future__ import annotations

import numpy as np

M0, M1 = 0xD2E7470EE14C6C93, 0xCA5A826395121157
W0, W1 = 0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B
ROW_STRIDE = 16
_MASK32 = np.uint64(0xFFFFFFFF)


def _mulhilo(a: np.ndarray, m: int):
    """128-bit product of uint64 array a and constant m: (hi, lo) uint64 arrays."""
    m_lo, m_hi = np.uint64(m & 0xFFFFFFFF), np.uint64(m >> 32)
    a_lo, a_hi = a & _MASK32, a >> np.uint64(32)
    ll = a_lo * m_lo
    hl = a_hi * m_lo
    lh = a_lo * m_hi
    hh = a_hi * m_hi
    mid = (ll >> np.uint64(32)) + (hl & _MASK32) + (lh & _MASK32)
    hi = hh + (hl >> np.uint64(32)) + (lh >> np.uint64(32)) + (mid >> np.uint64(32))
    lo = a * np.uint64(m)  # wraps modulo 2^64
    return hi, lo


def philox4x64(c0, c1, c2, c3, k0: int, k1: int):
    """Philox4x64-10 on counter words (uint64 arrays, broadcast together) and a key: 4 arrays."""
    with np.errstate(over="ignore"):
        c = [np.asarray(x, dtype=np.uint64) for x in np.broadcast_arrays(c0, c1, c2, c3)]
        key0, key1 = np.uint64(k0), np.uint64(k1)
        for r in range(10):
            if r:
                key0 = np.uint64((int(key0) + W0) & 0xFFFFFFFFFFFFFFFF)
                key1 = np.uint64((int(key1) + W1) & 0xFFFFFFFFFFFFFFFF)
            hi0, lo0 = _mulhilo(c[0], M0)
            hi1, lo1 = _mulhilo(c[2], M1)
            c = [hi1 ^ c[1] ^ key0, lo1, hi0 ^ c[3] ^ key1, lo0]
    return c


def uniforms(V: int, seed: int, step, row: int) -> np.ndarray:
    """u_v for v in 0..V-1 (float64, exact dyadic values in (0, 1)); step may be an array
    (then the result is [len(step), V])."""
    step = np.atleast_1d(np.asarray(step, dtype=np.uint64))
    blocks = np.arange((V + 3) // 4, dtype=np.uint64)
    x = philox4x64(blocks[None, :], np.uint64(row), step[:, None], np.uint64(0), seed, 0)
    words = np.stack(x, axis=-1).reshape(step.size, -1)[:, :V]       # [steps, V], v = 4*block + k
    u = ((words >> np.uint64(41)).astype(np.float64) * 2.0 + 1.0) / float(1 << 24)
    return u


def gumbel(V: int, seed: int, step, row: int) -> np.ndarray:
    u = uniforms(V, seed, step, row)
    return -np.log(-np.log(u))


def sample_scores(z, tau: float, seed: int, step: int, row: int) -> np.ndarray:
    """z / tau + g for one draft (float64 [V])."""
    z = np.asarray(z, dtype=np.float64).reshape(-1)
    return z / tau + gumbel(z.size, seed, step, row)[0]
