"""Philox4x64-10 counter-based generator (Salmon, Moraes, Dror, Shaw, SC'11,
"Parallel random numbers: as easy as 1, 2, 3").

ORACLE / TEST INFRASTRUCTURE. The sampler's randomness (the uniforms of
Algorithm 1 and of the acceptance-rejection loop of Theorem 1, the categorical
and Gaussian draws of the naive AR sampler of §4.2) is indexed by a counter so
that the CPU oracle and the GPU path can draw the same numbers independently.
This is the published generator, written here from its definition; the GPU
side carries its own implementation.

Counter words: (c0, c1, c2, c3) = (sequence, round-or-event, slot, tag).
Key words:     (k0, k1) = (seed, 0).
Each block yields four 64-bit words; a word x becomes the uniform
u = (2 * (x >> 41) + 1) * 2^-24, an odd multiple of 2^-24 in (0, 1), exact
in float32 and float64.
"""
from __future__ import annotations

import numpy as np

MASK64 = (1 << 64) - 1
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
PHILOX_W0 = 0x9E3779B97F4A7C15
PHILOX_W1 = 0xBB67AE8584CAA73B

# counter tags (fourth counter word)
TAG_AR = 1
TAG_DRAFT = 2
TAG_ACCEPT = 3
TAG_RES_T = 4
TAG_RES_K = 5
TAG_BONUS = 6


def philox4x64_10(ctr, key):
    """One Philox4x64 block with 10 rounds on Python ints."""
    x0, x1, x2, x3 = (int(c) & MASK64 for c in ctr)
    k0, k1 = (int(k) & MASK64 for k in key)
    for r in range(10):
        if r > 0:
            k0 = (k0 + PHILOX_W0) & MASK64
            k1 = (k1 + PHILOX_W1) & MASK64
        p0 = PHILOX_M0 * x0
        p1 = PHILOX_M1 * x2
        hi0, lo0 = p0 >> 64, p0 & MASK64
        hi1, lo1 = p1 >> 64, p1 & MASK64
        x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
    return x0, x1, x2, x3


def _mulhilo(a: np.ndarray, m: int):
    """64x64 -> 128-bit product of uint64 array a with constant m, as (hi, lo)."""
    a = a.astype(np.uint64)
    mask32 = np.uint64(0xFFFFFFFF)
    a_lo, a_hi = a & mask32, a >> np.uint64(32)
    m_lo, m_hi = np.uint64(m & 0xFFFFFFFF), np.uint64(m >> 32)
    ll = a_lo * m_lo
    lh = a_lo * m_hi
    hl = a_hi * m_lo
    hh = a_hi * m_hi
    mid = (ll >> np.uint64(32)) + (lh & mask32) + (hl & mask32)
    lo = (ll & mask32) | ((mid & mask32) << np.uint64(32))
    hi = hh + (lh >> np.uint64(32)) + (hl >> np.uint64(32)) + (mid >> np.uint64(32))
    return hi, lo


def philox4x64_10_np(c0, c1, c2, c3, k0: int, k1: int = 0):
    """Vectorised Philox4x64-10 over broadcastable uint64 counter arrays."""
    shape = np.broadcast(np.asarray(c0), np.asarray(c1), np.asarray(c2), np.asarray(c3)).shape
    x0 = np.broadcast_to(np.asarray(c0, dtype=np.uint64), shape).copy()
    x1 = np.broadcast_to(np.asarray(c1, dtype=np.uint64), shape).copy()
    x2 = np.broadcast_to(np.asarray(c2, dtype=np.uint64), shape).copy()
    x3 = np.broadcast_to(np.asarray(c3, dtype=np.uint64), shape).copy()
    kk0, kk1 = k0 & MASK64, k1 & MASK64
    with np.errstate(over="ignore"):
        for r in range(10):
            if r > 0:
                kk0 = (kk0 + PHILOX_W0) & MASK64
                kk1 = (kk1 + PHILOX_W1) & MASK64
            hi0, lo0 = _mulhilo(x0, PHILOX_M0)
            hi1, lo1 = _mulhilo(x2, PHILOX_M1)
            x0, x1, x2, x3 = hi1 ^ x1 ^ np.uint64(kk0), lo1, hi0 ^ x3 ^ np.uint64(kk1), lo0
    return x0, x1, x2, x3


def word_to_uniform(x) -> np.ndarray:
    """Top 23 bits of a 64-bit word -> odd multiple of 2^-24 in (0, 1)."""
    top = (np.asarray(x, dtype=np.uint64) >> np.uint64(41)).astype(np.float64)
    return (2.0 * top + 1.0) * 2.0 ** -24


def uniforms(seed: int, seq, c1, c2, tag: int) -> np.ndarray:
    """Four uniforms per counter (seq, c1, c2, tag); returns array [..., 4] float64."""
    words = philox4x64_10_np(seq, c1, c2, np.uint64(tag), seed, 0)
    return np.stack([word_to_uniform(w) for w in words], axis=-1)
