"""Pins for oracle.philox: Philox4x64-10 against numpy's implementation."""
import numpy as np
import pytest

from oracle.philox import (MASK64, philox4x64_10, philox4x64_10_np, uniforms,
                           word_to_uniform)


def _numpy_first_block(ctr, key):
    # numpy advances the 256-bit counter by one before producing its first block
    return np.random.Philox(counter=np.array(ctr, dtype=np.uint64),
                            key=np.array(key, dtype=np.uint64)).random_raw(4)


def _inc256(ctr):
    c = list(ctr)
    for i in range(4):
        c[i] = (c[i] + 1) & MASK64
        if c[i] != 0:
            break
    return c


CASES = [
    ((0, 0, 0, 0), (0, 0)),
    ((5, 7, 11, 3), (123, 0)),
    ((MASK64, (1 << 63) + 5, 17, 2), (MASK64 - 2, 9)),
    ((MASK64, MASK64, 3, 4), (0xDEADBEEF, 0xFEEDFACE)),
    ((1234567, 89, 0, 6), (2026, 0)),
]


@pytest.mark.parametrize("ctr,key", CASES)
def test_philox_matches_numpy(ctr, key):
    want = [int(x) for x in _numpy_first_block(ctr, key)]
    got = list(philox4x64_10(_inc256(ctr), key))
    assert got == want


def test_vectorised_equals_scalar():
    rng = np.random.default_rng(1)
    c = rng.integers(0, 2**63, size=(4, 50), dtype=np.uint64)
    c[0, :3] = np.uint64(MASK64)
    got = philox4x64_10_np(c[0], c[1], c[2], c[3], 77, 5)
    for i in range(50):
        want = philox4x64_10([int(c[j, i]) for j in range(4)], (77, 5))
        assert [int(g[i]) for g in got] == list(want)


def test_uniform_grid():
    words = np.array([0, 1, (1 << 41) - 1, 1 << 41, MASK64, MASK64 - (1 << 41)], dtype=np.uint64)
    u = word_to_uniform(words)
    assert np.all(u > 0) and np.all(u < 1)
    assert u[0] == 2.0 ** -24 and u[4] == 1 - 2.0 ** -24
    assert np.all(u.astype(np.float32).astype(np.float64) == u)   # exact in float32
    U = uniforms(3, np.arange(1000), 2, 5, 3)
    assert U.shape == (1000, 4)
    assert abs(U.mean() - 0.5) < 0.02
