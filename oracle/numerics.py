"""Small numeric helpers for the oracle: bf16 rounding emulation, fp32 rounding.

ORACLE / TEST INFRASTRUCTURE (see oracle/__init__.py).
"""
from __future__ import annotations

import numpy as np


def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value (ties to even), as float64.

    bfloat16 keeps 8 significant bits. With x = m * 2^e, 0.5 <= |m| < 1
    (frexp), the rounded value is rint(m * 2^8) * 2^(e - 8); numpy's rint
    rounds halves to even. Values here stay far from the bf16 overflow and
    subnormal ranges.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(m * 256.0), e - 8)


def f32(x) -> np.ndarray:
    """Round to float32 and return as float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def log_softmax(z: np.ndarray, axis: int = -1) -> np.ndarray:
    zmax = np.max(z, axis=axis, keepdims=True)
    s = z - zmax
    return s - np.log(np.sum(np.exp(s), axis=axis, keepdims=True))


def logsumexp(z: np.ndarray, axis: int = -1) -> np.ndarray:
    zmax = np.max(z, axis=axis, keepdims=True)
    return np.squeeze(zmax, axis) + np.log(np.sum(np.exp(z - zmax), axis=axis))
