"""Sampling at the controlled temperature (oracle, float64).

Test infrastructure: see the package docstring.
"""
from __future__ import annotations

import numpy as np


def _cdf(z: np.ndarray, temp: float):
    y = np.asarray(z, dtype=np.float64) / float(temp)
    e = np.exp(y - np.max(y))
    return e, np.cumsum(e)


def sample(z: np.ndarray, temp: float, u: float):
    """Token drawn from p = softmax(z / T) by inverse CDF at the uniform u
    (Sections 2.1 and 3.3: the next token is sampled at the controlled
    temperature).

    Reading: full-vocabulary inverse CDF in index order with one uniform per
    row, x = min{j : C_j > u S} with C the running sum of exp(y_j - max y) and
    S its total; if rounding leaves no such j, the last token of positive
    mass.  Also returns the margin r = min(|C_{x-1} - uS|, |C_x - uS|) / S,
    the relative distance of uS to the edges of x's CDF interval.

    Returns (token, margin)."""
    e, C = _cdf(z, temp)
    S = C[-1]
    target = float(u) * S
    x = int(np.searchsorted(C, target, side="right"))
    if x >= len(C):
        x = int(np.nonzero(e > 0)[0][-1])
    lo = C[x - 1] if x > 0 else 0.0
    margin = min(abs(lo - target), abs(C[x] - target)) / S
    return x, float(margin)


def cdf_interval(z: np.ndarray, temp: float, x: int):
    """(C_{x-1}/S, C_x/S): the CDF interval of token x (for validity checks)."""
    e, C = _cdf(z, temp)
    S = C[-1]
    lo = C[x - 1] if x > 0 else 0.0
    return lo / S, C[x] / S


def sample_many(z: np.ndarray, temp: float, us: np.ndarray) -> np.ndarray:
    """`sample` for many uniforms of one row (same rule, vectorised)."""
    e, C = _cdf(z, temp)
    S = C[-1]
    x = np.searchsorted(C, np.asarray(us, dtype=np.float64) * S, side="right")
    last = int(np.nonzero(e > 0)[0][-1])
    return np.where(x >= len(C), last, x)
