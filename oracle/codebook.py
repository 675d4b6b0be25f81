"""Fixed Gaussian codebook (Sec. 2.1, Eq. 3).

After the randomized Hadamard rotation each coordinate of a unit vector is
approximately N(0, 1/d); the fixed codebook is built from that reference
distribution. Reading taken here: the 2^b-level Lloyd-Max (minimum mean squared
error) quantizer of N(0, 1/d), i.e. the N(0, 1) Lloyd-Max levels scaled by
1/sqrt(d). The decision thresholds are the midpoints between adjacent levels,
which is what ``argmin_l |z - cb_l|`` of Eq. 3 selects.

The Lloyd iteration alternates the two optimality conditions: every level is
the centroid of its cell (closed form for a Gaussian: (phi(a) - phi(b)) /
(Phi(b) - Phi(a))), and every threshold is the midpoint of its neighbours.
"""

from __future__ import annotations

import math

import numpy as np


def _phi(x: float) -> float:
    return 0.0 if math.isinf(x) else math.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)


def _cdf(x: float) -> float:
    if math.isinf(x):
        return 0.0 if x < 0 else 1.0
    return 0.5 * math.erfc(-x / math.sqrt(2.0))


def lloyd_max_gaussian(levels: int = 4, tol: float = 1e-15, max_iter: int = 100000):
    """Lloyd-Max levels and thresholds for N(0, 1), float64, ascending."""
    c = [(-(levels - 1) / 2.0 + i) for i in range(levels)]
    for _ in range(max_iter):
        t = [(c[i] + c[i + 1]) / 2.0 for i in range(levels - 1)]
        edges = [-math.inf] + t + [math.inf]
        new = [(_phi(edges[i]) - _phi(edges[i + 1])) / (_cdf(edges[i + 1]) - _cdf(edges[i]))
               for i in range(levels)]
        delta = max(abs(a - b) for a, b in zip(new, c))
        c = new
        if delta < tol:
            break
    # enforce the exact symmetry of the Gaussian
    c = [(c[i] - c[levels - 1 - i]) / 2.0 for i in range(levels)]
    t = [(c[i] + c[i + 1]) / 2.0 for i in range(levels - 1)]
    return np.array(c), np.array(t)


def codebook(d: int = 128, bits: int = 2):
    """(cb, tau): levels and thresholds of the Lloyd-Max quantizer of N(0, 1/d), float64."""
    c, t = lloyd_max_gaussian(2 ** bits)
    s = 1.0 / math.sqrt(d)
    return c * s, t * s


def thresholds_f32(d: int = 128) -> np.ndarray:
    """Thresholds as float32 (the precision the value-code decision is taken in)."""
    return codebook(d)[1].astype(np.float32)


def mse_closed_form(c: np.ndarray, t: np.ndarray) -> float:
    """E[(X - Q(X))^2] for X ~ N(0, 1) and the quantizer (c, t), by the Gaussian moment formulas."""
    edges = [-math.inf] + list(t) + [math.inf]
    total = 0.0
    for i, ci in enumerate(c):
        a, b = edges[i], edges[i + 1]
        p = _cdf(b) - _cdf(a)
        m1 = _phi(a) - _phi(b)
        # int x^2 phi = p + a phi(a) - b phi(b)
        m2 = p + (0.0 if math.isinf(a) else a * _phi(a)) - (0.0 if math.isinf(b) else b * _phi(b))
        total += m2 - 2 * ci * m1 + ci * ci * p
    return total
