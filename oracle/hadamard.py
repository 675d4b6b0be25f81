"""Randomized Hadamard transform (Sec. 2.1, Eq. 2).

Reading: H = (1/sqrt(d)) * Had_d * diag(s), with Had_d the Sylvester Hadamard
matrix (Had_1 = [1], Had_2n = [[Had_n, Had_n], [Had_n, -Had_n]]) in natural
order and s a given +-1 vector. The signs act first; H is orthogonal, so
H^T = diag(s) Had_d / sqrt(d) (Had_d is symmetric).

``fwht_f32`` is the documented fp32 operation order for the unnormalized
transform Had_d (s * x): in-place butterflies for h = 1, 2, 4, ..., d/2, each
replacing (w_j, w_{j+h}) by (w_j + w_{j+h}, w_j - w_{j+h}) for every j with
(j & h) == 0, each add and subtract rounded to fp32.
"""

from __future__ import annotations

import numpy as np


def sylvester(d: int) -> np.ndarray:
    """Sylvester Hadamard matrix of order d (a power of two), float64."""
    assert d >= 1 and d & (d - 1) == 0
    h = np.ones((1, 1))
    while h.shape[0] < d:
        h = np.block([[h, h], [h, -h]])
    return h


def randomized_hadamard(signs: np.ndarray) -> np.ndarray:
    """H = Had diag(s) / sqrt(d), float64 [d][d]."""
    s = np.asarray(signs, np.float64)
    d = s.shape[0]
    return sylvester(d) * s[None, :] / np.sqrt(d)


def fwht_f32(w: np.ndarray) -> np.ndarray:
    """Unnormalized Walsh-Hadamard transform along the last axis, fp32 butterflies, h ascending."""
    w = np.array(w, dtype=np.float32, copy=True)
    d = w.shape[-1]
    h = 1
    while h < d:
        v = w.reshape(w.shape[:-1] + (d // (2 * h), 2, h))
        a = v[..., 0, :].copy()
        b = v[..., 1, :].copy()
        v[..., 0, :] = a + b
        v[..., 1, :] = a - b
        w = v.reshape(w.shape)
        h *= 2
    return w


def fwht_f64(w: np.ndarray) -> np.ndarray:
    """The same butterflies in float64 (exact for small integers)."""
    w = np.array(w, dtype=np.float64, copy=True)
    d = w.shape[-1]
    h = 1
    while h < d:
        v = w.reshape(w.shape[:-1] + (d // (2 * h), 2, h))
        a = v[..., 0, :].copy()
        b = v[..., 1, :].copy()
        v[..., 0, :] = a + b
        v[..., 1, :] = a - b
        w = v.reshape(w.shape)
        h *= 2
    return w
