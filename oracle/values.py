"""Value codec with modality-aware rotation (Eq. 6 with the codebook of Eq. 3).

For a value v of a token of modality m (audio 0, video 1, text 2):

  u = v / ||v||,   z = R_m u,   r_c = argmin_l |z_c - cb_l|,   vhat = ||v|| R_m^T cb[r]

R_m is the calibrated rotation H U_m^T of Eq. 6; here it is an input (one
[3][d][d] fp32 table per layer, shared by the heads -- reading R13).

Readings:

* R6  -- cb is the Lloyd-Max codebook of N(0, 1/d); thresholds are midpoints;
* R7  -- a coordinate exactly on a threshold takes the lower code (the first
  index of argmin);
* R14 -- the decision compares y = R_m v with fl(n16 * tau_k) instead of
  dividing y by the norm: y_c > n16 tau_k  <=>  z_c > tau_k in exact arithmetic;
* R8  -- a zero vector gives y = 0 and thresholds n16 * tau = 0 (signed zeros
  compare equal), so every code is 0; it reconstructs as 0 because the stored
  norm is 0.

FMT "exact mode" order (bit-exact contract with the GPU's sequential mode):

  n16   = fp16(sqrt_rn(halving-tree sum of x_c^2))           (as for keys)
  y_c   = acc, acc = 0; for j = 0..d-1: acc = fl(acc + fl(R_cj * x_j))
  T_k   = fl(n16 * tau32_k)
  code  = #{k : y_c > T_k}
"""

from __future__ import annotations

import numpy as np

from .codebook import codebook, thresholds_f32
from .keys import f16_sat, norm_tree_f32

F32 = np.float32


def rotate_values_f32_sequential(v16: np.ndarray, modality: np.ndarray, rot: np.ndarray) -> np.ndarray:
    """y [n][d] fp32 = R_{m_i} v_i with a sequential fp32 dot product (j ascending, no fusion)."""
    x = np.asarray(v16, np.float16).astype(F32)
    rot = np.asarray(rot, F32)
    y = np.zeros(x.shape, F32)
    for m in range(rot.shape[0]):
        sel = np.nonzero(modality == m)[0]
        if len(sel) == 0:
            continue
        xm = x[sel]
        acc = np.zeros(xm.shape, F32)
        rm = rot[m]
        for j in range(x.shape[1]):
            acc = acc + xm[:, j:j + 1] * rm[None, :, j]
        y[sel] = acc
    return y


def quantize_values_fmt(v16: np.ndarray, modality: np.ndarray, rot: np.ndarray, length: int):
    """Exact-mode value quantization of [n][d] fp16 values -> dict(codes uint8, n16 fp16, y fp32, thr fp32)."""
    length = int(length)
    d = v16.shape[-1]
    n16 = f16_sat(norm_tree_f32(v16[:length]))
    y = rotate_values_f32_sequential(v16[:length], np.asarray(modality)[:length], rot)
    tau = thresholds_f32(d)
    thr = n16.astype(F32)[:, None] * tau[None, :]          # [n][3]
    codes = ((y[:, :, None] > thr[:, None, :]).sum(-1)).astype(np.uint8)
    return dict(codes=codes, n16=n16, y=y, thr=thr)


def quantize_values_f64(v16: np.ndarray, modality: np.ndarray, rot: np.ndarray, length: int):
    """F64 reading of Eq. 6: z = R_m v / n16, code = argmin_l |z - cb_l| (first index on ties)."""
    length = int(length)
    x = np.asarray(v16[:length], np.float64)
    mod = np.asarray(modality)[:length]
    r = np.asarray(rot, np.float64)
    n16 = f16_sat(np.sqrt((x * x).sum(-1)).astype(F32)).astype(np.float64)
    y = np.einsum("nij,nj->ni", r[mod], x)
    with np.errstate(divide="ignore", invalid="ignore"):
        z = np.where((n16 == 0)[:, None], 0.0, y / n16[:, None])
    cb, _ = codebook(x.shape[1])
    codes = np.argmin(np.abs(z[:, :, None] - cb[None, None, :]), axis=-1).astype(np.uint8)
    return dict(codes=codes, n16=n16, y=y, z=z)


def dequantize_values(codes: np.ndarray, n16: np.ndarray, modality: np.ndarray, rot: np.ndarray) -> np.ndarray:
    """vhat [n][d] float64 = n16 * R_m^T cb[code] (Eq. 6)."""
    cb, _ = codebook(codes.shape[1])
    zhat = cb[codes.astype(np.int64)]
    r = np.asarray(rot, np.float64)
    mod = np.asarray(modality)[:codes.shape[0]]
    return n16.astype(np.float64)[:, None] * np.einsum("nij,ni->nj", r[mod], zhat)


def rotation_error_bound(v16: np.ndarray, modality: np.ndarray, rot: np.ndarray, rel: float = 2.0 ** -16):
    """Per-element band eps = rel * sum_j |R_cj v_j| used to judge codes whose y lies near a threshold."""
    x = np.abs(np.asarray(v16, np.float64))
    r = np.abs(np.asarray(rot, np.float64))
    mod = np.asarray(modality)[:x.shape[0]]
    return rel * np.einsum("nij,nj->ni", r[mod], x)
