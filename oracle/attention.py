"""Decode attention over the quantized cache (Eq. 1), in float64.

Attention for one query per head: alpha = softmax(q K^T / sqrt(d)), o = alpha V
(Eq. 1). During decoding the cached keys and values are the dequantized ones.

Two formulations are given, which agree in exact arithmetic:

* ``decode_bruteforce`` -- dequantize every key (n16 * H^T zhat) and every value
  (n16 * R_m^T cb[code]) and run textbook softmax attention;
* ``decode_rotated`` -- what the fused kernel computes (Sec. 2.3): rotate the
  query once per head (q' = H q) and score against the rotated-space key
  directions, s_i = n16_i * (q' . zhat_i) / sqrt(d); keep one value accumulator
  per modality in the rotated space, acc_m = sum_{i in m} p_i n16_i cb[code_i],
  and apply the inverse rotation once per modality after aggregation,
  o = sum_m R_m^T acc_m / sum_i p_i.

GQA reading (R11): query head j reads KV head j // G with G = Hq / Hkv.
An empty cache (length 0) has no softmax; its output is defined as zeros.
"""

from __future__ import annotations

import numpy as np

from .codebook import codebook
from .hadamard import randomized_hadamard
from .keys import dequantize_directions, dequantize_keys
from .values import dequantize_values


def softmax_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, sm_scale: float) -> np.ndarray:
    """Textbook attention for one query q [d] over k, v [n][d], float64 (max subtracted)."""
    s = sm_scale * (np.asarray(k, np.float64) @ np.asarray(q, np.float64))
    p = np.exp(s - s.max())
    return (p @ np.asarray(v, np.float64)) / p.sum()


def decode_bruteforce(q16, kc, m16, st16, nk, vc, nv, modality, length, signs, rot, sm_scale, group):
    """o [G][d] for the G query heads q16 [G][d] sharing one KV head (unpacked cache fields)."""
    L = int(length)
    if L == 0:
        return np.zeros((group, q16.shape[-1]))
    khat = dequantize_keys(kc[:L], m16, st16, nk[:L], signs)
    vhat = dequantize_values(vc[:L], nv[:L], modality[:L], rot)
    return np.stack([softmax_attention(q16[j], khat, vhat, sm_scale) for j in range(group)])


def decode_rotated(q16, kc, m16, st16, nk, vc, nv, modality, length, signs, rot, sm_scale, group):
    """Same as ``decode_bruteforce`` in the rotated-space order of the fused kernel."""
    L = int(length)
    if L == 0:
        return np.zeros((group, q16.shape[-1]))
    hm = randomized_hadamard(signs)
    cb, _ = codebook(kc.shape[1])
    zhat = dequantize_directions(kc[:L], m16, st16)
    nkf = nk[:L].astype(np.float64)
    nvf = nv[:L].astype(np.float64)
    mod = np.asarray(modality)[:L]
    vz = nvf[:, None] * cb[vc[:L].astype(np.int64)]
    r = np.asarray(rot, np.float64)
    out = []
    for j in range(group):
        qr = hm @ np.asarray(q16[j], np.float64)
        s = sm_scale * nkf * (zhat @ qr)
        p = np.exp(s - s.max())
        o = np.zeros(kc.shape[1])
        for m in range(r.shape[0]):
            sel = mod == m
            if sel.any():
                o += (p[sel] @ vz[sel]) @ r[m]
        out.append(o / p.sum())
    return np.stack(out)


def decode_dense(q16, k16, v16, length, sm_scale, group):
    """Unquantized fp16 cache: o [G][d] (the dense baseline's reference)."""
    L = int(length)
    if L == 0:
        return np.zeros((group, q16.shape[-1]))
    return np.stack([softmax_attention(q16[j], k16[:L], v16[:L], sm_scale) for j in range(group)])
