"""TurboQuant codec for keys (Sec. 2.1, Eq. 2 and Eq. 3) -- TEST INFRASTRUCTURE (oracle).

The paper's baseline quantizes every cached key and value the same way: the direction u = x / ||x||
is rotated by the randomized Hadamard transform, z = H u (Eq. 2), each coordinate takes the nearest
entry of the fixed Gaussian codebook, r_c = argmin_l |z_c - cb_l|, and xhat = ||x|| H^T cb[r]
(Eq. 3). Its values are this package's value codec with R_m = H for every modality (the single
global rotation); its keys are coded here.

Readings:
* R29 -- the key direction z and the fp16 norm are those of the key codec (the FMT order of
  ``oracle.keys.key_direction_fmt``: halving-tree norm, fp32 butterflies, z = w * fl(kappa / n16));
  the codebook is the Lloyd-Max quantizer of N(0, 1/d) with midpoint thresholds (R6), and a
  coordinate exactly on a threshold takes the lower code (R7): code = #{k : z_c > tau32_k};
* R30 -- the codes use the key byte layout (token-major, 32 bytes per token), and a cache of
  TurboQuant keys stores no window metadata: 68 bytes per token per KV head with the values,
  Tab. 3's 2.125 bits per element.
"""

from __future__ import annotations

import numpy as np

from .attention import softmax_attention
from .codebook import codebook, thresholds_f32
from .hadamard import randomized_hadamard
from .keys import WINDOW, key_direction_fmt
from .values import dequantize_values

F32 = np.float32


def quantize_keys_tq_fmt(k16: np.ndarray, length: int, signs: np.ndarray, window: int = WINDOW):
    """TurboQuant key codes of one (sequence, KV head) block [n][d] -> dict(codes uint8 [n_pad][d],
    n16 fp16 [n_pad], z fp32 [length][d]); slots beyond ``length`` (up to the next multiple of the
    window, as the cache stores whole windows) hold code 0 and norm 0."""
    length = int(length)
    d = k16.shape[-1]
    n_pad = -(-length // window) * window
    z, n16 = key_direction_fmt(k16[:length], signs)
    tau = thresholds_f32(d)
    codes = np.zeros((n_pad, d), np.uint8)
    codes[:length] = (z[:, :, None] > tau[None, None, :]).sum(-1).astype(np.uint8)
    norms = np.zeros(n_pad, np.float16)
    norms[:length] = n16
    return dict(codes=codes, n16=norms, z=z)


def dequantize_keys_tq(codes: np.ndarray, n16: np.ndarray, signs: np.ndarray) -> np.ndarray:
    """khat [n][d] float64 = n16 H^T cb[code] (Eq. 3)."""
    cb, _ = codebook(codes.shape[1])
    hm = randomized_hadamard(signs)
    return n16.astype(np.float64)[:, None] * (cb[codes.astype(np.int64)] @ hm)


def decode_tq_bruteforce(q16, kc, nk, vc, nv, modality, length, signs, rot, sm_scale, group):
    """o [G][d] float64 over a cache with TurboQuant keys: dequantize every key and value and run
    textbook softmax attention (Eq. 1)."""
    L = int(length)
    if L == 0:
        return np.zeros((group, q16.shape[-1]))
    khat = dequantize_keys_tq(kc[:L], nk[:L], signs)
    vhat = dequantize_values(vc[:L], nv[:L], modality[:L], rot)
    return np.stack([softmax_attention(q16[j], khat, vhat, sm_scale) for j in range(group)])


def decode_tq_rotated(q16, kc, nk, vc, nv, modality, length, signs, rot, sm_scale, group):
    """The same in the rotated space (the fused kernel's order): q' = H q once per head,
    s_i = n16_i (q' . cb[code_i]) sm_scale; values as in ``oracle.attention.decode_rotated``."""
    L = int(length)
    if L == 0:
        return np.zeros((group, q16.shape[-1]))
    hm = randomized_hadamard(signs)
    cb, _ = codebook(kc.shape[1])
    zk = cb[kc[:L].astype(np.int64)]
    nkf = nk[:L].astype(np.float64)
    vz = nv[:L].astype(np.float64)[:, None] * cb[vc[:L].astype(np.int64)]
    mod = np.asarray(modality)[:L]
    r = np.asarray(rot, np.float64)
    out = []
    for j in range(group):
        s = sm_scale * nkf * (zk @ (hm @ np.asarray(q16[j], np.float64)))
        p = np.exp(s - s.max())
        o = np.zeros(kc.shape[1])
        for m in range(r.shape[0]):
            sel = mod == m
            if sel.any():
                o += (p[sel] @ vz[sel]) @ r[m]
        out.append(o / p.sum())
    return np.stack(out)
