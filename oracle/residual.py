"""The fp16 residual of the captioning protocol (Sec. 3.1) -- TEST INFRASTRUCTURE (oracle).

For captioning the paper quantizes keys every 128 tokens, in groups of 32, and keeps values in
a 128-token sliding fp16 window before they are quantized. A decode step at length L therefore
attends over a mixed cache:

  key i    dequantized (Eq. 2, Eq. 4) if i < Kq = 128 * floor(L / 128), else the fp16 key;
  value i  dequantized (Eq. 6)        if i < L - 128,                   else the fp16 value.

Readings (the paper gives the protocol in one sentence):
* R22 -- key blocks of 128 are aligned to token 0 and quantized as four ordinary 32-token
  windows once complete; a window's statistics depend only on its own tokens (R9), so its codes
  equal those of the windowed codec applied at any later time;
* R23 -- "sliding" keeps the last min(L, 128) values in fp16 at every step; a value is quantized
  as it leaves the window, and since value codes are per token the time of quantization does not
  change them;
* R24 -- the fp16 keys and values are the inputs themselves, and the softmax runs over all L
  tokens with both kinds mixed.
"""

from __future__ import annotations

import numpy as np

from .attention import softmax_attention
from .keys import dequantize_keys
from .values import dequantize_values

RESIDUAL = 128


def residual_boundaries(length: int, window: int = RESIDUAL):
    """(Kq, Vq): keys below Kq and values below Vq are read quantized."""
    L = int(length)
    if window <= 0:
        return L, L
    return window * (L // window), max(L - window, 0)


def decode_residual(q16, kc, m, st, nk, vc, nv, modality, k16, v16, length, signs, rot, sm_scale, group,
                    window: int = RESIDUAL):
    """o [G][d] float64 for the G query heads q16 [G][d] of one KV head over the mixed cache.

    kc, m, st, nk, vc, nv, modality: the unpacked quantized cache of the sequence (as for
    ``oracle.attention.decode_bruteforce``); k16, v16 [>= L][d]: its fp16 keys and values."""
    L = int(length)
    d = q16.shape[-1]
    if L == 0:
        return np.zeros((group, d))
    kq, vq = residual_boundaries(L, window)
    khat = np.asarray(k16[:L], np.float64).copy()
    if kq:
        khat[:kq] = dequantize_keys(kc[:kq], m, st, nk[:kq], signs)
    vhat = np.asarray(v16[:L], np.float64).copy()
    if vq:
        vhat[:vq] = dequantize_values(vc[:vq], nv[:vq], modality[:vq], rot)
    return np.stack([softmax_attention(q16[j], khat, vhat, sm_scale) for j in range(group)])


def decode_layer_residual(cache, k16, v16, q16, lens, signs, rot, sm_scale, window: int = RESIDUAL):
    """fp64 outputs [B][Hq][d] of one decode step over a packed cache with the fp16 residual.

    cache: packed buffers (as built by ``oracle.cache.quantize_layer`` or read back from the
    device); k16, v16 [B][H][>= max(lens)][d]: the fp16 keys and values the cache was built from."""
    from .cache import unpacked_fields
    B, Hq, D = q16.shape
    H = cache["k_codes"].shape[1]
    G = Hq // H
    out = np.zeros((B, Hq, D))
    for b in range(B):
        for h in range(H):
            kc, m, st, nk, vc, nv, mod = unpacked_fields(cache, b, h)
            out[b, h * G:(h + 1) * G] = decode_residual(q16[b, h * G:(h + 1) * G], kc, m, st, nk, vc, nv, mod,
                                                        k16[b, h], v16[b, h], lens[b], signs, rot, sm_scale, G,
                                                        window=window)
    return out
