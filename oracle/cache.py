"""Whole-layer quantization into the packed cache buffers, and decode over them.

Builds exactly the byte contents the GPU library writes for a layer
([B][Hkv] sequences of keys and values, a modality map, per-sequence lengths),
from the FMT codecs of ``keys`` and ``values`` and the pack maps of ``layout``.
Slots beyond a sequence's length are zero. Appending a sequence in chunks must
give the same bytes as this one-shot quantization of the concatenation
(reading of the cache reuse of Sec. 2.1 and the streaming protocol of Sec. 3.1).
"""

from __future__ import annotations

import numpy as np

from .attention import decode_bruteforce, decode_dense, decode_rotated
from .keys import quantize_keys_fmt, quantize_keys_mx_fmt
from .layout import MX_RECORD, WINDOW, pack_keys, pack_mx_meta, pack_values, unpack_keys, unpack_mx_meta, unpack_values
from .mxfp4 import mx_dequantize
from .values import quantize_values_fmt


def quantize_layer(k, v, modality, lens, signs, rot, capacity=None, key_meta="fp16"):
    """Dict of packed buffers (numpy) for k, v [B][H][N][d] fp16, modality [B][N], lens [B].

    key_meta "fp16": fp16 window minimum and step (k_min, k_step); "mxfp4": one 136-byte MXFP4
    record per window (k_mx, layout in ``oracle.layout``); "turboquant": TurboQuant keys (Gaussian
    codebook after the Hadamard rotation, no window metadata; ``oracle.turboquant``).
    """
    B, H, N, D = k.shape
    cap = int(capacity or -(-N // WINDOW) * WINDOW)
    nw = cap // WINDOW
    out = dict(
        k_codes=np.zeros((B, H, cap, D // 4), np.uint8),
        v_codes=np.zeros((B, H, nw, 1024), np.uint8),
        k_norm=np.zeros((B, H, cap), np.float16),
        v_norm=np.zeros((B, H, cap), np.float16),
        modality=np.zeros((B, cap), np.uint8),
    )
    if key_meta == "fp16":
        out["k_min"] = np.zeros((B, H, nw, D), np.float16)
        out["k_step"] = np.zeros((B, H, nw, D), np.float16)
    elif key_meta == "mxfp4":
        out["k_mx"] = np.zeros((B, H, nw, MX_RECORD), np.uint8)
    elif key_meta != "turboquant":
        raise ValueError(key_meta)
    for b in range(B):
        L = int(lens[b])
        out["modality"][b, :L] = modality[b, :L]
        for h in range(H):
            if key_meta == "fp16":
                kq = quantize_keys_fmt(k[b, h], L, signs)
                nwl = kq["codes"].shape[0] // WINDOW
                out["k_min"][b, h, :nwl] = kq["m16"]
                out["k_step"][b, h, :nwl] = kq["step16"]
            elif key_meta == "turboquant":
                from .turboquant import quantize_keys_tq_fmt
                kq = quantize_keys_tq_fmt(k[b, h], L, signs)
            else:
                kq = quantize_keys_mx_fmt(k[b, h], L, signs)
                nwl = kq["codes"].shape[0] // WINDOW
                out["k_mx"][b, h, :nwl] = pack_mx_meta(kq["m_codes"], kq["s_codes"], kq["m_scale"], kq["s_scale"])
            npad = kq["codes"].shape[0]
            out["k_codes"][b, h, :npad] = pack_keys(kq["codes"])
            out["k_norm"][b, h, :npad] = kq["n16"]
            vq = quantize_values_fmt(v[b, h], modality[b], rot, L)
            vcodes = np.zeros((npad, D), np.uint8)
            vcodes[:L] = vq["codes"]
            out["v_codes"][b, h, :npad // WINDOW] = pack_values(vcodes)
            out["v_norm"][b, h, :L] = vq["n16"]
    return out


def key_metadata(cache, b, h):
    """(minimum, step) [n_win][d] of one sequence and KV head: the fp16 fields, or the MXFP4
    records dequantized (float32, exact)."""
    if "k_mx" in cache:
        mc, sc, ms, ss = unpack_mx_meta(cache["k_mx"][b, h])
        return mx_dequantize(mc, ms).astype(np.float32), mx_dequantize(sc, ss).astype(np.float32)
    return cache["k_min"][b, h], cache["k_step"][b, h]


def unpacked_fields(cache, b, h):
    """(kc, m, st, nk, vc, nv, modality) for one sequence and KV head of a packed cache."""
    m, st = key_metadata(cache, b, h)
    return (unpack_keys(cache["k_codes"][b, h]), m, st, cache["k_norm"][b, h],
            unpack_values(cache["v_codes"][b, h]), cache["v_norm"][b, h], cache["modality"][b])


def decode_layer(cache, q16, lens, signs, rot, sm_scale, rotated=True, heads=None):
    """fp64 outputs [B][Hq][d] of one decode step over a packed cache (TurboQuant keys when the
    cache holds neither window metadata field).

    ``heads`` optionally restricts the work to a list of (b, kv head) pairs; other rows are NaN.
    """
    B, Hq, D = q16.shape
    H = cache["k_codes"].shape[1]
    G = Hq // H
    out = np.full((B, Hq, D), np.nan)
    fn = decode_rotated if rotated else decode_bruteforce
    tq = "k_min" not in cache and "k_mx" not in cache
    if tq:
        from .turboquant import decode_tq_bruteforce, decode_tq_rotated
        ftq = decode_tq_rotated if rotated else decode_tq_bruteforce
    for b in range(B):
        for h in range(H):
            if heads is not None and (b, h) not in heads:
                continue
            if tq:
                out[b, h * G:(h + 1) * G] = ftq(q16[b, h * G:(h + 1) * G], unpack_keys(cache["k_codes"][b, h]),
                                                cache["k_norm"][b, h], unpack_values(cache["v_codes"][b, h]),
                                                cache["v_norm"][b, h], cache["modality"][b], lens[b], signs, rot,
                                                sm_scale, G)
                continue
            kc, m16, st16, nk, vc, nv, mod = unpacked_fields(cache, b, h)
            out[b, h * G:(h + 1) * G] = fn(q16[b, h * G:(h + 1) * G], kc, m16, st16, nk, vc, nv, mod,
                                           lens[b], signs, rot, sm_scale, G)
    return out


def decode_layer_dense(k16, v16, q16, lens, sm_scale):
    B, Hq, D = q16.shape
    H = k16.shape[1]
    G = Hq // H
    out = np.zeros((B, Hq, D))
    for b in range(B):
        for h in range(H):
            out[b, h * G:(h + 1) * G] = decode_dense(q16[b, h * G:(h + 1) * G], k16[b, h], v16[b, h],
                                                     lens[b], sm_scale, G)
    return out
