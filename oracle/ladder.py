"""Bit-width ladder: b-bit keys and values for b = 2, 3, 4 -- TEST INFRASTRUCTURE (oracle).

The paper compares the method with TurboQuant at 2, 3 and 4 bits for both keys and values (the
K2V2 / K3V3 / K4V4 columns of Tab. 5) and quotes TurboQuant K3/V2 next to the method with fp16
metadata at the same 2.625 bits (Tab. 3). The codecs are those of ``oracle.keys``,
``oracle.turboquant`` and ``oracle.values`` with 2^b levels instead of 4:

* keys of the method (Eq. 4): per 32-token window and channel the minimum m and the step
  (max - min) / (2^b - 1) in fp16, code = clamp(rint((z - m16) fl(1 / step16)), 0, 2^b - 1);
* TurboQuant keys (Eq. 2, Eq. 3) and every value (Eq. 6 with the codebook of Eq. 3): the 2^b-level
  Lloyd-Max quantizer of N(0, 1/d), code = #{k : x > tau_k}.

Readings:
* R31 -- the method's b-bit key grid is the uniform (2^b)-level grid on the window range, the
  b-bit form of R1 / R2, with the same fp32 operation order (R17);
* R32 -- the b-bit codebook is the (2^b)-level Lloyd-Max quantizer of N(0, 1/d) with midpoint
  thresholds (R6) and the lower code on a tie (R7);
* R33 -- storage (the paper fixes none): a token's d codes as a little-endian bit stream, channel
  c at bits [b c, b c + b) of the token's d b / 8 bytes, for keys and values alike; the fp16
  window metadata as for 2 bits.

At b = 2 every function here gives the codes of the 2-bit oracle (a test checks it); only the
storage layout differs from the tuned 2-bit one.
"""

from __future__ import annotations

import numpy as np

from .attention import softmax_attention
from .codebook import codebook
from .hadamard import randomized_hadamard
from .keys import F32, WINDOW, f16_sat, key_direction_fmt, norm_tree_f32
from .values import rotate_values_f32_sequential

BITS = (2, 3, 4)


def thresholds_bits_f32(bits: int, d: int = 128) -> np.ndarray:
    """The 2^b - 1 decision thresholds of the b-bit codebook as float32."""
    return codebook(d, bits)[1].astype(F32)


# ---- keys of the method: b-bit uniform grid on each window's range (Eq. 4) ----

def window_stats_bits_fmt(z_valid: np.ndarray, bits: int):
    """(m16, step16) fp16 [d] over the valid tokens [n][d] of one window: step = (hi - lo) / (2^b - 1)."""
    lo = z_valid.min(axis=0).astype(F32) + F32(0.0)
    hi = z_valid.max(axis=0).astype(F32) + F32(0.0)
    step = (hi - lo) / F32(2 ** bits - 1)
    return lo.astype(np.float16), step.astype(np.float16)


def key_codes_bits_fmt(z: np.ndarray, m16: np.ndarray, step16: np.ndarray, bits: int) -> np.ndarray:
    """uint8 codes 0 .. 2^b - 1 of fp32 z [n][d] against one window's fp16 (minimum, step)."""
    m = m16.astype(F32)
    s = step16.astype(F32)
    with np.errstate(divide="ignore", invalid="ignore"):
        inv = F32(1.0) / s
        t = (z - m) * inv
    code = np.clip(np.rint(t), F32(0.0), F32(2 ** bits - 1))
    code = np.where(s == 0, F32(0.0), code)
    return code.astype(np.uint8)


def quantize_keys_bits_fmt(k16: np.ndarray, length: int, signs: np.ndarray, bits: int, window: int = WINDOW):
    """One (sequence, KV head) key block [n][d] -> codes uint8 [n_pad][d], m16 / step16 fp16 [n_win][d],
    n16 fp16 [n_pad], z fp32 [length][d] (n_pad = length rounded up to the window; padded slots
    hold code 0 and norm 0)."""
    length = int(length)
    d = k16.shape[-1]
    n_win = -(-length // window)
    n_pad = n_win * window
    z, n16 = key_direction_fmt(k16[:length], signs)
    codes = np.zeros((n_pad, d), np.uint8)
    m16 = np.zeros((n_win, d), np.float16)
    st16 = np.zeros((n_win, d), np.float16)
    norms = np.zeros(n_pad, np.float16)
    norms[:length] = n16
    for g in range(n_win):
        a, b = g * window, min((g + 1) * window, length)
        m16[g], st16[g] = window_stats_bits_fmt(z[a:b], bits)
        codes[a:b] = key_codes_bits_fmt(z[a:b], m16[g], st16[g], bits)
    return dict(codes=codes, m16=m16, step16=st16, n16=norms, z=z)


# ---- TurboQuant keys and all values: b-bit Lloyd-Max codebook ----

def quantize_keys_tq_bits_fmt(k16: np.ndarray, length: int, signs: np.ndarray, bits: int, window: int = WINDOW):
    """TurboQuant b-bit keys: code = #{k : z_c > tau32_k} on the key direction of the key codec."""
    length = int(length)
    d = k16.shape[-1]
    n_pad = -(-length // window) * window
    z, n16 = key_direction_fmt(k16[:length], signs)
    tau = thresholds_bits_f32(bits, d)
    codes = np.zeros((n_pad, d), np.uint8)
    codes[:length] = (z[:, :, None] > tau[None, None, :]).sum(-1).astype(np.uint8)
    norms = np.zeros(n_pad, np.float16)
    norms[:length] = n16
    return dict(codes=codes, n16=norms, z=z)


def quantize_values_bits_fmt(v16: np.ndarray, modality: np.ndarray, rot: np.ndarray, length: int, bits: int):
    """b-bit values in the exact fp32 order of the value codec: y = R_m v sequentially, code =
    #{k : y_c > fl(n16 tau32_k)} -> dict(codes uint8 [length][d], n16, y, thr)."""
    length = int(length)
    d = v16.shape[-1]
    n16 = f16_sat(norm_tree_f32(v16[:length]))
    y = rotate_values_f32_sequential(v16[:length], np.asarray(modality)[:length], rot)
    thr = n16.astype(F32)[:, None] * thresholds_bits_f32(bits, d)[None, :]
    codes = (y[:, :, None] > thr[:, None, :]).sum(-1).astype(np.uint8)
    return dict(codes=codes, n16=n16, y=y, thr=thr)


# ---- storage: little-endian bit stream per token (R33) ----

def pack_bits(codes: np.ndarray, bits: int) -> np.ndarray:
    """codes uint8 [..., d] (values < 2^b) -> bytes [..., d b / 8]: channel c at bits b c .. b c + b - 1."""
    codes = np.asarray(codes, np.uint8)
    d = codes.shape[-1]
    assert (d * bits) % 8 == 0
    bitplane = ((codes[..., :, None].astype(np.uint16) >> np.arange(bits, dtype=np.uint16)) & 1).astype(np.uint8)
    stream = bitplane.reshape(codes.shape[:-1] + (d * bits,))           # bit b c + j = bit j of code c
    return np.packbits(stream, axis=-1, bitorder="little")


def unpack_bits(packed: np.ndarray, bits: int, d: int = 128) -> np.ndarray:
    """Inverse of ``pack_bits``."""
    stream = np.unpackbits(np.asarray(packed, np.uint8), axis=-1, bitorder="little")[..., :d * bits]
    planes = stream.reshape(stream.shape[:-1] + (d, bits)).astype(np.uint16)
    return (planes << np.arange(bits, dtype=np.uint16)).sum(-1).astype(np.uint8)


def bytes_per_token_head(key_bits: int, value_bits: int, key_meta: str = "fp16", d: int = 128,
                         window: int = WINDOW) -> float:
    """Cache bytes per token and KV head: codes, fp16 norms, fp16 window minimum and step (method)."""
    meta = 2 * 2 * d / window if key_meta == "fp16" else 0.0
    return d * key_bits / 8 + d * value_bits / 8 + 2 + 2 + meta


# ---- a whole layer ----

def quantize_layer_bits(k, v, modality, lens, signs, rot, capacity, key_bits, value_bits, key_meta="fp16"):
    """Packed buffers (numpy) of a layer in the ladder layout: k_codes [B][H][cap][16 kb],
    v_codes [B][H][cap][16 vb], k_norm / v_norm fp16 [B][H][cap], k_min / k_step fp16
    [B][H][cap/32][d] (key_meta "fp16"), modality [B][cap]."""
    B, H, N, D = k.shape
    cap = int(capacity)
    nw = cap // WINDOW
    out = dict(k_codes=np.zeros((B, H, cap, D * key_bits // 8), np.uint8),
               v_codes=np.zeros((B, H, cap, D * value_bits // 8), np.uint8),
               k_norm=np.zeros((B, H, cap), np.float16), v_norm=np.zeros((B, H, cap), np.float16),
               modality=np.zeros((B, cap), np.uint8))
    if key_meta == "fp16":
        out["k_min"] = np.zeros((B, H, nw, D), np.float16)
        out["k_step"] = np.zeros((B, H, nw, D), np.float16)
    elif key_meta != "turboquant":
        raise ValueError(key_meta)
    for b in range(B):
        L = int(lens[b])
        out["modality"][b, :L] = modality[b, :L]
        for h in range(H):
            if key_meta == "fp16":
                kq = quantize_keys_bits_fmt(k[b, h], L, signs, key_bits)
                nwl = kq["codes"].shape[0] // WINDOW
                out["k_min"][b, h, :nwl] = kq["m16"]
                out["k_step"][b, h, :nwl] = kq["step16"]
            else:
                kq = quantize_keys_tq_bits_fmt(k[b, h], L, signs, key_bits)
            npad = kq["codes"].shape[0]
            out["k_codes"][b, h, :npad] = pack_bits(kq["codes"], key_bits)
            out["k_norm"][b, h, :npad] = kq["n16"]
            vq = quantize_values_bits_fmt(v[b, h], modality[b], rot, L, value_bits)
            out["v_codes"][b, h, :L] = pack_bits(vq["codes"], value_bits)
            out["v_norm"][b, h, :L] = vq["n16"]
    return out


def _fields(cache, b, h, L, key_bits, value_bits):
    kc = unpack_bits(cache["k_codes"][b, h, :L], key_bits)
    vc = unpack_bits(cache["v_codes"][b, h, :L], value_bits)
    return kc, vc


def key_directions_bits(cache, b, h, L, key_bits):
    """zhat [L][d] float64: m + step code per window (method), or cb[code] (TurboQuant)."""
    kc = unpack_bits(cache["k_codes"][b, h, :L], key_bits).astype(np.int64)
    if "k_min" in cache:
        g = np.arange(L) // WINDOW
        return cache["k_min"][b, h].astype(np.float64)[g] + cache["k_step"][b, h].astype(np.float64)[g] * kc
    cb, _ = codebook(kc.shape[1], key_bits)
    return cb[kc]


def decode_layer_bits(cache, q16, lens, signs, rot, sm_scale, key_bits, value_bits, rotated=True):
    """fp64 outputs [B][Hq][d] of one decode step over a ladder cache. rotated=False dequantizes every
    key (n16 H^T zhat) and value (n16 R_m^T cb[code]) and runs textbook attention; rotated=True
    scores against H q and applies R_m once per modality after the weighted sum (Sec. 2.3)."""
    B, Hq, D = q16.shape
    H = cache["k_codes"].shape[1]
    G = Hq // H
    hm = randomized_hadamard(signs)
    r = np.asarray(rot, np.float64)
    cbv, _ = codebook(D, value_bits)
    out = np.zeros((B, Hq, D))
    for b in range(B):
        L = int(lens[b])
        if L == 0:
            continue
        mod = np.asarray(cache["modality"][b, :L])
        for h in range(H):
            zhat = key_directions_bits(cache, b, h, L, key_bits)
            nk = cache["k_norm"][b, h, :L].astype(np.float64)
            nv = cache["v_norm"][b, h, :L].astype(np.float64)
            vc = unpack_bits(cache["v_codes"][b, h, :L], value_bits).astype(np.int64)
            vz = nv[:, None] * cbv[vc]
            for j in range(G):
                qj = np.asarray(q16[b, h * G + j], np.float64)
                if not rotated:
                    khat = nk[:, None] * (zhat @ hm)
                    vhat = np.einsum("nij,ni->nj", r[mod], vz)
                    out[b, h * G + j] = softmax_attention(qj, khat, vhat, sm_scale)
                    continue
                s = sm_scale * nk * (zhat @ (hm @ qj))
                p = np.exp(s - s.max())
                o = np.zeros(D)
                for m in range(r.shape[0]):
                    sel = mod == m
                    if sel.any():
                        o += (p[sel] @ vz[sel]) @ r[m]
                out[b, h * G + j] = o / p.sum()
    return out
