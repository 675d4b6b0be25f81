"""Key codec: norm split, randomized Hadamard, per-window range adaptation (Eq. 2, Eq. 4).

What is computed for each key k (a head_dim-vector, fp16):

1. norm  n = ||k||_2, stored as fp16 ``n16`` (Eq. 2 separates magnitude and direction);
2. direction z = H k / n16 (Eq. 2; the Hadamard basis is kept for keys, Sec. 2.3);
3. for every group g of W = 32 consecutive tokens and every coordinate c, the
   minimum m_gc and the range of z over the group (Eq. 4, temporal range
   adaptation); the normalized coordinate (z - m)/range lies in [0, 1];
4. the fixed codebook applied to the normalized coordinate.

Readings (the paper is silent or ambiguous on these):

* R1 -- the "fixed codebook" applied to the normalized key coordinate is the
  uniform 4-level grid {0, 1/3, 2/3, 1} on [0, 1] (asymmetric 2-bit integer
  quantization), because Eq. 4's normalized coordinate lives in [0, 1];
* R2 -- the stored scale is the step range/3 (fp16) next to the fp16 minimum;
* R4 -- the direction is normalized by the stored fp16 norm, so n16 * H^T zhat
  reconstructs without a norm-rounding error;
* R5 -- H = Had diag(s) / sqrt(d) with the signs acting first;
* R7 -- codes round half to even; fp16 conversions round to nearest even;
* R8 -- a zero-range group codes everything 0; a zero norm gives z = 0;
  -0 is canonicalized to +0 in the stored minimum and step; norms beyond
  the fp16 range saturate to 65504;
* R9 -- a partial last group takes its statistics over its valid tokens only.

FMT operation order (bit-exact contract with the GPU):

  t_c   = x_c * x_c                                   (exact in fp32)
  sum   = halving tree: t <- t[:n/2] + t[n/2:] until one value
  n32   = sqrt_rn(sum);  n16 = fp16_rne_saturating(n32)
  w     = fwht_f32(s * x)                              (butterflies h = 1 .. 64)
  cinv  = fl(KAPPA / n16), KAPPA = fp32(1/sqrt(128))
  z     = fl(w * cinv)                                 (z = 0 when n16 == 0)
  lo    = min z + 0.0f,  hi = max z + 0.0f             (over the group's valid tokens)
  step  = fl(fl(hi - lo) / 3.0f);  m16 = fp16(lo);  step16 = fp16(step)
  code  = 0 if step16 == 0 else clamp(rint(fl(fl(z - m16) * fl(1.0f / step16))), 0, 3)
"""

from __future__ import annotations

import numpy as np

from .hadamard import fwht_f32, randomized_hadamard

F32 = np.float32
KAPPA32 = np.float32(1.0 / np.sqrt(np.float64(128.0)))
WINDOW = 32
LEVELS = 3  # 2-bit: codes 0..3, step = range / 3


def f16_sat(x32: np.ndarray) -> np.ndarray:
    """fp32 -> fp16, round to nearest even, saturating at +-65504 instead of overflowing to inf."""
    x32 = np.asarray(x32, F32)
    with np.errstate(over="ignore"):
        r = x32.astype(np.float16)
    return np.where(np.isinf(r), np.copysign(np.float16(65504.0), x32).astype(np.float16), r)


def norm_tree_f32(x16: np.ndarray) -> np.ndarray:
    """fp32 Euclidean norm of fp16 rows by the halving tree (last axis must be a power of two)."""
    t = np.asarray(x16).astype(F32)
    t = t * t
    n = t.shape[-1]
    while n > 1:
        n //= 2
        t = t[..., :n] + t[..., n:2 * n]
    return np.sqrt(t[..., 0])


def key_direction_fmt(x16: np.ndarray, signs: np.ndarray):
    """(z fp32 [..., d], n16 fp16 [...]) for fp16 keys [..., d]."""
    x16 = np.asarray(x16, np.float16)
    n16 = f16_sat(norm_tree_f32(x16))
    w = fwht_f32(x16.astype(F32) * np.asarray(signs, F32))
    n16f = n16.astype(F32)
    with np.errstate(divide="ignore", invalid="ignore"):
        cinv = KAPPA32 / n16f
        z = w * cinv[..., None]
    z = np.where((n16f == 0)[..., None], F32(0.0), z).astype(F32)
    return z, n16


def window_stats_fmt(z_valid: np.ndarray):
    """(m16, step16) fp16 [d] for the valid tokens [n][d] of one window (n >= 1)."""
    lo = z_valid.min(axis=0).astype(F32) + F32(0.0)
    hi = z_valid.max(axis=0).astype(F32) + F32(0.0)
    step = (hi - lo) / F32(LEVELS)
    return lo.astype(np.float16), step.astype(np.float16)


def key_codes_fmt(z: np.ndarray, m16: np.ndarray, step16: np.ndarray) -> np.ndarray:
    """uint8 codes 0..3 for fp32 z [n][d] against one window's (m16, step16) [d] (fp16, or the
    fp32 dequantized MXFP4 metadata)."""
    m = m16.astype(F32)
    s = step16.astype(F32)
    with np.errstate(divide="ignore"):
        inv = F32(1.0) / s
    t = (z - m) * inv
    code = np.clip(np.rint(t), F32(0.0), F32(LEVELS))
    code = np.where(s == 0, F32(0.0), code)
    return code.astype(np.uint8)


def quantize_keys_fmt(k16: np.ndarray, length: int, signs: np.ndarray, window: int = WINDOW):
    """Quantize one (sequence, KV head) key block [n][d] -> dict of unpacked cache fields.

    Returns codes uint8 [n_pad][d] (n_pad = length rounded up to the window; slots beyond
    ``length`` hold code 0), m16 / step16 fp16 [n_win][d], n16 fp16 [n_pad] (0 beyond length),
    and the fp32 directions z [length][d].
    """
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
        m16[g], st16[g] = window_stats_fmt(z[a:b])
        codes[a:b] = key_codes_fmt(z[a:b], m16[g], st16[g])
    return dict(codes=codes, m16=m16, step16=st16, n16=norms, z=z)


def quantize_keys_mx_fmt(k16: np.ndarray, length: int, signs: np.ndarray, window: int = WINDOW):
    """The key codec with MXFP4 window metadata (readings R18-R21 of ``oracle.mxfp4``).

    Per window: lo = min z + 0, hi = max z + 0, step = fl(fl(hi - lo) / 3) in fp32 as in the fp16
    variant; the 128-vectors lo and step are stored as MXFP4 (4 blocks of 32 channels each) and
    the codes are taken against their dequantized values m, s (fp32, exact).
    Returns codes [n_pad][d], m_codes / s_codes uint8 [n_win][d], m_scale / s_scale uint8
    [n_win][d / 32], m / s fp32 [n_win][d] (dequantized), n16 [n_pad], z [length][d].
    """
    from .mxfp4 import mx_dequantize, mx_quantize

    length = int(length)
    d = k16.shape[-1]
    n_win = -(-length // window)
    n_pad = n_win * window
    z, n16 = key_direction_fmt(k16[:length], signs)
    codes = np.zeros((n_pad, d), np.uint8)
    out = {f: np.zeros((n_win, d), np.uint8) for f in ("m_codes", "s_codes")}
    out.update({f: np.zeros((n_win, d // 32), np.uint8) for f in ("m_scale", "s_scale")})
    out.update({f: np.zeros((n_win, d), F32) for f in ("m", "s")})
    norms = np.zeros(n_pad, np.float16)
    norms[:length] = n16
    for g in range(n_win):
        a, b = g * window, min((g + 1) * window, length)
        lo = z[a:b].min(axis=0).astype(F32) + F32(0.0)
        hi = z[a:b].max(axis=0).astype(F32) + F32(0.0)
        step = (hi - lo) / F32(LEVELS)
        out["m_codes"][g], out["m_scale"][g] = mx_quantize(lo)
        out["s_codes"][g], out["s_scale"][g] = mx_quantize(step)
        out["m"][g] = mx_dequantize(out["m_codes"][g], out["m_scale"][g]).astype(F32)
        out["s"][g] = mx_dequantize(out["s_codes"][g], out["s_scale"][g]).astype(F32)
        codes[a:b] = key_codes_fmt(z[a:b], out["m"][g], out["s"][g])
    return dict(codes=codes, n16=norms, z=z, **out)


def quantize_keys_f64(k16: np.ndarray, length: int, signs: np.ndarray, window: int = WINDOW):
    """The F64 reading of Eq. 2 + Eq. 4: exact range, exact step, round half to even.

    z = H k / n16 in float64 (n16 the fp16 norm, reading R4); per window and channel
    lo = min z, hi = max z, step = (hi - lo) / 3, code = clamp(round((z - lo) / step), 0, 3).
    """
    length = int(length)
    k = np.asarray(k16[:length], np.float64)
    n16 = f16_sat(np.sqrt((k * k).sum(-1)).astype(F32)).astype(np.float64)
    hm = randomized_hadamard(signs)
    with np.errstate(divide="ignore", invalid="ignore"):
        z = (k @ hm.T) / n16[:, None]
    z = np.where((n16 == 0)[:, None], 0.0, z)
    n_win = -(-length // window)
    lo = np.zeros((n_win, k.shape[1]))
    step = np.zeros_like(lo)
    codes = np.zeros(z.shape, np.uint8)
    for g in range(n_win):
        a, b = g * window, min((g + 1) * window, length)
        lo[g] = z[a:b].min(0)
        step[g] = (z[a:b].max(0) - lo[g]) / LEVELS
        with np.errstate(divide="ignore", invalid="ignore"):
            t = (z[a:b] - lo[g]) / step[g]
        codes[a:b] = np.where(step[g] == 0, 0, np.clip(np.rint(t), 0, LEVELS)).astype(np.uint8)
    return dict(z=z, lo=lo, step=step, codes=codes, n16=n16)


def dequantize_directions(codes: np.ndarray, m16: np.ndarray, step16: np.ndarray, window: int = WINDOW):
    """zhat [n][d] float64 = m16 + step16 * code, per token's window (Eq. 4 inverted)."""
    n = codes.shape[0]
    g = np.arange(n) // window
    return m16.astype(np.float64)[g] + step16.astype(np.float64)[g] * codes.astype(np.float64)


def dequantize_keys(codes, m16, step16, n16, signs, window: int = WINDOW):
    """khat [n][d] float64 = n16 * H^T zhat (Eq. 3 reconstruction with the Eq. 4 range restored)."""
    zhat = dequantize_directions(codes, m16, step16, window)
    hm = randomized_hadamard(signs)
    return n16.astype(np.float64)[:, None] * (zhat @ hm)
