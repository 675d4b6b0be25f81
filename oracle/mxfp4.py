"""MXFP4 storage of the key window metadata -- TEST INFRASTRUCTURE (oracle).

The paper stores the per-group key minimum m_gc and scale s_gc of Eq. 4 with MXFP4
metadata by default (Sec. 3.1, implementation details; Tab. 3 row "Ours (MXFP4 meta.)",
2.258 bits per element). MXFP4 is the OCP Microscaling format with FP4 elements: a block of
32 values shares one 8-bit power-of-two scale (E8M0, exponent bias 127) and each value is a
4-bit E2M1 float (sign bit, 2 exponent bits with bias 1, 1 mantissa bit, no inf or nan).

Conversion of a block V (the published MX definition, written out):
  e    = floor(log2(max_i |V_i|)) - 2      (2 = the largest E2M1 exponent, 6 = 1.5 * 2^2),
         clamped to the E8M0 range [-127, 127]; stored as the byte e + 127
  P_i  = the E2M1 value nearest to V_i / 2^e, ties to the even mantissa, saturating at +-6
  V_i ~ P_i * 2^e

Readings (the paper says only "MXFP4 metadata"):
* R18 -- a block is 32 consecutive channels of one window's minimum vector (or of its step
  vector): 4 blocks per window and field, so a window's metadata is final when the window is;
* R19 -- an all-zero block gets e = -127 and zero elements; a negative value that rounds to
  zero keeps its sign (code 8, -0);
* R20 -- the key codes are computed against the dequantized minimum and step (what a reader
  of the cache reconstructs), with the FMT order of the fp16 variant: code = 0 if step == 0,
  else clamp(rint(fl(fl(z - m) * fl(1 / step))), 0, 3);
* R21 -- the quantity stored is the step (max - min) / 3 in fp32, as in the fp16 variant.

Everything here is a plain statement of the definition: the E2M1 value set is built from its
bit fields and rounding is a brute-force nearest-value search.
"""

from __future__ import annotations

import numpy as np

BLOCK = 32
E8M0_BIAS = 127
E2M1_EMAX = 2


def e2m1_value(code) -> np.ndarray:
    """float64 value of 4-bit E2M1 codes: sign bit 3, exponent bits 2..1 (bias 1), mantissa bit 0.

    Exponent field 0 is subnormal: 0.M * 2^0; otherwise 1.M * 2^(E - 1).
    """
    code = np.asarray(code, np.int64)
    sign = np.where(code & 8, -1.0, 1.0)
    E = (code >> 1) & 3
    M = code & 1
    mag = np.where(E == 0, 0.5 * M, (1.0 + 0.5 * M) * np.exp2(E - 1.0))
    return sign * mag


MAGNITUDES = e2m1_value(np.arange(8))  # codes 0..7: the non-negative values


def e2m1_round(t) -> np.ndarray:
    """uint8 E2M1 codes of float values t: nearest magnitude (ties to the even mantissa, i.e. the
    even code), saturating at 6 (the nearest finite value beyond it); sign bit = t < 0."""
    t = np.asarray(t, np.float64)
    a = np.abs(t)
    dist = np.abs(a[..., None] - MAGNITUDES)                 # [..., 8]
    best = dist.min(axis=-1, keepdims=True)
    cand = dist == best                                     # one or two nearest codes
    even = cand & ((np.arange(8) & 1) == 0)
    pick = np.where(even.any(axis=-1), np.argmax(even, axis=-1), np.argmax(cand, axis=-1))
    return (pick + np.where(t < 0, 8, 0)).astype(np.uint8)


def block_exponent(v32: np.ndarray) -> np.ndarray:
    """Shared exponent e (int) of each block along the last axis (length 32)."""
    amax = np.abs(np.asarray(v32, np.float64)).max(axis=-1)
    _, ex = np.frexp(amax)  # amax = f * 2^ex with f in [0.5, 1): floor(log2(amax)) = ex - 1
    e = np.where(amax > 0, ex - 1 - E2M1_EMAX, -E8M0_BIAS)
    return np.clip(e, -E8M0_BIAS, E8M0_BIAS).astype(np.int64)


def mx_quantize(v: np.ndarray):
    """(codes uint8 [..., n], scale bytes uint8 [..., n / 32]) of fp32 values, blocks of 32 along
    the last axis."""
    v = np.asarray(v, np.float32).astype(np.float64)
    blocks = v.reshape(v.shape[:-1] + (v.shape[-1] // BLOCK, BLOCK))
    e = block_exponent(blocks)
    t = blocks * np.exp2(-e.astype(np.float64))[..., None]   # exact: a power-of-two scaling
    codes = e2m1_round(t).reshape(v.shape)
    return codes, (e + E8M0_BIAS).astype(np.uint8)


def mx_dequantize(codes: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """float64 values P * 2^(X - 127) (exact in float32 as well: at most two significant bits)."""
    codes = np.asarray(codes)
    n = codes.shape[-1]
    vals = e2m1_value(codes).reshape(codes.shape[:-1] + (n // BLOCK, BLOCK))
    e = np.asarray(scale, np.int64) - E8M0_BIAS
    return (vals * np.exp2(e.astype(np.float64))[..., None]).reshape(codes.shape)
