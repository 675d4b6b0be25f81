"""Pins of the MXFP4 key-metadata oracle (E2M1 elements, E8M0 block scales, the key codec on them).

The E2M1 value set and its rounding are fixed by the format definition; the block scale by the
rule that the largest magnitude of a block lands in [4, 8) before rounding; the key codec by the
error bound of a clamped uniform quantizer and by a brute-force nearest-level search.
"""

import os

import numpy as np
import pytest

from oracle.keys import quantize_keys_fmt, quantize_keys_mx_fmt
from oracle.layout import MX_RECORD, cache_bytes_per_token_head, pack_mx_meta, unpack_mx_meta
from oracle.mxfp4 import block_exponent, e2m1_round, e2m1_value, mx_dequantize, mx_quantize
from synth import gen_layer, workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

# FP4 E2M1: codes 0-7 are +0, 0.5, 1, 1.5, 2, 3, 4, 6; codes 8-15 the same with the sign set
E2M1_TABLE = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]


def test_e2m1_value_set():
    vals = e2m1_value(np.arange(16))
    assert np.array_equal(vals[:8], E2M1_TABLE)
    assert np.array_equal(vals[8:], [-x for x in E2M1_TABLE])
    assert np.signbit(vals[8])  # code 8 is -0


@pytest.mark.parametrize("t, code", [
    (0.0, 0), (0.2, 0), (0.25, 0), (0.26, 1), (0.75, 2), (1.25, 2), (1.3, 3), (1.75, 4), (2.5, 4),
    (2.6, 5), (3.5, 6), (4.9, 6), (5.0, 6), (5.1, 7), (6.0, 7), (7.0, 7), (1e9, 7),
    (-0.1, 8), (-0.75, 10), (-5.0, 14), (-100.0, 15)])
def test_e2m1_round_midpoints_and_saturation(t, code):
    """Ties go to the even mantissa (codes 0, 2, 4, 6); beyond 6 the value saturates."""
    assert int(e2m1_round(t)) == code


def test_e2m1_round_error_and_monotone():
    t = np.linspace(-9, 9, 200001)
    c = e2m1_round(t)
    p = e2m1_value(c)
    a = np.abs(t)
    gap = np.where(a < 2, 0.5, np.where(a < 4, 1.0, 2.0))
    assert np.all(np.abs(np.clip(t, -6, 6) - p) <= gap / 2 + 1e-12)
    assert np.all(np.diff(p) >= 0)


def test_block_exponent_brackets_the_block_maximum():
    rng = np.random.default_rng(1)
    v = rng.standard_normal((500, 32)) * np.exp2(rng.integers(-30, 10, (500, 1)))
    e = block_exponent(v)
    amax = np.abs(v).max(1)
    assert np.all(2.0 ** (e + 2) <= amax) and np.all(amax < 2.0 ** (e + 3))
    codes, scale = mx_quantize(v.astype(np.float32))
    top = np.abs(e2m1_value(codes)).max(1)
    assert set(np.unique(top)) <= {4.0, 6.0}
    assert np.array_equal(scale.ravel(), e + 127)


def test_representable_blocks_round_trip():
    rng = np.random.default_rng(2)
    codes = rng.integers(0, 16, (200, 32)).astype(np.uint8)
    codes[:, 0] = rng.choice([6, 7, 14, 15], 200)  # a block maximum of magnitude 4 or 6
    codes[codes == 8] = 0  # -0 and +0 are the same value; keep the canonical +0
    e = rng.integers(-40, 5, 200)
    v = e2m1_value(codes) * np.exp2(e)[:, None]
    c2, s2 = mx_quantize(v.astype(np.float32))
    assert np.array_equal(s2.ravel(), e + 127)
    assert np.array_equal(e2m1_value(c2), e2m1_value(codes))


def test_zero_block_and_relative_error():
    c, s = mx_quantize(np.zeros(64, np.float32))
    assert np.all(c == 0) and np.all(s == 0)
    rng = np.random.default_rng(3)
    v = rng.standard_normal(32 * 100).astype(np.float32)
    c, s = mx_quantize(v)
    d = mx_dequantize(c, s)
    e = s.astype(np.int64) - 127
    # in units of 2^e: error <= half the widest E2M1 gap (1) below 6, < 2 in the saturated range (6, 8)
    bound = np.repeat(np.exp2(e + 1.0), 32)
    assert np.all(np.abs(v - d) <= bound)


def test_mx_record_layout():
    rng = np.random.default_rng(4)
    mc = rng.integers(0, 16, (3, 128)).astype(np.uint8)
    sc = rng.integers(0, 16, (3, 128)).astype(np.uint8)
    ms = rng.integers(0, 255, (3, 4)).astype(np.uint8)
    ss = rng.integers(0, 255, (3, 4)).astype(np.uint8)
    rec = pack_mx_meta(mc, sc, ms, ss)
    assert rec.shape == (3, MX_RECORD)
    # channel 5: channel quad 1, nibble 1 -> byte 4, bits 4..7; its step code -> byte 6, bits 4..7
    assert rec[0, 4] >> 4 == mc[0, 5] and rec[0, 6] >> 4 == sc[0, 5]
    # channel 126: quad 31, nibble 2 -> byte 125, bits 0..3
    assert rec[1, 125] & 15 == mc[1, 126] and rec[1, 127] & 15 == sc[1, 126]
    assert rec[2, 128 + 2 * 3] == ms[2, 3] and rec[2, 129 + 2 * 1] == ss[2, 1]
    back = unpack_mx_meta(rec)
    for x, y in zip(back, (mc, sc, ms, ss)):
        assert np.array_equal(x, y)


def test_mxfp4_bits_per_element_matches_tab3():
    """72.25 bytes per token and KV head over 256 elements: the "Ours (MXFP4 meta.)" row."""
    printed = {}
    for line in open(os.path.join(GOLDEN, "tab3_bits_per_element.txt")):
        if line.strip() and not line.startswith("#"):
            name, val = line.split()
            printed[name] = float(val)
    per_tok = sum(cache_bytes_per_token_head(key_meta="mxfp4").values())
    assert per_tok == 72.25
    assert abs(per_tok * 8 / 256 - printed["ours_mxfp4_meta"]) < 5e-4


@pytest.fixture(scope="module")
def tiny_keys():
    wl = workload("tiny_1k")
    lay = gen_layer(wl, 0)
    return lay["k"][0, 0], lay["signs"]


@pytest.mark.parametrize("length", [1024, 1000, 33, 7])
def test_mx_key_codec_error_bound(tiny_keys, length):
    """|z - zhat| <= max(s / 2, m - lo, hi - (m + 3 s)) for every valid element: the bound of a
    uniform 4-level quantizer with levels m + s c, c = 0..3, clamped at both ends."""
    k, signs = tiny_keys
    r = quantize_keys_mx_fmt(k, length, signs)
    z = r["z"].astype(np.float64)
    n_win = -(-length // 32)
    for g in range(n_win):
        a, b = 32 * g, min(32 * g + 32, length)
        lo, hi = z[a:b].min(0), z[a:b].max(0)
        m, s = r["m"][g].astype(np.float64), r["s"][g].astype(np.float64)
        zh = m + s * r["codes"][a:b]
        bound = np.maximum(np.maximum(s / 2, m - lo), hi - (m + 3 * s))
        assert np.all(np.abs(z[a:b] - zh) <= bound * (1 + 1e-6) + 1e-12)
    assert np.all(r["codes"][length:] == 0) and np.all(r["n16"][length:] == 0)
    assert r["codes"].max() <= 3


def test_mx_key_codes_equal_brute_force_nearest_level(tiny_keys):
    """Away from exact ties the rint formula picks the nearest of the four levels m + s c."""
    k, signs = tiny_keys
    r = quantize_keys_mx_fmt(k, 1024, signs)
    z = r["z"].astype(np.float64)
    g = np.arange(1024) // 32
    m, s = r["m"][g].astype(np.float64), r["s"][g].astype(np.float64)
    levels = m[..., None] + s[..., None] * np.arange(4)
    d = np.abs(z[..., None] - levels)
    best = d.argmin(-1)
    srt = np.sort(d, -1)
    clear = (srt[..., 1] - srt[..., 0] > 1e-6 * np.maximum(s, 1e-30)) & (s > 0)
    assert clear.mean() > 0.99
    assert np.array_equal(r["codes"][clear], best[clear])
    assert np.all(r["codes"][s == 0] == 0)


def test_mx_metadata_is_the_mx_conversion_of_fp32_stats(tiny_keys):
    """The stored records are the MX conversion of the fp32 minimum and step of the fp16 variant,
    and the directions and norms are those of the fp16 variant."""
    k, signs = tiny_keys
    r = quantize_keys_mx_fmt(k, 1000, signs)
    f = quantize_keys_fmt(k, 1000, signs)
    assert np.array_equal(r["n16"].view(np.uint16), f["n16"].view(np.uint16))
    assert np.array_equal(r["z"].view(np.uint32), f["z"].view(np.uint32))
    # fp16(minimum) of the fp16 variant is within half an fp16 ulp of the fp32 minimum; the MX
    # minimum is within the E2M1 error of the same fp32 value
    m32 = f["m16"].astype(np.float64)
    e = r["m_scale"].astype(np.int64) - 127
    assert np.all(np.abs(r["m"] - m32) <= np.repeat(np.exp2(e + 1.0), 32, axis=1) + np.abs(m32) * 2.0 ** -10)
