"""Pins of the bit-width ladder oracle (oracle.ladder: b-bit keys and values, b = 2, 3, 4).

* the 8- and 16-level codebooks against Max's published tables (tests/golden);
* at b = 2 every codec gives the codes of the pinned 2-bit oracle;
* the method's b-bit key codes: brute-force nearest grid point away from ties, both end codes
  used in every window, the error bound step / 2 in float64, idempotence of re-quantizing the
  dequantized directions;
* Lloyd-Max codes (TurboQuant keys, values) equal a brute-force nearest level away from ties;
* the bit-stream layout on hand-worked bytes (a 3-bit code straddling a byte) and round trips;
* Tab. 3's 2.625 bits of TurboQuant K3/V2 from the layout's bytes;
* decode: the rotated-space order equals textbook attention over dequantized keys and values,
  and at b = 2 the ladder decode equals the 2-bit cache's decode.
"""

import math
import os

import numpy as np
import pytest

from oracle.cache import decode_layer, quantize_layer
from oracle.codebook import codebook, lloyd_max_gaussian, mse_closed_form
from oracle.keys import quantize_keys_fmt
from oracle.ladder import (BITS, bytes_per_token_head, decode_layer_bits, key_directions_bits, pack_bits,
                           quantize_keys_bits_fmt, quantize_keys_tq_bits_fmt, quantize_layer_bits,
                           quantize_values_bits_fmt, unpack_bits)
from oracle.turboquant import quantize_keys_tq_fmt
from oracle.values import quantize_values_fmt
from synth import gen_layer, gen_queries, workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "lloyd_max_gaussian_8_16level.txt")
SM = 1 / math.sqrt(128)


def _golden():
    rows = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        k, *vals = line.split()
        rows[k] = np.array([float(x) for x in vals])
    return rows


@pytest.mark.parametrize("levels", [8, 16])
def test_codebook_matches_max_tables(levels):
    g = _golden()
    c, t = lloyd_max_gaussian(levels)

    def printed_tol(x):  # half a unit of the 4th significant digit, plus the table's own 1e-4
        mag = np.floor(np.log10(np.maximum(np.abs(x), 1e-3)))
        return 0.5 * 10.0 ** (mag - 3) + 1e-4

    for ours, ref in ((c[levels // 2:], g[f"levels_{levels}"]), (t[levels // 2 - 1:], g[f"thresholds_{levels}"])):
        assert np.all(np.abs(ours - ref) <= printed_tol(ref)), (ours, ref)
    assert abs(mse_closed_form(c, t) - g[f"mse_{levels}"][0]) <= 1e-3 * g[f"mse_{levels}"][0]


def _layer(L=200, layer=1):
    wl = workload("tiny_1k")
    lay = gen_layer(wl, layer, lengths=np.array([L], np.int32), n_tokens=L)
    return wl, lay


def test_two_bits_reduce_to_the_two_bit_oracle():
    wl, lay = _layer(171)
    k, v = lay["k"][0, 0], lay["v"][0, 0]
    a = quantize_keys_bits_fmt(k, 171, lay["signs"], 2)
    b = quantize_keys_fmt(k, 171, lay["signs"])
    for n in ("codes", "m16", "step16", "n16"):
        np.testing.assert_array_equal(a[n].view(np.uint8), b[n].view(np.uint8))
    np.testing.assert_array_equal(quantize_keys_tq_bits_fmt(k, 171, lay["signs"], 2)["codes"],
                                  quantize_keys_tq_fmt(k, 171, lay["signs"])["codes"])
    np.testing.assert_array_equal(quantize_values_bits_fmt(v, lay["modality"][0], lay["rot"], 171, 2)["codes"],
                                  quantize_values_fmt(v, lay["modality"][0], lay["rot"], 171)["codes"])


@pytest.mark.parametrize("bits", [3, 4])
def test_method_key_codes_brute_force_and_bounds(bits):
    wl, lay = _layer(150)
    kq = quantize_keys_bits_fmt(lay["k"][0, 0], 150, lay["signs"], bits)
    z, codes = kq["z"].astype(np.float64), kq["codes"][:150].astype(np.int64)
    top = 2 ** bits - 1
    assert codes.max() == top and codes.min() == 0
    for g in range(kq["m16"].shape[0]):
        a, b = 32 * g, min(32 * g + 32, 150)
        m, s = kq["m16"][g].astype(np.float64), kq["step16"][g].astype(np.float64)
        grid = m[None, :, None] + s[None, :, None] * np.arange(top + 1)[None, None, :]
        dist = np.abs(z[a:b, :, None] - grid)
        best = dist.argmin(-1)
        second = np.sort(dist, axis=-1)[..., 1]
        clear = (second - dist.min(-1)) > 1e-5 * np.maximum(s[None, :], 1e-30)
        live = (s > 0)[None, :] & clear
        np.testing.assert_array_equal(codes[a:b][live], best[live])
        # every channel's window uses code 0 at its minimum and the top code at its maximum
        nz = s > 0
        assert np.all(codes[a:b][z[a:b].argmin(0)[nz], np.nonzero(nz)[0]] == 0)
        assert np.all(codes[a:b][z[a:b].argmax(0)[nz], np.nonzero(nz)[0]] == top)
        # reconstruction error within step / 2 (plus fp16 rounding of m and step)
        zhat = m[None, :] + s[None, :] * codes[a:b]
        assert np.all(np.abs(zhat - z[a:b]) <= 0.5 * s[None, :] * (1 + 1e-2) + 1e-3 * np.abs(m)[None, :] + 1e-7)


@pytest.mark.parametrize("bits", [3, 4])
def test_method_key_codes_idempotent(bits):
    """Re-quantizing the dequantized directions with the same metadata gives the same codes."""
    wl, lay = _layer(96)
    kq = quantize_keys_bits_fmt(lay["k"][0, 0], 96, lay["signs"], bits)
    from oracle.ladder import key_codes_bits_fmt
    for g in range(3):
        zhat = (kq["m16"][g].astype(np.float32) + kq["step16"][g].astype(np.float32)
                * kq["codes"][32 * g:32 * g + 32].astype(np.float32))
        np.testing.assert_array_equal(key_codes_bits_fmt(zhat, kq["m16"][g], kq["step16"][g], bits),
                                      kq["codes"][32 * g:32 * g + 32])


@pytest.mark.parametrize("bits", [3, 4])
def test_lloyd_max_codes_are_nearest_levels(bits):
    wl, lay = _layer(120)
    cb, tau = codebook(128, bits)
    kq = quantize_keys_tq_bits_fmt(lay["k"][0, 0], 120, lay["signs"], bits)
    z = kq["z"].astype(np.float64)
    d = np.abs(z[:, :, None] - cb[None, None, :])
    clear = np.min(np.abs(z[:, :, None] - tau[None, None, :]), -1) > 1e-6
    np.testing.assert_array_equal(kq["codes"][:120][clear], d.argmin(-1)[clear])
    vq = quantize_values_bits_fmt(lay["v"][0, 0], lay["modality"][0], lay["rot"], 120, bits)
    zv = vq["y"].astype(np.float64) / vq["n16"].astype(np.float64)[:, None]
    dv = np.abs(zv[:, :, None] - cb[None, None, :])
    clear = np.min(np.abs(zv[:, :, None] - tau[None, None, :]), -1) > 1e-5
    np.testing.assert_array_equal(vq["codes"][clear], dv.argmin(-1)[clear])
    assert vq["codes"].max() == 2 ** bits - 1 and vq["codes"].min() == 0


def test_bit_stream_layout_by_hand():
    codes = np.zeros(128, np.uint8)
    codes[0], codes[1], codes[10], codes[127] = 5, 2, 7, 6
    p = pack_bits(codes, 3)
    assert p.shape == (48,)
    assert p[0] == 5 | (2 << 3)          # channel 0 bits 0-2, channel 1 bits 3-5
    assert p[3] == 0b11 << 6             # channel 10 = bits 30-32: its low two bits end byte 3 ...
    assert p[4] == 0b1                   # ... and its high bit opens byte 4
    assert p[47] == 6 << 5               # channel 127 = bits 381-383
    c4 = np.arange(128, dtype=np.uint8) % 16
    p4 = pack_bits(c4, 4)
    assert p4[0] == 0x10 and p4[7] == 0xFE       # two channels per byte, low nibble first
    rng = np.random.default_rng(0)
    for bits in BITS:
        c = rng.integers(0, 2 ** bits, (7, 128)).astype(np.uint8)
        np.testing.assert_array_equal(unpack_bits(pack_bits(c, bits), bits), c)


def test_bits_per_element_of_the_ladder():
    bpe = lambda kb, vb, meta: bytes_per_token_head(kb, vb, meta) * 8 / 256
    assert bpe(3, 2, "turboquant") == 2.625      # Tab. 3, TurboQuant K3/V2
    assert bpe(2, 2, "turboquant") == 2.125      # Tab. 3, TurboQuant K2/V2
    assert bpe(2, 2, "fp16") == 2.625            # Tab. 3, the method with fp16 metadata
    assert bpe(3, 3, "fp16") == 3.625 and bpe(4, 4, "fp16") == 4.625


@pytest.mark.parametrize("kb,vb,meta", [(3, 3, "fp16"), (4, 4, "fp16"), (3, 2, "turboquant"), (4, 4, "turboquant")])
def test_decode_rotated_equals_bruteforce(kb, vb, meta):
    wl = workload("omni7b_32k")
    lens = [77, 0, 130]
    lay = gen_layer(wl, 2, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :1].copy(), lay["v"][:, :1].copy()
    q = gen_queries(wl.wid, 2, 3, 7)
    c = quantize_layer_bits(k, v, lay["modality"], lens, lay["signs"], lay["rot"], 160, kb, vb, meta)
    a = decode_layer_bits(c, q, lens, lay["signs"], lay["rot"], SM, kb, vb, rotated=True)
    b = decode_layer_bits(c, q, lens, lay["signs"], lay["rot"], SM, kb, vb, rotated=False)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-10)
    assert np.all(a[1] == 0)


def test_two_bit_ladder_decode_equals_two_bit_cache_decode():
    wl = workload("omni7b_32k")
    lens = [100, 33]
    lay = gen_layer(wl, 3, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :1].copy(), lay["v"][:, :1].copy()
    q = gen_queries(wl.wid, 3, 2, 7)
    for meta in ("fp16", "turboquant"):
        c = quantize_layer_bits(k, v, lay["modality"], lens, lay["signs"], lay["rot"], 128, 2, 2, meta)
        ref = quantize_layer(k, v, lay["modality"], np.asarray(lens), lay["signs"], lay["rot"], 128, key_meta=meta)
        a = decode_layer_bits(c, q, lens, lay["signs"], lay["rot"], SM, 2, 2)
        b = decode_layer(ref, q, np.asarray(lens), lay["signs"], lay["rot"], SM)
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_more_bits_reconstruct_better():
    """The directions' reconstruction error shrinks with each extra bit (method and TurboQuant)."""
    wl, lay = _layer(256)
    for meta in ("fp16", "turboquant"):
        errs = []
        for bits in BITS:
            c = quantize_layer_bits(lay["k"], lay["v"], lay["modality"], [256], lay["signs"], lay["rot"], 256, bits,
                                    bits, meta)
            kq = quantize_keys_bits_fmt(lay["k"][0, 0], 256, lay["signs"], bits)
            zhat = key_directions_bits(c, 0, 0, 256, bits)
            errs.append(float(np.mean((zhat - kq["z"].astype(np.float64)) ** 2)))
        assert errs[0] > 2 * errs[1] > 4 * errs[2], (meta, errs)
