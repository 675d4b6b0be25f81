"""Pins of the TurboQuant key codec oracle (Eq. 2, Eq. 3): nearest-codebook codes by brute force,
agreement with the value codec run with R = H (a different code path: a dense rotation instead of
butterflies), idempotence at the direction level, the two decode formulations, their special
cases, and Tab. 3's 2.125 bits per element from the layout's byte count."""

import math

import numpy as np

from oracle.codebook import codebook
from oracle.hadamard import randomized_hadamard
from oracle.layout import bits_per_element, pack_keys, unpack_keys
from oracle.turboquant import decode_tq_bruteforce, decode_tq_rotated, dequantize_keys_tq, quantize_keys_tq_fmt
from oracle.values import dequantize_values, quantize_values_f64
from synth import gen_layer, gen_queries, workload

SM = 1 / math.sqrt(128)


def _keys(n=300, seed=0):
    wl = workload("tiny_1k")
    lay = gen_layer(wl, seed, lengths=np.array([n], np.int32), n_tokens=n)
    return lay, lay["k"][0, 0]


def test_codes_are_nearest_codebook_entries():
    lay, k = _keys()
    kq = quantize_keys_tq_fmt(k, 300, lay["signs"])
    cb, _ = codebook(128)
    z = kq["z"].astype(np.float64)
    dist = np.abs(z[:, :, None] - cb[None, None, :])
    brute = np.argmin(dist, axis=-1)
    srt = np.sort(dist, axis=-1)
    clear = (srt[..., 1] - srt[..., 0]) > 1e-9          # no exact tie
    assert clear.mean() > 0.999
    np.testing.assert_array_equal(kq["codes"][:300][clear], brute[clear])
    assert np.all(kq["codes"][300:] == 0) and np.all(kq["n16"][300:] == 0)
    # all four codes occur (the direction coordinates are near N(0, 1/128))
    assert set(np.unique(kq["codes"][:300])) == {0, 1, 2, 3}


def test_equals_value_codec_with_hadamard_rotation():
    """TurboQuant treats keys like values: the value codec with R_m = H (float64, dense rotation)
    gives the same codes except where z lies within rounding distance of a threshold."""
    lay, k = _keys(200, seed=1)
    kq = quantize_keys_tq_fmt(k, 200, lay["signs"])
    H = randomized_hadamard(lay["signs"])
    vq = quantize_values_f64(k, np.zeros(200, np.uint8), np.stack([H] * 3), 200)
    _, tau = codebook(128)
    near = np.abs(vq["z"][:, :, None] - tau[None, None, :]).min(-1) <= 1e-6
    diff = kq["codes"][:200] != vq["codes"]
    assert not np.any(diff & ~near)
    np.testing.assert_array_equal(kq["n16"][:200], vq["n16"].astype(np.float16))


def test_idempotent_on_codebook_points():
    """A direction equal to codebook entries codes back to the same indices (each level lies in its
    own cell): quantize n16 H^T cb[code] and compare."""
    lay, k = _keys(64, seed=2)
    kq = quantize_keys_tq_fmt(k, 64, lay["signs"])
    khat = dequantize_keys_tq(kq["codes"][:64], kq["n16"][:64], lay["signs"])
    k2 = quantize_keys_tq_fmt(khat.astype(np.float16), 64, lay["signs"])
    agree = (k2["codes"][:64] == kq["codes"][:64]).mean()
    assert agree > 0.995, agree   # fp16 rounding of khat and its new norm move a few coordinates


def test_decode_formulations_and_special_cases():
    wl = workload("tiny_1k")
    lay = gen_layer(wl, 0, lengths=np.array([500], np.int32), n_tokens=500)
    kq = quantize_keys_tq_fmt(lay["k"][0, 0], 500, lay["signs"])
    from oracle.values import quantize_values_fmt
    vq = quantize_values_fmt(lay["v"][0, 0], lay["modality"][0], lay["rot"], 500)
    q = gen_queries(wl.wid, 0, 1, 4)[0]
    args = (kq["codes"], kq["n16"], vq["codes"], vq["n16"], lay["modality"][0])
    for L in (1, 37, 500):
        a = decode_tq_bruteforce(q, *args, L, lay["signs"], lay["rot"], SM, 4)
        b = decode_tq_rotated(q, *args, L, lay["signs"], lay["rot"], SM, 4)
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12 * np.abs(a).max())
    vhat = dequantize_values(vq["codes"][:500], vq["n16"], lay["modality"][0][:500], lay["rot"])
    one = decode_tq_rotated(q, *args, 1, lay["signs"], lay["rot"], SM, 4)
    np.testing.assert_allclose(one, np.stack([vhat[0]] * 4), rtol=1e-12)
    zero = decode_tq_rotated(np.zeros_like(q), *args, 500, lay["signs"], lay["rot"], SM, 4)
    np.testing.assert_allclose(zero[0], vhat.mean(0), rtol=1e-10, atol=1e-14)


def test_layout_round_trip_and_tab3_bits():
    lay, k = _keys(96, seed=3)
    kq = quantize_keys_tq_fmt(k, 96, lay["signs"])
    np.testing.assert_array_equal(unpack_keys(pack_keys(kq["codes"])), kq["codes"])
    per_token_head = 32 + 2 + 32 + 2          # key codes, key norm, value codes, value norm
    assert per_token_head * 8 / (2 * 128) == bits_per_element("turboquant_k2v2") == 2.125
