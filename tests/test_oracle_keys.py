"""Pins of the oracle's key codec (Eq. 2 + Eq. 4, readings R1-R9)."""

import math

import numpy as np

from oracle.hadamard import randomized_hadamard
from oracle.keys import (KAPPA32, dequantize_directions, f16_sat, key_codes_fmt, key_direction_fmt,
                         norm_tree_f32, quantize_keys_f64, quantize_keys_fmt, window_stats_fmt)
from synth import gen_keys, gen_signs


def _keys(n=256, seed=0):
    return gen_keys(1, seed, 0, 0, n), gen_signs(1, seed)


def _ulp16(x):
    x = np.abs(np.asarray(x, np.float16))
    return (np.nextafter(x, np.float16(np.inf)) - x).astype(np.float64)


def test_norm_tree_close_to_exact_and_saturates():
    k, _ = _keys()
    n32 = norm_tree_f32(k)
    exact = np.sqrt((k.astype(np.float64) ** 2).sum(-1))
    assert np.all(np.abs(n32 - exact) <= 8 * 2.0 ** -24 * exact)
    big = np.full((1, 128), 60000, np.float16)
    assert f16_sat(norm_tree_f32(big))[0] == np.float16(65504)
    assert norm_tree_f32(np.zeros((1, 128), np.float16))[0] == 0


def test_kappa_is_fp32_inverse_sqrt_128():
    assert KAPPA32 == np.float32(math.sqrt(2) / 16)
    assert KAPPA32.view(np.uint32) == 0x3DB504F3


def test_direction_matches_randomized_hadamard():
    k, s = _keys()
    z, n16 = key_direction_fmt(k, s)
    ref = (k.astype(np.float64) @ randomized_hadamard(s).T) / n16.astype(np.float64)[:, None]
    assert np.max(np.abs(z - ref)) < 2e-6
    np.testing.assert_allclose(np.linalg.norm(ref, axis=1), np.linalg.norm(k.astype(np.float64), axis=1)
                               / n16.astype(np.float64), rtol=1e-12)


def test_f64_error_bound_range_over_six():
    k, s = _keys(512)
    q = quantize_keys_f64(k, 512, s)
    g = np.arange(512) // 32
    zhat = q["lo"][g] + q["step"][g] * q["codes"]
    rng_ = 3 * q["step"][g]
    assert np.all(np.abs(q["z"] - zhat) <= rng_ / 6 + 1e-15)


def test_f64_rint_equals_bruteforce_argmin():
    k, s = _keys(512)
    q = quantize_keys_f64(k, 512, s)
    g = np.arange(512) // 32
    levels = q["lo"][g][..., None] + q["step"][g][..., None] * np.arange(4)
    brute = np.argmin(np.abs(q["z"][..., None] - levels), axis=-1)
    t = (q["z"] - q["lo"][g]) / q["step"][g]
    away = np.abs(t - np.floor(t) - 0.5) > 1e-9
    np.testing.assert_array_equal(brute[away], q["codes"][away])


def test_every_window_channel_uses_both_end_codes():
    k, s = _keys(512)
    for q in (quantize_keys_f64(k, 512, s), quantize_keys_fmt(k, 512, s)):
        c = q["codes"][:512].reshape(16, 32, 128)
        assert np.all(c.min(1) == 0) and np.all(c.max(1) == 3)


def test_fmt_error_bound_with_fp16_metadata():
    k, s = _keys(1024)
    q = quantize_keys_fmt(k, 1024, s)
    g = np.arange(1024) // 32
    zh = dequantize_directions(q["codes"], q["m16"], q["step16"])
    z = q["z"].astype(np.float64)
    lo = z.reshape(32, 32, 128).min(1)[g]
    hi = z.reshape(32, 32, 128).max(1)[g]
    bound = (hi - lo) / 6 + _ulp16(q["m16"])[g] + 2 * _ulp16(q["step16"])[g] + 1e-7
    assert np.all(np.abs(z - zh) <= bound)


def test_fmt_agrees_with_f64_away_from_ties():
    k, s = _keys(1024)
    a = quantize_keys_fmt(k, 1024, s)
    b = quantize_keys_f64(k, 1024, s)
    mism = a["codes"] != b["codes"]
    assert mism.mean() < 2e-3
    # every disagreement is within fp16-metadata rounding of a decision boundary
    g = np.arange(1024) // 32
    t = (b["z"] - b["lo"][g]) / b["step"][g]
    assert np.all(np.abs(t[mism] - np.floor(t[mism]) - 0.5) < 0.01)


def test_idempotence_at_the_direction_level():
    k, s = _keys(512)
    q = quantize_keys_f64(k, 512, s)
    g = np.arange(512) // 32
    zhat = q["lo"][g] + q["step"][g] * q["codes"]
    for w in range(16):
        zz = zhat[w * 32:(w + 1) * 32]
        lo, step = zz.min(0), (zz.max(0) - zz.min(0)) / 3
        np.testing.assert_allclose(lo, q["lo"][w], rtol=0, atol=1e-15)
        np.testing.assert_allclose(step, q["step"][w], rtol=1e-12)
        np.testing.assert_array_equal(np.clip(np.rint((zz - lo) / step), 0, 3), q["codes"][w * 32:(w + 1) * 32])
    # FMT: re-quantizing the fp32-dequantized directions reproduces codes and metadata
    f = quantize_keys_fmt(k, 512, s)
    zh32 = dequantize_directions(f["codes"], f["m16"], f["step16"]).astype(np.float32)
    for w in range(16):
        m16, st16 = window_stats_fmt(zh32[w * 32:(w + 1) * 32])
        np.testing.assert_array_equal(m16, f["m16"][w])
        codes = key_codes_fmt(zh32[w * 32:(w + 1) * 32], m16, st16)
        np.testing.assert_array_equal(codes, f["codes"][w * 32:(w + 1) * 32])


def test_closed_form_basis_vector_windows():
    s = np.ones(128, np.int8)
    s[0] = -1
    # all tokens a * e_0: z_c = s_0 * kappa for every channel -> zero range -> all codes 0
    k = np.zeros((32, 128), np.float16)
    k[:, 0] = np.float16(3.0)
    q = quantize_keys_fmt(k, 32, s)
    assert np.all(q["codes"] == 0) and np.all(q["step16"] == 0)
    np.testing.assert_array_equal(q["m16"][0], np.full(128, -KAPPA32, np.float32).astype(np.float16))
    # alternating +e_0 / -e_0: z = +-kappa -> lo = -kappa, hi = +kappa, codes 0 and 3
    k[1::2, 0] = np.float16(-3.0)
    q = quantize_keys_fmt(k, 32, s)
    zsign = np.where(np.arange(32) % 2 == 0, -1, 1)     # s_0 = -1 flips the sign
    np.testing.assert_array_equal(q["codes"][:, 5], np.where(zsign > 0, 3, 0))
    assert q["step16"][0, 5] == np.float16(np.float32(2 * KAPPA32) / np.float32(3))


def test_degenerate_zero_norm_and_partial_window():
    k, s = _keys(40)
    k[3] = 0
    q = quantize_keys_fmt(k, 40, s)
    assert q["n16"][3] == 0 and np.all(q["z"][3] == 0)
    assert q["codes"].shape == (64, 128) and np.all(q["codes"][40:] == 0) and np.all(q["n16"][40:] == 0)
    # partial window statistics use valid tokens only
    m16, st16 = window_stats_fmt(q["z"][32:40])
    np.testing.assert_array_equal(q["m16"][1], m16)
    np.testing.assert_array_equal(q["step16"][1], st16)
    # -0 canonicalized in the stored minimum
    zz = np.full((4, 128), -0.0, np.float32)
    m16, st16 = window_stats_fmt(zz)
    assert np.all(np.signbit(m16) == False) and np.all(np.signbit(st16) == False)  # noqa: E712


def test_planted_mistakes_are_caught():
    """A dropped sign flip or a transposed Hadamard must break the pinned direction."""
    k, s = _keys(64)
    z, n16 = key_direction_fmt(k, s)
    z_nosign, _ = key_direction_fmt(k, np.ones(128, np.int8))
    ref = (k.astype(np.float64) @ randomized_hadamard(s).T) / n16.astype(np.float64)[:, None]
    assert np.max(np.abs(z_nosign - ref)) > 1e-2
    wrong = (k.astype(np.float64) @ randomized_hadamard(s)) / n16.astype(np.float64)[:, None]
    assert np.max(np.abs(wrong - ref)) > 1e-2
