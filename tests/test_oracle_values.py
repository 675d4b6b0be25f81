"""Pins of the oracle's value codec (Eq. 6 with the Eq. 3 codebook, readings R6-R8, R14)."""

import math

import numpy as np

from oracle.codebook import codebook, lloyd_max_gaussian, mse_closed_form
from oracle.hadamard import fwht_f64, randomized_hadamard
from oracle.values import (dequantize_values, quantize_values_f64, quantize_values_fmt,
                           rotate_values_f32_sequential, rotation_error_bound)
from synth import gen_rotations, gen_signs, gen_values, modality_layout


def _vals(n=384):
    mod = modality_layout(n, 128, 64, 64)
    return gen_values(1, 0, 0, 0, mod), mod, gen_rotations(1, 0)


def test_rotations_orthogonal():
    rot = gen_rotations(1, 0).astype(np.float64)
    for r in rot:
        np.testing.assert_allclose(r @ r.T, np.eye(128), atol=1e-6)   # fp32-rounded inputs


def test_sequential_rotation_error_bound():
    v, mod, rot = _vals()
    y32 = rotate_values_f32_sequential(v, mod, rot).astype(np.float64)
    y64 = np.einsum("nij,nj->ni", rot.astype(np.float64)[mod], v.astype(np.float64))
    # recursive summation: |err| <= gamma_{d} sum |R_cj x_j| (+ the rounding of each product)
    assert np.all(np.abs(y32 - y64) <= rotation_error_bound(v, mod, rot, rel=129 * 2.0 ** -24) + 1e-30)


def test_threshold_count_equals_bruteforce_argmin_away_from_band():
    v, mod, rot = _vals()
    f = quantize_values_fmt(v, mod, rot, len(mod))
    d = quantize_values_f64(v, mod, rot, len(mod))
    eps = rotation_error_bound(v, mod, rot) + np.abs(f["thr"]).max(1, keepdims=True) * 2.0 ** -22
    dist = np.min(np.abs(d["y"][:, :, None] - d["n16"][:, None, None] * codebook(128)[1][None, None, :]), -1)
    clear = dist > eps
    np.testing.assert_array_equal(f["codes"][clear], d["codes"][clear])
    assert clear.mean() > 0.999


def test_turboquant_special_case_via_butterflies():
    """R_m = H for every modality reduces Eq. 6 to TurboQuant's Eq. 2-3 on the same codebook."""
    v, mod, _ = _vals(128)
    s = gen_signs(1, 0)
    h = randomized_hadamard(s)
    d = quantize_values_f64(v, mod, np.stack([h, h, h]), len(mod))
    x = v.astype(np.float64)
    z = fwht_f64(x * s) / math.sqrt(128) / d["n16"][:, None]
    cb, _ = codebook(128)
    tq = np.argmin(np.abs(z[:, :, None] - cb), -1)
    np.testing.assert_array_equal(tq, d["codes"])


def test_closed_form_basis_vector():
    rot = np.stack([np.eye(128, dtype=np.float32)] * 3)
    v = np.zeros((2, 128), np.float16)
    v[0, 7] = 5.0
    f = quantize_values_fmt(v, np.array([0, 1]), rot, 2)
    expect = np.ones(128, np.uint8)      # zero coordinates sit above the first (negative) threshold
    expect[7] = 3
    np.testing.assert_array_equal(f["codes"][0], expect)
    np.testing.assert_array_equal(f["codes"][1], np.zeros(128, np.uint8))   # zero vector: all code 0
    vh = dequantize_values(f["codes"], f["n16"], np.array([0, 1]), rot)
    cb, _ = codebook(128)
    assert abs(vh[0, 7] - 5.0 * cb[3]) < 1e-12 and abs(vh[0, 0] - 5.0 * cb[1]) < 1e-12
    assert np.all(vh[1] == 0)


def test_exact_threshold_takes_lower_code():
    tau = codebook(128)[1].astype(np.float32)
    rot = np.stack([np.eye(128, dtype=np.float32)] * 3)
    # choose a value whose norm is exactly representable and one coordinate exactly on T_2
    v = np.zeros((1, 128), np.float16)
    v[0, 0] = 64.0
    f = quantize_values_fmt(v, np.array([2]), rot, 1)
    thr = np.float32(64.0) * tau[2]
    y = f["y"].copy()
    y[0, 1] = thr
    code = int((y[0, 1] > f["thr"][0]).sum())
    assert code == 2


def test_lloyd_max_mse_on_gaussian_directions():
    """Random unit directions rotated by an orthogonal R_m have coordinates ~N(0,1/d): the per-
    coordinate squared error of the 2-bit value codec must match the Lloyd-Max MSE / d."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((4000, 128)).astype(np.float16)
    mod = np.zeros(4000, np.int64)
    rot = gen_rotations(1, 3)
    d = quantize_values_f64(x, mod, rot, 4000)
    cb, _ = codebook(128)
    err = (d["z"] - cb[d["codes"]]) ** 2
    c, t = lloyd_max_gaussian(4)
    assert abs(err.mean() * 128 / mse_closed_form(c, t) - 1) < 0.03


def test_dequantize_inverts_rotation():
    v, mod, rot = _vals(64)
    d = quantize_values_f64(v, mod, rot, 64)
    vh = dequantize_values(d["codes"], d["n16"], mod, rot)
    # the rotated reconstruction equals cb[code] scaled by the norm
    cb, _ = codebook(128)
    back = np.einsum("nij,nj->ni", rot.astype(np.float64)[mod], vh)
    np.testing.assert_allclose(back, d["n16"][:, None] * cb[d["codes"]], atol=1e-5)
    # planted mistake: dequantizing with the wrong modality's rotation is far off
    wrong = dequantize_values(d["codes"], d["n16"], (mod + 1) % 3, rot)
    assert np.linalg.norm(wrong - vh) > 0.5 * np.linalg.norm(vh)
