"""Pins of the oracle's codebook (Eq. 3) and randomized Hadamard transform (Eq. 2)."""

import math

import numpy as np
import pytest
import scipy.integrate
import scipy.linalg
import scipy.stats

from oracle.codebook import codebook, lloyd_max_gaussian, mse_closed_form, thresholds_f32
from oracle.hadamard import fwht_f32, fwht_f64, randomized_hadamard, sylvester


def test_lloyd_max_matches_textbook_table(golden):
    g = golden("lloyd_max_gaussian_4level.txt")
    c, t = lloyd_max_gaussian(4)
    np.testing.assert_allclose(c, g["levels"], atol=6e-4)
    np.testing.assert_allclose(t, g["thresholds"], atol=6e-5)
    assert abs(mse_closed_form(c, t) - g["mse"][0]) < 6e-5


def test_lloyd_max_fixed_point_by_quadrature():
    c, t = lloyd_max_gaussian(4)
    edges = [-np.inf] + list(t) + [np.inf]
    pdf = scipy.stats.norm.pdf
    for i, ci in enumerate(c):
        mass = scipy.integrate.quad(pdf, edges[i], edges[i + 1])[0]
        mom = scipy.integrate.quad(lambda x: x * pdf(x), edges[i], edges[i + 1])[0]
        assert abs(mom / mass - ci) < 1e-9          # every level is its cell's centroid
    for i in range(3):
        assert abs(t[i] - (c[i] + c[i + 1]) / 2) < 1e-15   # thresholds are midpoints


def _mse_quad(c, t):
    edges = [-np.inf] + list(t) + [np.inf]
    pdf = scipy.stats.norm.pdf
    return sum(scipy.integrate.quad(lambda x, ci=ci: (x - ci) ** 2 * pdf(x), edges[i], edges[i + 1])[0]
               for i, ci in enumerate(c))


def test_lloyd_max_mse_and_local_optimality():
    c, t = lloyd_max_gaussian(4)
    base = _mse_quad(c, t)
    assert abs(base - mse_closed_form(c, t)) < 1e-10
    for i in range(4):
        for d in (-1e-3, 1e-3):
            cc = c.copy()
            cc[i] += d
            tt = np.array([(cc[k] + cc[k + 1]) / 2 for k in range(3)])
            assert _mse_quad(cc, tt) > base


def test_codebook_scaling_and_thresholds():
    cb, tau = codebook(128)
    c, t = lloyd_max_gaussian(4)
    np.testing.assert_allclose(cb * math.sqrt(128), c, rtol=1e-15)
    assert np.all(np.diff(cb) > 0) and tau[1] == 0.0
    assert thresholds_f32(128).dtype == np.float32
    # a 2-level Lloyd-Max quantizer of N(0,1) is +-sqrt(2/pi) (closed form)
    c2, _ = lloyd_max_gaussian(2)
    np.testing.assert_allclose(c2, [-math.sqrt(2 / math.pi), math.sqrt(2 / math.pi)], rtol=1e-12)


def test_sylvester_matches_scipy():
    for d in (1, 2, 8, 128):
        np.testing.assert_array_equal(sylvester(d), scipy.linalg.hadamard(d))


def test_randomized_hadamard_orthogonal():
    rng = np.random.default_rng(1)
    s = np.where(rng.integers(0, 2, 128) == 1, 1, -1)
    h = randomized_hadamard(s)
    np.testing.assert_allclose(h @ h.T, np.eye(128), atol=1e-12)
    np.testing.assert_allclose(h[:, 0], s[0] / math.sqrt(128) * np.ones(128), rtol=0)


def test_fwht_equals_sylvester_product_exactly_on_integers():
    rng = np.random.default_rng(2)
    x = rng.integers(-50, 50, size=(16, 128)).astype(np.float64)
    ref = x @ scipy.linalg.hadamard(128).T
    np.testing.assert_array_equal(fwht_f64(x), ref)
    np.testing.assert_array_equal(fwht_f32(x.astype(np.float32)), ref.astype(np.float32))
    e0 = np.zeros(128)
    e0[0] = 1
    np.testing.assert_array_equal(fwht_f64(e0), np.ones(128))


def test_fwht_f32_close_to_f64():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((64, 128)).astype(np.float32)
    a = fwht_f32(x).astype(np.float64)
    b = x.astype(np.float64) @ scipy.linalg.hadamard(128).T
    bound = 7 * 2.0 ** -24 * (np.abs(x).astype(np.float64) @ np.ones((128, 128)))
    assert np.all(np.abs(a - b) <= bound)


def test_fwht_butterfly_order_is_h_ascending():
    """x = e_0 + e_1 + 2^-24 e_2, hand-worked. With h ascending the first stage pairs neighbours:
    w_0 = 2, w_1 = 0 (exact cancellation), w_2 = w_3 = 2^-24; every later stage adds exact values,
    so each odd row i ends at Had[i, 2] 2^-24 exactly and each even row at 2 Had[i, 0] (2 + 2^-24
    rounds back to 2). With h descending, x_0 and x_2 meet first (h = 2): 1 + 2^-24 is a tie and
    rounds to 1 (even), so the rows where they add lose the 2^-24 before x_1 cancels the 1: those
    odd rows end at 0, not +-2^-24."""
    d = 128
    x = np.zeros(d, np.float32)
    x[0] = 1
    x[1] = 1
    x[2] = 2.0 ** -24
    had = scipy.linalg.hadamard(d)
    want = np.where(np.arange(d) % 2 == 1, had[:, 2] * 2.0 ** -24, 2.0 * had[:, 0]).astype(np.float32)
    got = fwht_f32(x)
    np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))
    # the same butterflies with h descending give other bits
    w = x.copy()
    for h in (64, 32, 16, 8, 4, 2, 1):
        v = w.reshape(d // (2 * h), 2, h)
        a, b = v[:, 0, :].copy(), v[:, 1, :].copy()
        v[:, 0, :], v[:, 1, :] = a + b, a - b
        w = v.reshape(d)
    assert not np.array_equal(w.view(np.uint32), got.view(np.uint32))
    assert np.all(w[1::2][had[1::2, 2] > 0] == 0)