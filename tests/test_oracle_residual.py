"""Pins of the fp16-residual decode oracle (captioning protocol, Sec. 3.1): the zones where keys and
values are read quantized or fp16, and the special cases that reduce to the dense fp16 cache and to
the fully quantized cache."""

import math

import numpy as np
import pytest

from oracle.attention import decode_bruteforce, decode_dense
from oracle.cache import quantize_layer, unpacked_fields
from oracle.residual import decode_residual, residual_boundaries
from synth import gen_layer, gen_queries, workload

SM = 1 / math.sqrt(128)


@pytest.fixture(scope="module")
def layer():
    wl = workload("tiny_1k")
    lay = gen_layer(wl, 0)
    cache = quantize_layer(lay["k"], lay["v"], lay["modality"], lay["lens"], lay["signs"], lay["rot"], 1024)
    q = gen_queries(wl.wid, 0, 1, 4)[0]
    return lay, cache, q


def _run(layer, L, k16=None, v16=None, window=128):
    lay, cache, q = layer
    f = unpacked_fields(cache, 0, 0)
    k16 = lay["k"][0, 0] if k16 is None else k16
    v16 = lay["v"][0, 0] if v16 is None else v16
    return decode_residual(q, *f[:6], f[6], k16, v16, L, lay["signs"], lay["rot"], SM, 4, window=window)


def test_boundaries():
    assert residual_boundaries(0) == (0, 0)
    assert residual_boundaries(127) == (0, 0)
    assert residual_boundaries(128) == (128, 0)
    assert residual_boundaries(130) == (128, 2)
    assert residual_boundaries(300) == (256, 172)
    assert residual_boundaries(300, 0) == (300, 300)


@pytest.mark.parametrize("L", [1, 77, 127])
def test_short_sequence_is_the_dense_fp16_cache(layer, L):
    lay, _, q = layer
    ref = decode_dense(q, lay["k"][0, 0], lay["v"][0, 0], L, SM, 4)
    np.testing.assert_allclose(_run(layer, L), ref, rtol=0, atol=1e-13)


def test_window_zero_is_the_quantized_cache(layer):
    lay, cache, q = layer
    f = unpacked_fields(cache, 0, 0)
    ref = decode_bruteforce(q, *f, 700, lay["signs"], lay["rot"], SM, 4)
    np.testing.assert_allclose(_run(layer, 700, window=0), ref, rtol=0, atol=1e-13)


@pytest.mark.parametrize("L", [130, 256, 300, 1000])
def test_zones_by_perturbation(layer, L):
    """Changing an fp16 input changes the output exactly where the protocol reads it raw."""
    lay, _, _ = layer
    kq, vq = residual_boundaries(L)
    base = _run(layer, L)
    k16, v16 = lay["k"][0, 0], lay["v"][0, 0]

    def moved(i, which):
        kk, vv = k16.copy(), v16.copy()
        (kk if which == "k" else vv)[i] += np.float16(0.5)
        return np.abs(_run(layer, L, kk, vv) - base).max() > 0

    for i in (kq - 1, vq - 1, 0):
        if i >= 0:
            assert not moved(i, "k") if i < kq else moved(i, "k")
            assert not moved(i, "v") if i < vq else moved(i, "v")
    for i in (kq, vq, L - 1):
        if i < L:
            assert moved(i, "k") == (i >= kq)
            assert moved(i, "v") == (i >= vq)
