"""The synthetic workload generators: shapes, modality mixes and determinism."""

import numpy as np

from synth import (MOD_AUDIO, MOD_TEXT, MOD_VIDEO, WORKLOADS, gen_keys, gen_lengths, gen_values,
                   modality_layout, stream_chunk_modalities)


def _counts(m):
    return [(m == x).sum() for x in (MOD_VIDEO, MOD_AUDIO, MOD_TEXT)]


def test_modality_mixes():
    assert _counts(modality_layout(1024, 128, 64, 64)) == [640, 320, 64]
    assert _counts(modality_layout(32768, 150, 25, 256)) == [27887, 4625, 256]
    assert _counts(modality_layout(65536, 144, 16, 256)) == [58752, 6528, 256]
    m = modality_layout(131072, 150, 25, 256)
    assert _counts(m) == [747 * 150 + 91, 747 * 25, 256]
    # video first inside every chunk, text at the end
    assert m[0] == MOD_VIDEO and m[150] == MOD_AUDIO and m[-1] == MOD_TEXT


def test_streaming_continues_the_chunk_pattern():
    wl = WORKLOADS["omni3b_b4_64k_stream"]
    m = stream_chunk_modalities(wl, 0, 512)
    assert _counts(m)[:2] == [144 * 3 + 32, 16 * 3] and m[144] == MOD_AUDIO


def test_generators_deterministic_and_shaped():
    a = gen_keys(2, 0, 0, 1, 300)
    b = gen_keys(2, 0, 0, 1, 300)
    assert a.dtype == np.float16 and a.shape == (300, 128)
    np.testing.assert_array_equal(a, b)
    assert not np.array_equal(a, gen_keys(2, 0, 0, 2, 300))
    v = gen_values(2, 0, 0, 0, modality_layout(300, 150, 25, 20))
    assert v.dtype == np.float16 and np.isfinite(v).all()
    lens = gen_lengths(WORKLOADS["omni7b_b16_ragged16k"])
    assert lens.min() >= 8192 and lens.max() <= 16384 and len(set(lens.tolist())) > 8


def test_key_drift_is_local():
    """Windows of contiguous tokens span a smaller range than shuffled ones (the Tab. 6 effect)."""
    k = gen_keys(2, 0, 0, 0, 4096).astype(np.float64)
    contiguous = np.ptp(k.reshape(128, 32, 128), axis=1).mean()
    perm = np.random.default_rng(0).permutation(4096)
    shuffled = np.ptp(k[perm].reshape(128, 32, 128), axis=1).mean()
    assert contiguous < 0.8 * shuffled
