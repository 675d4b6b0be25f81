"""The device-side layer generator (synth.device, used by the 48-layer benchmark) follows the
recipe of synth.workloads: value spread of a rank-16 subspace plus noise, keys with four outlier
channels scaled by 8 and a per-64-token random-walk mean, the workload's token stream, distinct
layers for distinct seeds. Run on the CPU device."""

import numpy as np
import pytest

from synth import modality_layout, workload
from synth.device import gen_layer_device


def test_device_generator_follows_the_recipe():
    torch = pytest.importorskip("torch")
    wl = workload("tiny_1k")
    lay = gen_layer_device(wl, 3, "cpu")
    k = lay["k"].float().numpy()[0, 0]          # [1024][128]
    v = lay["v"].float().numpy()[0, 0]
    assert lay["k"].dtype == torch.float16 and lay["k"].shape == (1, 1, 1024, 128)
    # values: a rank-16 orthonormal subspace per modality (each coordinate's variance 16 / 128) plus
    # N(0, 0.05^2) noise
    assert abs(v.var() - (16 / 128 + 0.05 ** 2)) < 0.01
    # keys: 4 outlier channels carry ~8x the spread of the others (after removing the drift)
    dk = np.diff(k, axis=0)                     # the drift cancels inside a 64-token block
    spread = dk.std(axis=0)
    top = np.sort(spread)[-4:]
    rest = np.sort(spread)[:-4]
    assert top.min() > 5 * rest.max()
    # the random-walk mean moves between 64-token blocks (std 0.5 per step and channel)
    blocks = k[:1024].reshape(16, 64, 128).mean(axis=1)
    normal = np.argsort(spread)[:-4]
    steps = np.diff(blocks[:, normal], axis=0)
    assert 0.3 < steps.std() < 0.8
    np.testing.assert_array_equal(lay["modality_np"][0], modality_layout(1024, wl.video_per_chunk, wl.audio_per_chunk,
                                                                          wl.text_tail))
    other = gen_layer_device(wl, 4, "cpu")
    assert not np.array_equal(other["k"].numpy(), lay["k"].numpy())
    again = gen_layer_device(wl, 3, "cpu")
    np.testing.assert_array_equal(again["k"].numpy(), lay["k"].numpy())
