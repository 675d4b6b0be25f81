"""GPU parity of the key and value codecs against the oracle (bit-exact / band rule)."""

import numpy as np
import pytest

from oracle.cache import quantize_layer
from oracle.keys import quantize_keys_fmt
from oracle.layout import unpack_values
from oracle.values import quantize_values_fmt, rotation_error_bound
from synth import gen_layer, gen_rotations, gen_signs, workload

pytestmark = pytest.mark.gpu


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _ragged_layer(lens, H=2, n_tokens=None, layer=7):
    wl = workload("omni7b_32k")
    n = int(n_tokens or max(lens))
    return gen_layer(wl, layer, lengths=np.asarray(lens, np.int32), n_tokens=n)


def _check_keys(gpu, ref):
    for name in ("k_codes", "k_norm", "k_min", "k_step"):
        a, b = gpu[name], ref[name]
        if a.dtype == np.float16:
            a, b = a.view(np.uint16), b.view(np.uint16)
        mism = np.argwhere(a != b)
        assert len(mism) == 0, f"{name}: {len(mism)} mismatches, first at {mism[:5].tolist()}"


def test_keys_bit_exact_tiny_config():
    from gpu_helpers import quantize_stateless
    wl = workload("tiny_1k")
    lay = gen_layer(wl, 0)
    _announce("keys tiny_1k B1 H1 N1024")
    gpu = quantize_stateless(lay["k"], lay["v"], lay["modality"], lay["lens"], lay["signs"], lay["rot"], 1024, 4)
    ref = quantize_layer(lay["k"], lay["v"], lay["modality"], lay["lens"], lay["signs"], lay["rot"], 1024)
    _check_keys(gpu, ref)


def test_keys_bit_exact_ragged_and_degenerate():
    from gpu_helpers import quantize_stateless
    lens = [1000, 37, 64, 1, 0, 95]
    lay = _ragged_layer(lens)
    k = lay["k"]
    k[0, 0, 5] = 0                       # zero-norm token
    k[0, 1, 64:96] = k[0, 1, 64]         # a zero-range window: all tokens identical
    k[2, 0, :32, :] = np.float16(60000)  # huge norm: saturates the fp16 norm
    k[3, 1, 0, 7] = np.float16(-0.0)
    _announce(f"keys ragged lens={lens}")
    gpu = quantize_stateless(k, lay["v"], lay["modality"], lens, lay["signs"], lay["rot"], 1024, 4)
    ref = quantize_layer(k, lay["v"], lay["modality"], np.asarray(lens), lay["signs"], lay["rot"], 1024)
    _check_keys(gpu, ref)


def test_values_exact_mode_bit_exact():
    from gpu_helpers import quantize_stateless
    lens = [1024, 333, 5]
    lay = _ragged_layer(lens, layer=3)
    v = lay["v"]
    v[1, 0, 17] = 0                      # zero vector
    _announce(f"values exact lens={lens}")
    gpu = quantize_stateless(lay["k"], v, lay["modality"], lens, lay["signs"], lay["rot"], 1024, 4, exact=True)
    ref = quantize_layer(lay["k"], v, lay["modality"], np.asarray(lens), lay["signs"], lay["rot"], 1024)
    for name in ("v_codes", "v_norm"):
        a, b = gpu[name], ref[name]
        if a.dtype == np.float16:
            a, b = a.view(np.uint16), b.view(np.uint16)
        assert np.array_equal(a, b), f"{name}: {(a != b).sum()} mismatches"


def _band_compare(gpu_vcodes, v16, modality, rot, length):
    """MFMA-mode codes equal the exact order except where y is within the band of a threshold."""
    ref = quantize_values_fmt(v16, modality, rot, length)
    got = unpack_values(gpu_vcodes)[:length]
    eps = rotation_error_bound(v16[:length], modality[:length], rot)
    dist = np.abs(ref["y"][:, :, None].astype(np.float64) - ref["thr"][:, None, :].astype(np.float64)).min(-1)
    in_band = dist <= eps
    diff = got != ref["codes"]
    assert not np.any(diff & ~in_band), f"{int((diff & ~in_band).sum())} codes differ outside the band"
    assert np.all(np.abs(got.astype(int) - ref["codes"].astype(int)) <= 1)
    return int(diff.sum()), int(in_band.sum())


def test_values_mfma_band_rule_and_norms():
    from gpu_helpers import quantize_stateless
    lens = [1024, 700, 31]
    lay = _ragged_layer(lens, layer=4)
    _announce(f"values mfma lens={lens}")
    gpu = quantize_stateless(lay["k"], lay["v"], lay["modality"], lens, lay["signs"], lay["rot"], 1024, 4)
    ref = quantize_layer(lay["k"], lay["v"], lay["modality"], np.asarray(lens), lay["signs"], lay["rot"], 1024)
    assert np.array_equal(gpu["v_norm"].view(np.uint16), ref["v_norm"].view(np.uint16))
    total_diff = 0
    for b in range(3):
        for h in range(lay["k"].shape[1]):
            d, nb = _band_compare(gpu["v_codes"][b, h], lay["v"][b, h], lay["modality"][b], lay["rot"], lens[b])
            total_diff += d
    print(f"mfma codes differing (all in band): {total_diff}")
    # padded slots of the last window carry code 0
    pad = unpack_values(gpu["v_codes"][2, 0])[31:32]
    assert np.all(pad == 0)


def test_full_size_sampled_parity():
    """omni7b_32k shapes (B1, H4, 32768 tokens) in one launch each; sampled windows vs the oracle."""
    from gpu_helpers import quantize_stateless
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 0)
    _announce("codec full size omni7b_32k")
    gpu = quantize_stateless(lay["k"], lay["v"], lay["modality"], lay["lens"], lay["signs"], lay["rot"],
                             wl.capacity, wl.num_q_heads)
    rng = np.random.default_rng(11)
    for h in range(wl.num_kv_heads):
        for w in sorted(set(rng.integers(0, 1024, 12).tolist()) | {0, 1023}):
            a, b = 32 * w, 32 * w + 32
            kq = quantize_keys_fmt(lay["k"][0, h, a:b], 32, lay["signs"])
            np.testing.assert_array_equal(gpu["k_norm"][0, h, a:b].view(np.uint16), kq["n16"].view(np.uint16))
            np.testing.assert_array_equal(gpu["k_min"][0, h, w].view(np.uint16), kq["m16"][0].view(np.uint16))
            np.testing.assert_array_equal(gpu["k_step"][0, h, w].view(np.uint16), kq["step16"][0].view(np.uint16))
            from oracle.layout import pack_keys
            np.testing.assert_array_equal(gpu["k_codes"][0, h, a:b], pack_keys(kq["codes"]))
            _band_compare(gpu["v_codes"][0, h, w:w + 1], lay["v"][0, h, a:b], lay["modality"][0, a:b],
                          lay["rot"], 32)


def test_global_rotation_special_case_single_accumulator():
    """All three rotations equal: value codes do not depend on the modality labels."""
    from gpu_helpers import quantize_stateless
    lens = [512]
    lay = _ragged_layer(lens, layer=5)
    rot = np.stack([gen_rotations(9, 0)[0]] * 3)
    _announce("values identical rotations")
    a = quantize_stateless(lay["k"], lay["v"], lay["modality"], lens, lay["signs"], rot, 512, 4)
    m2 = (lay["modality"] + 1) % 3
    b = quantize_stateless(lay["k"], lay["v"], m2.astype(np.uint8), lens, lay["signs"], rot, 512, 4)
    assert np.array_equal(a["v_codes"], b["v_codes"])
    assert gen_signs(9, 0).shape == (128,)
