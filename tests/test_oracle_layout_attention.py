"""Pins of the pack maps, the Tab. 3 byte accounting and the attention oracle (Eq. 1)."""

import math

import numpy as np
import scipy.special

from oracle.attention import decode_bruteforce, decode_rotated, softmax_attention
from oracle.cache import decode_layer, quantize_layer, unpacked_fields
from oracle.keys import dequantize_keys
from oracle.layout import (bits_per_element, cache_bytes_per_token_head, pack_keys, pack_values, unpack_keys,
                           unpack_values, value_byte_index)
from oracle.values import dequantize_values
from synth import gen_layer, workload


def test_tab3_bits_per_element(golden):
    g = golden("tab3_bits_per_element.txt")
    for scheme, (bits,) in g.items():
        assert abs(bits_per_element(scheme) - bits) < 5e-4, scheme
    per_tok = sum(cache_bytes_per_token_head().values())
    assert per_tok == 84
    assert per_tok * 8 / 256 == g["ours_fp16_meta"][0]


def test_key_pack_examples_and_roundtrip():
    codes = np.zeros((3, 128), np.uint8)
    codes[2, 5] = 3        # odd channel of pair 2 in word 0: high half, bits 16 + 4
    codes[1, 8] = 1        # even channel of pair 4: low half, bits 8
    codes[0, 127] = 2      # odd channel of pair 7 in word 7: high half, bits 16 + 14
    p = pack_keys(codes)
    assert p[2, 2] == 0b110000 and p[1, 1] == 0b1 and p[0, 31] == 0b10000000
    assert int(p.astype(np.int64).sum()) == 48 + 1 + 128
    words = p.view("<u4")  # word t of a token: channel pair (16 t + 2 j, +1) under mask 3 * 0x00010001 << 2 j
    assert (int(words[2, 0]) >> 16) & 0b110000 == 0b110000 and int(words[1, 0]) & (0x00030003 << 8) == 1 << 8
    rng = np.random.default_rng(0)
    c = rng.integers(0, 4, (64, 128)).astype(np.uint8)
    np.testing.assert_array_equal(unpack_keys(pack_keys(c)), c)


def test_value_pack_bijection_examples_and_roundtrip():
    t, c = np.meshgrid(np.arange(32), np.arange(128), indexing="ij")
    idx = value_byte_index(t, c) * 4 + (t & 3)
    assert len(np.unique(idx)) == 32 * 128 and idx.max() == 4095
    assert value_byte_index(np.array(0), np.array(0)) == 0
    assert value_byte_index(np.array(17), np.array(33)) == 26
    codes = np.zeros((32, 128), np.uint8)
    codes[17, 33] = 2
    p = pack_values(codes)
    assert p[0, 26] == 2 << 2 and p.sum() == 8
    rng = np.random.default_rng(1)
    cc = rng.integers(0, 4, (96, 128)).astype(np.uint8)
    np.testing.assert_array_equal(unpack_values(pack_values(cc)), cc)


def test_softmax_attention_matches_library_softmax():
    rng = np.random.default_rng(2)
    q, k, v = rng.standard_normal(16), rng.standard_normal((9, 16)), rng.standard_normal((9, 16))
    ref = scipy.special.softmax(k @ q / 4.0) @ v
    np.testing.assert_allclose(softmax_attention(q, k, v, 0.25), ref, rtol=1e-13)


def _tiny_cache(n=200):
    wl = workload("tiny_1k")
    lay = gen_layer(wl, 0, lengths=np.array([n]), n_tokens=n)
    cache = quantize_layer(lay["k"], lay["v"], lay["modality"], lay["lens"], lay["signs"], lay["rot"])
    return wl, lay, cache


def test_rotated_formulation_equals_bruteforce():
    wl, lay, cache = _tiny_cache()
    args = unpacked_fields(cache, 0, 0)
    q = lay["q"][0]
    a = decode_rotated(q, *args, 200, lay["signs"], lay["rot"], 1 / math.sqrt(128), 4)
    b = decode_bruteforce(q, *args, 200, lay["signs"], lay["rot"], 1 / math.sqrt(128), 4)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12 * np.abs(b).max())


def test_attention_special_cases():
    wl, lay, cache = _tiny_cache(64)
    kc, m16, st16, nk, vc, nv, mod = unpacked_fields(cache, 0, 0)
    vhat = dequantize_values(vc[:64], nv[:64], mod[:64], lay["rot"])
    khat = dequantize_keys(kc[:64], m16, st16, nk[:64], lay["signs"])
    sc = 1 / math.sqrt(128)
    # one-token cache -> the output is that token's dequantized value
    one = decode_rotated(lay["q"][0], kc, m16, st16, nk, vc, nv, mod, 1, lay["signs"], lay["rot"], sc, 4)
    np.testing.assert_allclose(one, np.repeat(vhat[:1], 4, 0), rtol=1e-12, atol=1e-14)
    # q = 0 -> uniform weights -> mean of the dequantized values
    zq = np.zeros((4, 128), np.float16)
    o = decode_rotated(zq, kc, m16, st16, nk, vc, nv, mod, 64, lay["signs"], lay["rot"], sc, 4)
    np.testing.assert_allclose(o, np.repeat(vhat.mean(0, keepdims=True), 4, 0), rtol=1e-10, atol=1e-13)
    # a query aligned with one key and scaled up picks that key's value
    big = (khat[10] / np.linalg.norm(khat[10]) * 3000).astype(np.float16)[None].repeat(4, 0)
    o = decode_rotated(big, kc, m16, st16, nk, vc, nv, mod, 64, lay["signs"], lay["rot"], sc, 4)
    sel = np.argmax(khat @ big[0].astype(np.float64))
    np.testing.assert_allclose(o[0], vhat[sel], rtol=1e-3, atol=1e-3 * np.abs(vhat[sel]).max())


def test_gqa_mapping_and_planted_transpose():
    wl = workload("tiny_1k")
    n = 96
    lay = gen_layer(wl, 0, lengths=np.array([n]), n_tokens=n)
    # two KV heads with different caches; 8 query heads -> G = 4
    k = np.concatenate([lay["k"], lay["k"][:, :, ::-1].copy()], axis=1)
    v = np.concatenate([lay["v"], lay["v"][:, :, ::-1].copy()], axis=1)
    cache = quantize_layer(k, v, lay["modality"], lay["lens"], lay["signs"], lay["rot"])
    q = np.concatenate([lay["q"], lay["q"][:, ::-1]], axis=1)
    out = decode_layer(cache, q, lay["lens"], lay["signs"], lay["rot"], 1 / math.sqrt(128))
    for j in range(8):
        h = j // 4
        ref = decode_rotated(q[0, j:j + 1], *unpacked_fields(cache, 0, h), n, lay["signs"], lay["rot"],
                             1 / math.sqrt(128), 1)
        np.testing.assert_allclose(out[0, j], ref[0], rtol=1e-12)
    # a transposed value rotation (R instead of R^T) gives a different output
    wrong = decode_rotated(q[0, :4], *unpacked_fields(cache, 0, 0), n, lay["signs"],
                           lay["rot"].transpose(0, 2, 1).copy(), 1 / math.sqrt(128), 4)
    assert np.abs(wrong - out[0, :4]).max() > 1e-2 * np.abs(out[0, :4]).max()


def test_prefix_windows_are_independent():
    wl = workload("tiny_1k")
    lay = gen_layer(wl, 0, lengths=np.array([200]), n_tokens=200)
    full = quantize_layer(lay["k"], lay["v"], lay["modality"], lay["lens"], lay["signs"], lay["rot"], 224)
    part = quantize_layer(lay["k"], lay["v"], lay["modality"], np.array([150]), lay["signs"], lay["rot"], 224)
    np.testing.assert_array_equal(full["k_codes"][0, 0, :128], part["k_codes"][0, 0, :128])
    np.testing.assert_array_equal(full["k_min"][0, 0, :4], part["k_min"][0, 0, :4])
    np.testing.assert_array_equal(unpack_values(full["v_codes"][0, 0])[:150], unpack_values(part["v_codes"][0, 0])[:150])
