"""GPU parity with MXFP4 key window metadata: records, codes and norms bit-exact against the oracle,
chunked appends equal to one-shot quantization, decode within 2e-3 of the output norm."""

import math

import numpy as np
import pytest

from oracle.cache import decode_layer, quantize_layer
from synth import gen_layer, gen_queries, workload

pytestmark = pytest.mark.gpu
TOL = 2e-3
SM = 1 / math.sqrt(128)
KEY_FIELDS = ("k_codes", "k_norm", "k_mx")


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _check(gpu, ref, fields=KEY_FIELDS):
    for name in fields:
        a, b = gpu[name], ref[name]
        if a.dtype == np.float16:
            a, b = a.view(np.uint16), b.view(np.uint16)
        mism = np.argwhere(a != b)
        assert len(mism) == 0, f"{name}: {len(mism)} mismatches, first at {mism[:5].tolist()}"


def test_mx_keys_bit_exact_tiny_config():
    import gpu_helpers as gh
    lay = gen_layer(workload("tiny_1k"), 0)
    _announce("mx keys tiny_1k")
    gpu = gh.quantize_stateless(lay["k"], lay["v"], lay["modality"], lay["lens"], lay["signs"], lay["rot"], 1024, 4,
                                key_meta="mxfp4")
    ref = quantize_layer(lay["k"], lay["v"], lay["modality"], lay["lens"], lay["signs"], lay["rot"], 1024,
                         key_meta="mxfp4")
    _check(gpu, ref)


def test_mx_keys_bit_exact_ragged_and_degenerate():
    import gpu_helpers as gh
    lens = [1000, 37, 64, 1, 0, 95]
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 7, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k = lay["k"]
    k[0, 0, 5] = 0                       # zero-norm token
    k[0, 1, 64:96] = k[0, 1, 64]         # a zero-range window: every step is 0 (an all-zero block)
    k[2, 0, :32, :] = np.float16(60000)  # huge norm: saturates the fp16 norm
    k[3, 1, 0, 7] = np.float16(-0.0)
    k[5, 2, 32:64, :] = 0                # an all-zero window: minimum and step blocks all zero
    _announce(f"mx keys ragged lens={lens}")
    gpu = gh.quantize_stateless(k, lay["v"], lay["modality"], lens, lay["signs"], lay["rot"], 1024, 4,
                                key_meta="mxfp4")
    ref = quantize_layer(k, lay["v"], lay["modality"], np.asarray(lens), lay["signs"], lay["rot"], 1024,
                         key_meta="mxfp4")
    _check(gpu, ref)
    # the zero-range window's step blocks have the all-zero scale byte
    assert np.all(gpu["k_mx"][0, 1, 2, 129::2] == 0)


@pytest.mark.parametrize("plan_name,plan", [
    ("one_shot", [[1000, 333, 64]]),
    ("ragged_chunks", [[7, 1, 31], [1, 40, 2], [100, 3, 5], [31, 200, 26], [900, 100, 0]]),
])
def test_mx_chunked_append_equals_one_shot(plan_name, plan):
    import gpu_helpers as gh
    lens = [1000, 333, 64]
    lay = gen_layer(workload("omni7b_32k"), 2, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :2].copy(), lay["v"][:, :2].copy()
    cache = gh.new_cache(3, 2, 14, 1024, lay["signs"], lay["rot"], key_meta="mxfp4")
    _announce(f"mx append plan={plan_name}")
    done = gh.append_chunks(cache, k, v, lay["modality"], lens, plan, exact=True)
    assert list(done) == lens
    got = gh.cache_to_numpy(cache)
    ref = quantize_layer(k, v, lay["modality"], np.asarray(lens), lay["signs"], lay["rot"], 1024, key_meta="mxfp4")
    _check(got, ref, KEY_FIELDS + ("v_codes", "v_norm", "modality"))
    assert np.array_equal(got["seq_lens"], np.asarray(lens, np.int32))


def _decode_case(wl_name, lens, layer=0, H=None, Hq=None, mfma=True):
    import gpu_helpers as gh
    wl = workload(wl_name)
    lay = gen_layer(wl, layer, lengths=np.asarray(lens, np.int32), n_tokens=max(max(lens), 1))
    k, v = lay["k"], lay["v"]
    if H is not None:
        k, v = k[:, :H].copy(), v[:, :H].copy()
    Hkv = k.shape[1]
    Hq = Hq or wl.num_q_heads * Hkv // wl.num_kv_heads
    q = gen_queries(wl.wid, layer, len(lens), Hq)
    cap = max(32, -(-max(lens) // 32) * 32)
    cache = gh.new_cache(len(lens), Hkv, Hq, cap, lay["signs"], lay["rot"], key_meta="mxfp4")
    _announce(f"mx decode {wl_name} lens={list(lens)[:6]} H={Hkv} Hq={Hq}")
    gh.append_chunks(cache, k, v, lay["modality"], lens, [list(lens)], exact=not mfma)
    out = gh.decode(cache, q, lens)
    arrays = gh.cache_to_numpy(cache)
    return out, arrays, lay, q, k, v


def test_mx_decode_tiny_and_ragged_gqa7():
    import gpu_helpers as gh
    out, arrays, lay, q, _, _ = _decode_case("tiny_1k", [1024])
    ref = decode_layer(arrays, q, np.asarray([1024]), lay["signs"], lay["rot"], SM)
    r = gh.attention_close(out, ref)
    print(f"mx tiny worst err / norm = {r:.2e}")
    assert r <= TOL
    lens = [1000, 517, 33, 1, 64, 2049, 0]
    out, arrays, lay, q, _, _ = _decode_case("omni7b_32k", lens, H=2, Hq=14)
    ref = decode_layer(arrays, q, np.asarray(lens), lay["signs"], lay["rot"], SM)
    assert np.all(out[6] == 0)
    r = gh.attention_close(out[:6], ref[:6])
    print(f"mx ragged worst err / norm = {r:.2e}")
    assert r <= TOL


def test_mx_decode_end_to_end_against_oracle_cache():
    """Oracle-quantized MXFP4 cache decoded by the oracle vs the GPU-quantized one decoded on the GPU."""
    import gpu_helpers as gh
    lens = [1024, 700]
    out, _, lay, q, k, v = _decode_case("omni3b_b4_64k_stream", lens, H=2, Hq=16, mfma=False)
    oc = quantize_layer(k, v, lay["modality"], np.asarray(lens), lay["signs"], lay["rot"], 1024, key_meta="mxfp4")
    ref = decode_layer(oc, q, np.asarray(lens), lay["signs"], lay["rot"], SM)
    r = gh.attention_close(out, ref)
    print(f"mx end-to-end worst err / norm = {r:.2e}")
    assert r <= TOL


def test_mx_full_size_omni7b_32k():
    """The benchmark workload (B1, H4, Hq28, 32768 tokens) with MXFP4 metadata: one prefill append,
    sampled windows bit-exact against the oracle, every decode row against the oracle."""
    import gpu_helpers as gh
    wl = workload("omni7b_32k")
    out, arrays, lay, q, _, _ = _decode_case("omni7b_32k", [wl.seq_len])
    ref = decode_layer(arrays, q, np.asarray([wl.seq_len]), lay["signs"], lay["rot"], SM)
    r = gh.attention_close(out, ref)
    print(f"mx omni7b_32k worst err / norm = {r:.2e}")
    assert r <= TOL
    rng = np.random.default_rng(5)
    for h in range(wl.num_kv_heads):
        for w in sorted(set(rng.integers(0, 1024, 6).tolist()) | {0, 1023}):
            gh.check_window(arrays, lay["k"][0, h], lay["v"][0, h], lay["modality"][0], lay["signs"], lay["rot"],
                            0, h, w, wl.seq_len)
