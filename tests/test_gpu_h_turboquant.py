"""GPU parity of the TurboQuant baseline (Eq. 2, Eq. 3): key codes and norms bit-exact against the
oracle (stateless calls and chunked appends), decode within 2e-3 of the output norm over caches
with TurboQuant keys -- with per-modality value rotations and with the single global rotation
R_m = H that makes the whole cache TurboQuant K2/V2."""

import math

import numpy as np
import pytest

from oracle.cache import decode_layer, quantize_layer
from oracle.hadamard import randomized_hadamard
from synth import gen_layer, gen_queries, gen_signs, workload

pytestmark = pytest.mark.gpu
TOL = 2e-3
SM = 1 / math.sqrt(128)


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _check_keys(gpu, ref):
    for name in ("k_codes", "k_norm"):
        a, b = gpu[name], ref[name]
        if a.dtype == np.float16:
            a, b = a.view(np.uint16), b.view(np.uint16)
        mism = np.argwhere(a != b)
        assert len(mism) == 0, f"{name}: {len(mism)} mismatches, first at {mism[:5].tolist()}"


def test_tq_keys_bit_exact_tiny_and_degenerate():
    import gpu_helpers as gh
    lens = [1000, 37, 64, 1, 0, 95]
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 5, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k = lay["k"]
    k[0, 0, 5] = 0                       # zero-norm token: z = 0, code 1 in every channel
    k[2, 0, :32, :] = np.float16(60000)  # saturated fp16 norm
    k[3, 1, 0, 7] = np.float16(-0.0)
    _announce(f"tq keys lens={lens}")
    gpu = gh.quantize_stateless(k, lay["v"], lay["modality"], lens, lay["signs"], lay["rot"], 1024, 28,
                                key_meta="turboquant")
    ref = quantize_layer(k, lay["v"], lay["modality"], np.asarray(lens), lay["signs"], lay["rot"], 1024,
                         key_meta="turboquant")
    _check_keys(gpu, ref)


@pytest.mark.parametrize("plan", [[[1024]], [[1], [31], [300], [692]]], ids=["one_shot", "chunks"])
def test_tq_append_equals_one_shot(plan):
    import gpu_helpers as gh
    wl = workload("tiny_1k")
    lay = gen_layer(wl, 0)
    cache = gh.new_cache(1, 1, 4, 1024, lay["signs"], lay["rot"], key_meta="turboquant")
    _announce(f"tq append plan={plan}")
    gh.append_chunks(cache, lay["k"], lay["v"], lay["modality"], [1024], plan)
    gpu = gh.cache_to_numpy(cache)
    ref = quantize_layer(lay["k"], lay["v"], lay["modality"], np.array([1024]), lay["signs"], lay["rot"], 1024,
                         key_meta="turboquant")
    _check_keys(gpu, ref)
    np.testing.assert_array_equal(gpu["v_norm"].view(np.uint16), ref["v_norm"].view(np.uint16))
    assert "k_min" not in gpu and "k_mx" not in gpu


@pytest.mark.parametrize("rotation", ["per_modality", "global_hadamard"])
def test_tq_decode_ragged_gqa7(rotation):
    """Lengths with partial windows and an empty sequence; values with the workload's per-modality
    rotations, or with R_m = H for every modality (TurboQuant values: the full K2/V2 baseline)."""
    import gpu_helpers as gh
    lens = [1000, 517, 33, 1, 0, 2049]
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 3, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :2].copy(), lay["v"][:, :2].copy()
    rot = lay["rot"]
    if rotation == "global_hadamard":
        rot = np.stack([randomized_hadamard(gen_signs(77, 3))] * 3).astype(np.float32)
    q = gen_queries(wl.wid, 3, len(lens), 14)
    cap = -(-max(lens) // 32) * 32
    cache = gh.new_cache(len(lens), 2, 14, cap, lay["signs"], rot, key_meta="turboquant")
    _announce(f"tq decode {rotation} lens={lens}")
    gh.append_chunks(cache, k, v, lay["modality"], lens, [list(lens)])
    out = gh.decode(cache, q, lens)
    arrays = gh.cache_to_numpy(cache)
    ref = decode_layer(arrays, q, np.asarray(lens), lay["signs"], rot, SM)
    assert np.all(out[4] == 0)
    live = [b for b, L in enumerate(lens) if L > 0]
    r = gh.attention_close(out[live], ref[live])
    print(f"tq decode {rotation}: worst err / norm = {r:.2e}", flush=True)
    assert r <= TOL
    # the cache itself against the oracle's: keys bit-exact; value codes equal to the exact order
    # except inside the rotation-error band of a threshold (one in-band flip on a token with a large
    # attention weight moves the output by more than the tolerance, so the cache is compared, not a
    # decode of the oracle-quantized cache)
    oc = quantize_layer(k, v, lay["modality"], np.asarray(lens), lay["signs"], rot, cap, key_meta="turboquant")
    _check_keys(arrays, oc)
    np.testing.assert_array_equal(arrays["v_norm"].view(np.uint16), oc["v_norm"].view(np.uint16))
    for b, L in enumerate(lens):
        for h in range(2):
            if L:
                gh.band_compare(arrays["v_codes"][b, h], v[b, h], lay["modality"][b], rot, L)


def test_tq_decode_full_size_sampled_rows():
    """The benchmark layer (4 KV heads, 28 query heads, 32768 tokens) with TurboQuant keys: two
    (sequence, KV head) rows against the oracle."""
    import gpu_helpers as gh
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 0)
    q = gen_queries(wl.wid, 0, 1, 28)
    cache = gh.new_cache(1, 4, 28, 32768, lay["signs"], lay["rot"], key_meta="turboquant")
    _announce("tq decode omni7b_32k")
    gh.append_chunks(cache, lay["k"], lay["v"], lay["modality"], [32768], [[32768]])
    out = gh.decode(cache, q, [32768])
    arrays = gh.cache_to_numpy(cache)
    ref = decode_layer(arrays, q, np.array([32768]), lay["signs"], lay["rot"], SM, heads=[(0, 0), (0, 3)])
    rows = list(range(0, 7)) + list(range(21, 28))
    r = gh.attention_close(out[:, rows], ref[:, rows])
    print(f"tq full size worst err / norm = {r:.2e}", flush=True)
    assert r <= TOL
