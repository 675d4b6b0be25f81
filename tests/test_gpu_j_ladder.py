"""GPU parity of the bit-width ladder (b-bit keys and values, b = 2, 3, 4; Tab. 3 K3/V2, Tab. 5
K2V2 / K3V3 / K4V4) against oracle.ladder: key codes, window metadata and norms bit-exact (the
method's keys and TurboQuant keys, every width, ragged and degenerate rows, and the benchmark layer
at full size), value codes and norms
bit-exact in the exact fp32 order and within the rotation band in the matrix-core mode, and decode within 2e-3 of the output norm -- over the GPU-written
cache and end to end against the oracle-written one -- for several width pairs, ragged GQA 7 with
an empty sequence, and the benchmark layer (4 KV heads, 28 query heads, 32768 tokens)."""

import math

import numpy as np
import pytest

from oracle.ladder import decode_layer_bits, quantize_layer_bits
from synth import gen_layer, gen_queries, workload

pytestmark = pytest.mark.gpu
TOL = 2e-3
SM = 1 / math.sqrt(128)


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _arrays(cache):
    return {n: t.cpu().numpy() for n, t in cache.views().items() if n != "seq_lens"}


def _same(a, b, name):
    if a.dtype == np.float16:
        a, b = a.view(np.uint16), b.view(np.uint16)
    mism = np.argwhere(a != b)
    assert len(mism) == 0, f"{name}: {len(mism)} mismatches, first at {mism[:5].tolist()}"


@pytest.mark.parametrize("meta", ["fp16", "turboquant"])
@pytest.mark.parametrize("bits", [2, 3, 4])
def test_ladder_codes_bit_exact(bits, meta):
    import gpu_helpers as gh
    lens = [1000, 37, 64, 1, 0, 95]
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 5, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :2].copy(), lay["v"][:, :2].copy()
    k[0, 0, 5] = 0                       # zero-norm token
    k[2, 0, :32, :] = np.float16(60000)  # saturated norm, zero-range window
    k[3, 1, 0, 7] = np.float16(-0.0)
    v[0, 1, 9] = 0
    cap = 1024
    _announce(f"ladder codes K{bits}V{bits} {meta} lens={lens}")
    cache = gh.ladder_cache(k, v, lay["modality"], lens, lay["signs"], lay["rot"], cap, 14, bits, bits, meta)
    got = _arrays(cache)
    ref = quantize_layer_bits(k, v, lay["modality"], lens, lay["signs"], lay["rot"], cap, bits, bits, meta)
    for name in ref:
        _same(got[name], ref[name], name)


@pytest.mark.parametrize("bits,meta", [(2, "fp16"), (3, "fp16"), (4, "fp16"), (3, "turboquant"), (4, "turboquant")],
                         ids=["K2_fp16", "K3_fp16", "K4_fp16", "K3_tq", "K4_tq"])
def test_ladder_keys_full_size_bit_exact(bits, meta):
    """The benchmark layer (32768 tokens, 4 KV heads) through the stateless key call the benchmark
    times: codes, window minimum / step and norms of KV heads 0 and 3 equal the oracle's bytes."""
    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    import torch
    from oracle.ladder import pack_bits, quantize_keys_bits_fmt, quantize_keys_tq_bits_fmt
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 0)
    lens = [int(x) for x in lay["lens"]]
    B, H, N, _ = lay["k"].shape
    _announce(f"ladder keys full size K{bits} {meta} lens={lens}")
    cache = okvq.KVCache(B, H, 28, wl.capacity, torch.from_numpy(lay["signs"]),
                         torch.from_numpy(np.ascontiguousarray(lay["rot"], np.float32)), key_meta=meta,
                         key_bits=bits, value_bits=bits)
    vw = cache.views()
    kd = gh.f16dev(lay["k"])
    if meta == "fp16":
        okvq.okvq_quantize_keys(cache.dims, kd, N, lens, cache.key_signs, vw["k_codes"], vw["k_min"], vw["k_step"],
                                vw["k_norm"])
    else:
        okvq.okvq_quantize_keys_tq(cache.dims, kd, N, lens, cache.key_signs, vw["k_codes"], vw["k_norm"])
    torch.cuda.synchronize()
    got = _arrays(cache)
    for b, L in enumerate(lens):
        for h in (0, 3):
            if meta == "fp16":
                kq = quantize_keys_bits_fmt(lay["k"][b, h], L, lay["signs"], bits)
                nwl = kq["codes"].shape[0] // 32
                _same(got["k_min"][b, h, :nwl], kq["m16"], f"k_min[{b},{h}]")
                _same(got["k_step"][b, h, :nwl], kq["step16"], f"k_step[{b},{h}]")
            else:
                kq = quantize_keys_tq_bits_fmt(lay["k"][b, h], L, lay["signs"], bits)
            npad = kq["codes"].shape[0]
            _same(got["k_codes"][b, h, :npad], pack_bits(kq["codes"], bits), f"k_codes[{b},{h}]")
            _same(got["k_norm"][b, h, :npad], kq["n16"], f"k_norm[{b},{h}]")


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_ladder_values_full_size_matrix_core(bits):
    """The benchmark layer (32768 tokens) through the stateless value call in the matrix-core mode the
    benchmark times: KV head 3's norms bit-exact and its codes within the band rule of the exact
    order (the modality map of the workload, audio runs inside video chunks and the text tail)."""
    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    import torch
    from oracle.ladder import quantize_values_bits_fmt
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 0)
    lens = [int(x) for x in lay["lens"]]
    B, H, N, _ = lay["v"].shape
    _announce(f"ladder values full size V{bits} lens={lens}")
    cache = okvq.KVCache(B, H, 28, wl.capacity, torch.from_numpy(lay["signs"]),
                         torch.from_numpy(np.ascontiguousarray(lay["rot"], np.float32)), key_bits=bits, value_bits=bits)
    vw = cache.views()
    okvq.okvq_quantize_values(cache.dims, gh.f16dev(lay["v"]), gh.dev(np.ascontiguousarray(lay["modality"], np.uint8)), N,
                              lens, cache.v_rot, 0, vw["v_codes"], vw["v_norm"])
    torch.cuda.synchronize()
    got = _arrays(cache)
    b, h, L = 0, 3, lens[0]
    ref = quantize_values_bits_fmt(lay["v"][b, h], lay["modality"][b], lay["rot"], L, bits)
    _same(got["v_norm"][b, h, :L], ref["n16"], "v_norm")
    diff, band = gh.band_compare_bits(got["v_codes"][b, h], lay["v"][b, h], lay["modality"][b], lay["rot"], L, bits)
    print(f"V{bits} full size: {diff} codes differ, {band} in the band", flush=True)


CASES = [(2, 2, "fp16"), (3, 3, "fp16"), (4, 4, "fp16"), (3, 2, "turboquant"), (4, 4, "turboquant"),
         (2, 4, "fp16"), (4, 3, "turboquant")]


@pytest.mark.parametrize("kb,vb,meta", CASES, ids=[f"K{a}V{b}_{m}" for a, b, m in CASES])
def test_ladder_decode_ragged_gqa7(kb, vb, meta):
    import gpu_helpers as gh
    lens = [1000, 517, 33, 1, 0, 2049, 300]
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 3, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :2].copy(), lay["v"][:, :2].copy()
    q = gen_queries(wl.wid, 3, len(lens), 14)
    cap = -(-max(lens) // 32) * 32
    _announce(f"ladder decode K{kb}V{vb} {meta} lens={lens}")
    cache = gh.ladder_cache(k, v, lay["modality"], lens, lay["signs"], lay["rot"], cap, 14, kb, vb, meta)
    out = gh.decode(cache, q, lens)
    arrays = _arrays(cache)
    ref = decode_layer_bits(arrays, q, lens, lay["signs"], lay["rot"], SM, kb, vb)
    assert np.all(out[4] == 0)
    live = [b for b, L in enumerate(lens) if L > 0]
    r = gh.attention_close(out[live], ref[live])
    print(f"K{kb}V{vb} {meta}: worst err / norm = {r:.2e}", flush=True)
    assert r <= TOL
    # the codecs are bit-exact, so the oracle-written cache is the same cache
    oc = quantize_layer_bits(k, v, lay["modality"], lens, lay["signs"], lay["rot"], cap, kb, vb, meta)
    for name in oc:
        _same(arrays[name], oc[name], name)


@pytest.mark.parametrize("kb,vb,meta", [(3, 3, "fp16"), (4, 2, "turboquant")], ids=["K3V3_fp16", "K4V2_tq"])
def test_ladder_decode_several_windows_per_wave(kb, vb, meta):
    """Lengths long enough that every wave of a split takes several windows (GQA 8)."""
    import gpu_helpers as gh
    lens = [20000, 7777]
    wl = workload("omni3b_b4_64k_stream")
    lay = gen_layer(wl, 1, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    q = gen_queries(wl.wid, 1, 2, 16)
    cap = -(-max(lens) // 32) * 32
    _announce(f"ladder decode K{kb}V{vb} {meta} lens={lens}")
    cache = gh.ladder_cache(lay["k"], lay["v"], lay["modality"], lens, lay["signs"], lay["rot"], cap, 16, kb, vb, meta)
    out = gh.decode(cache, q, lens)
    ref = decode_layer_bits(_arrays(cache), q, lens, lay["signs"], lay["rot"], SM, kb, vb)
    r = gh.attention_close(out, ref)
    print(f"K{kb}V{vb} {meta} long: worst err / norm = {r:.2e}", flush=True)
    assert r <= TOL


@pytest.mark.parametrize("kb,vb,meta", [(2, 2, "fp16"), (4, 4, "fp16"), (3, 2, "turboquant")],
                         ids=["K2V2_fp16", "K4V4_fp16", "K3V2_tq"])
def test_ladder_decode_full_size(kb, vb, meta):
    """The benchmark layer: every query head of two KV heads against the oracle."""
    import gpu_helpers as gh
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 0)
    lens = [int(x) for x in lay["lens"]]
    q = gen_queries(wl.wid, 0, 1, 28)
    _announce(f"ladder decode omni7b_32k K{kb}V{vb} {meta}")
    cache = gh.ladder_cache(lay["k"], lay["v"], lay["modality"], lens, lay["signs"], lay["rot"], wl.capacity, 28, kb,
                            vb, meta)
    out = gh.decode(cache, q, lens)
    arrays = _arrays(cache)
    sub = {n: (a[:, [0, 3]] if a.ndim >= 3 and n != "modality" else a) for n, a in arrays.items()}
    ref = decode_layer_bits(sub, q[:, list(range(0, 7)) + list(range(21, 28))], lens, lay["signs"], lay["rot"], SM,
                            kb, vb)
    rows = list(range(0, 7)) + list(range(21, 28))
    r = gh.attention_close(out[:, rows], ref)
    print(f"full size K{kb}V{vb} {meta}: worst err / norm = {r:.2e}", flush=True)
    assert r <= TOL


def test_ladder_300_sequences_and_both_value_modes():
    """More sequences than one codec launch's length table (256): every sequence's codes bit-exact
    in the exact order; the matrix-core mode gives the same norms and codes within the band."""
    import torch

    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    rng = np.random.default_rng(3)
    B = 300
    lens = [int(x) for x in rng.integers(0, 65, B)]
    lens[7] = 64
    wl = workload("tiny_1k")
    lay = gen_layer(wl, 2, lengths=np.full(B, 64, np.int32), n_tokens=64)
    k, v = lay["k"], lay["v"]                              # [300][1][64][128]
    mod = rng.integers(0, 3, (B, 64)).astype(np.uint8)     # all three rotations in every window
    _announce(f"ladder K3V3, {B} sequences")
    cache = gh.ladder_cache(k, v, mod, lens, lay["signs"], lay["rot"], 64, 4, 3, 3, "fp16")
    got = _arrays(cache)
    ref = quantize_layer_bits(k, v, mod, lens, lay["signs"], lay["rot"], 64, 3, 3, "fp16")
    for name in ref:
        _same(got[name], ref[name], name)
    vw = cache.views()
    vc2 = torch.zeros_like(vw["v_codes"])
    vn2 = torch.zeros_like(vw["v_norm"])
    okvq.okvq_quantize_values(cache.dims, gh.f16dev(v), gh.dev(np.ascontiguousarray(mod, np.uint8)), 64, lens,
                              cache.v_rot, 0, vc2, vn2)
    torch.cuda.synchronize()
    _same(vn2.cpu().numpy(), ref["v_norm"], "v_norm (matrix-core mode)")
    vc2 = vc2.cpu().numpy()
    diff = 0
    for b, L in enumerate(lens):
        if L:
            diff += gh.band_compare_bits(vc2[b, 0], v[b, 0], mod[b], lay["rot"], L, 3)[0]
        assert not np.any(vc2[b, 0, L:])
    print(f"matrix-core mode: {diff} of {128 * sum(lens)} codes differ (all in the band)", flush=True)


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_ladder_values_matrix_core_mode(bits):
    """The matrix-core value codec: norms bit-exact, codes within the rotation band of the exact
    order, slots beyond a length untouched; ragged lengths over several 128-token tiles, an empty
    sequence, a zero row and the workload's modality runs; then decode over that cache."""
    import gpu_helpers as gh
    lens = [1000, 130, 0, 1, 257, 64]
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 4, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :2].copy(), lay["v"][:, :2].copy()
    v[0, 1, 9] = 0
    cap = 1024
    _announce(f"ladder values, matrix-core mode, {bits} bits, lens={lens}")
    cache = gh.ladder_cache(k, v, lay["modality"], lens, lay["signs"], lay["rot"], cap, 14, 2, bits, "fp16",
                            value_flags=0)
    got = _arrays(cache)
    ref = quantize_layer_bits(k, v, lay["modality"], lens, lay["signs"], lay["rot"], cap, 2, bits, "fp16")
    _same(got["v_norm"], ref["v_norm"], "v_norm")
    diff = band = 0
    for b, L in enumerate(lens):
        for h in range(2):
            if L:
                d, n = gh.band_compare_bits(got["v_codes"][b, h], v[b, h], lay["modality"][b], lay["rot"], L, bits)
                diff, band = diff + d, band + n
            assert not np.any(got["v_codes"][b, h, L:])
    print(f"{bits} bits: {diff} codes differ, {band} in the band", flush=True)
    q = gen_queries(wl.wid, 4, len(lens), 14)
    out = gh.decode(cache, q, lens)
    dref = decode_layer_bits(got, q, lens, lay["signs"], lay["rot"], SM, 2, bits)
    live = [b for b, L in enumerate(lens) if L > 0]
    assert np.all(out[2] == 0)
    assert gh.attention_close(out[live], dref[live]) <= TOL


APPEND_CASES = [(2, 2, "fp16"), (3, 3, "fp16"), (4, 4, "fp16"), (2, 4, "fp16"), (3, 2, "turboquant"),
                (4, 4, "turboquant")]
APPEND_PLANS = {
    "one_shot": [[1000, 333, 64, 0]],
    "ragged_chunks": [[7, 1, 31, 0], [1, 40, 2, 0], [100, 3, 5, 0], [31, 200, 26, 0], [900, 100, 0, 0]],
    "single_tokens_then_bulk": [[1, 1, 1, 0]] * 40 + [[1000, 1000, 1000, 0]],
}


@pytest.mark.parametrize("plan_name", list(APPEND_PLANS))
@pytest.mark.parametrize("kb,vb,meta", APPEND_CASES, ids=[f"K{a}V{b}_{m}" for a, b, m in APPEND_CASES])
def test_ladder_append_chunked_equals_oracle(kb, vb, meta, plan_name):
    """Appending in any chunking gives the bytes of the one-shot oracle quantization: the method's
    keys re-quantize the open window from the stage, which then holds the raw keys of the new open
    window; TurboQuant keys and values are per token. An empty sequence stays empty."""
    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    import torch
    lens = [1000, 333, 64, 0]
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 6, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :2].copy(), lay["v"][:, :2].copy()
    k[0, 1, 40] = 0                       # a zero-norm key inside a window
    k[1, 0, 64:96, :] = np.float16(60000)  # saturated norm, zero-range window
    cap = 1024
    cache = okvq.KVCache(len(lens), 2, 14, cap, torch.from_numpy(lay["signs"]),
                         torch.from_numpy(np.ascontiguousarray(lay["rot"], np.float32)), key_meta=meta,
                         key_bits=kb, value_bits=vb)
    _announce(f"ladder append K{kb}V{vb} {meta} plan={plan_name}")
    done = gh.append_chunks(cache, k, v, lay["modality"], lens, APPEND_PLANS[plan_name], exact=True)
    assert list(done) == lens
    got = _arrays(cache)
    assert np.array_equal(cache.views()["seq_lens"].cpu().numpy(), np.asarray(lens, np.int32))
    ref = quantize_layer_bits(k, v, lay["modality"], lens, lay["signs"], lay["rot"], cap, kb, vb, meta)
    for name in ref:
        _same(got[name], ref[name], name)
    if meta == "fp16":
        for b, L in enumerate(lens):
            o = (L // 32) * 32
            np.testing.assert_array_equal(got["k_stage"][b, :, :L - o].view(np.uint16), k[b, :, o:L].view(np.uint16))


@pytest.mark.parametrize("kb,vb,meta", [(3, 3, "fp16"), (4, 2, "turboquant")], ids=["K3V3_fp16", "K4V2_turboquant"])
def test_ladder_append_mfma_equals_stateless_then_decode(kb, vb, meta):
    """Matrix-core values: a chunked append writes the bytes of the stateless matrix-core call
    (the codes of a token depend on its row alone); decode of the appended cache then matches the
    oracle, at every step of a streaming append."""
    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    import torch
    lens = [777, 96]
    wl = workload("omni3b_b4_64k_stream")
    lay = gen_layer(wl, 1, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :2].copy(), lay["v"][:, :2].copy()
    cap = 1024
    cache = okvq.KVCache(2, 2, 16, cap, torch.from_numpy(lay["signs"]),
                         torch.from_numpy(np.ascontiguousarray(lay["rot"], np.float32)), key_meta=meta,
                         key_bits=kb, value_bits=vb)
    _announce(f"ladder append mfma K{kb}V{vb} {meta}")
    cur = np.zeros(2, np.int64)
    for s, step in enumerate([[13, 5], [300, 50], [464, 41]]):
        cur = gh.append_chunks_from(cache, k, v, lay["modality"], cur, np.minimum(step, np.asarray(lens) - cur))
        q = gen_queries(wl.wid, 1, 2, 16, step=s + 1)
        out = gh.decode(cache, q, cur.tolist())
        ref = decode_layer_bits(_arrays(cache), q, cur.tolist(), lay["signs"], lay["rot"], SM, kb, vb)
        assert gh.attention_close(out, ref) <= TOL
    st = gh.ladder_cache(k, v, lay["modality"], lens, lay["signs"], lay["rot"], cap, 16, kb, vb, meta, value_flags=0)
    got, want = _arrays(cache), _arrays(st)
    for name in want:
        if name != "k_stage":
            _same(got[name], want[name], name)
