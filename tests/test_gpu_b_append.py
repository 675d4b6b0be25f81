"""GPU append: any chunking of a sequence gives the bytes of one-shot quantization (bit-exact)."""

import numpy as np
import pytest

from oracle.cache import quantize_layer
from synth import gen_layer, workload

pytestmark = pytest.mark.gpu

FIELDS = ("k_codes", "k_norm", "k_min", "k_step", "v_codes", "v_norm", "modality")


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _compare(got, ref, lens, exact_values=True):
    B = len(lens)
    for name in FIELDS:
        if name == "v_codes" and not exact_values:
            continue
        a, b = got[name], ref[name]
        if a.dtype == np.float16:
            a, b = a.view(np.uint16), b.view(np.uint16)
        assert np.array_equal(a, b), f"{name}: {(a != b).sum()} mismatching entries"
    assert np.array_equal(got["seq_lens"], np.asarray(lens, np.int32))


@pytest.mark.parametrize("plan_name,plan", [
    ("one_shot", [[1000, 333, 64]]),
    ("window_aligned", [[512, 128, 32]] * 2 + [[512, 512, 512]]),
    ("ragged_chunks", [[7, 1, 31], [1, 40, 2], [100, 3, 5], [31, 200, 26], [900, 100, 0]]),
    ("single_tokens_then_bulk", [[1, 1, 1]] * 40 + [[1000, 1000, 1000]]),
])
def test_chunked_append_equals_one_shot(plan_name, plan):
    import gpu_helpers as gh
    lens = [1000, 333, 64]
    wl = workload("omni7b_32k")
    lay = gen_layer(wl, 2, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :2].copy(), lay["v"][:, :2].copy()
    cap = 1024
    cache = gh.new_cache(3, 2, 14, cap, lay["signs"], lay["rot"])
    _announce(f"append plan={plan_name}")
    done = gh.append_chunks(cache, k, v, lay["modality"], lens, plan, exact=True)
    assert list(done) == lens
    got = gh.cache_to_numpy(cache)
    ref = quantize_layer(k, v, lay["modality"], np.asarray(lens), lay["signs"], lay["rot"], cap)
    _compare(got, ref, lens)
    # the stage holds the raw keys of each open window
    for b, L in enumerate(lens):
        open_ = (L // 32) * 32
        n = L - open_
        np.testing.assert_array_equal(got["k_stage"][b, :, :n].view(np.uint16), k[b, :, open_:L].view(np.uint16))


def test_mfma_append_matches_stateless_mfma():
    """Default (MFMA) value mode: chunked append gives the same bytes as the stateless MFMA call."""
    import gpu_helpers as gh
    lens = [777, 96]
    wl = workload("omni3b_b4_64k_stream")
    lay = gen_layer(wl, 1, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    cache = gh.new_cache(2, 2, 16, 1024, lay["signs"], lay["rot"])
    _announce("append mfma vs stateless")
    gh.append_chunks(cache, lay["k"], lay["v"], lay["modality"], lens, [[13, 5], [300, 50], [500, 41]])
    got = gh.cache_to_numpy(cache)
    st = gh.quantize_stateless(lay["k"], lay["v"], lay["modality"], lens, lay["signs"], lay["rot"], 1024, 16)
    for name in ("k_codes", "k_norm", "k_min", "k_step", "v_codes", "v_norm", "modality"):
        assert np.array_equal(got[name], st[name]), name
    # the fused launch advanced the lengths and returned its work-group counter to zero
    assert np.array_equal(got["seq_lens"], np.asarray(lens, np.int32))
    assert int(cache.buffers["seq_lens"][-1].item()) == 0


def test_streaming_append_then_decode_each_step():
    """omni3b-like streaming: prefill, then append 512-token audio-visual chunks and decode each step."""
    import math

    import gpu_helpers as gh
    from oracle.cache import decode_layer
    from synth import gen_queries
    wl = workload("omni3b_b4_64k_stream")
    pre, step, steps = 2048, 512, 3
    total = pre + step * steps
    lay = gen_layer(wl, 0, lengths=np.full(2, total, np.int32), n_tokens=total)
    cache = gh.new_cache(2, 2, 16, 4096, lay["signs"], lay["rot"])
    _announce("streaming append + decode")
    gh.append_chunks(cache, lay["k"][:2], lay["v"][:2], lay["modality"][:2], [pre, pre], [[pre, pre]])
    cur = pre
    for s in range(steps):
        plan = [[step, step]]
        k = lay["k"][:2, :, :cur + step]
        v = lay["v"][:2, :, :cur + step]
        # append only the new chunk
        import paper_2609_11582_amd as okvq
        import torch
        kn = np.ascontiguousarray(k[:, :, cur:])
        vn = np.ascontiguousarray(v[:, :, cur:])
        mn = np.ascontiguousarray(lay["modality"][:2, cur:cur + step])
        okvq.okvq_append(cache, [cur, cur], gh.f16dev(kn), gh.f16dev(vn), gh.dev(mn), [step, step],
                         gh.dev(np.array([step, step], np.int32)), step)
        torch.cuda.synchronize()
        cur += step
        q = gen_queries(wl.wid, 0, 2, 16, step=s + 1)
        out = gh.decode(cache, q, [cur, cur])
        ref = decode_layer(gh.cache_to_numpy(cache), q, np.array([cur, cur]), lay["signs"], lay["rot"],
                           1 / math.sqrt(128))
        assert gh.attention_close(out, ref) <= 2e-3
    del plan


def test_append_and_decode_beyond_256_sequences():
    """300 sequences: append and decode split the batch into several launches (256 sequences each);
    every sequence matches the one-shot oracle quantization and the decode oracle."""
    import math

    import gpu_helpers as gh
    from oracle.cache import decode_layer
    from synth import gen_queries
    rng = np.random.default_rng(5)
    lens = rng.integers(1, 80, 300).tolist()
    wl = workload("tiny_1k")
    lay = gen_layer(wl, 3, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    cache = gh.new_cache(300, 1, 4, 96, lay["signs"], lay["rot"])
    _announce("append B=300 (two launches)")
    gh.append_chunks(cache, lay["k"], lay["v"], lay["modality"], lens, [[40] * 300, [100] * 300])
    got = gh.cache_to_numpy(cache)
    assert np.array_equal(got["seq_lens"], np.asarray(lens, np.int32))
    assert int(cache.buffers["seq_lens"][-1].item()) == 0
    st = gh.quantize_stateless(lay["k"], lay["v"], lay["modality"], lens, lay["signs"], lay["rot"], 96, 4)
    for name in ("k_codes", "k_norm", "k_min", "k_step", "v_codes", "v_norm", "modality"):
        assert np.array_equal(got[name], st[name]), name
    ref = quantize_layer(lay["k"], lay["v"], lay["modality"], np.asarray(lens), lay["signs"], lay["rot"], 96)
    for name in ("k_codes", "k_norm", "k_min", "k_step"):
        a, b = got[name], ref[name]
        if a.dtype == np.float16:
            a, b = a.view(np.uint16), b.view(np.uint16)
        assert np.array_equal(a, b), name
    q = gen_queries(wl.wid, 3, 300, 4)
    out = gh.decode(cache, q, lens)
    dec = decode_layer(got, q, np.asarray(lens), lay["signs"], lay["rot"], 1 / math.sqrt(128),
                       heads={(b, 0) for b in (0, 1, 255, 256, 299)})
    assert gh.attention_close(out, dec) <= 2e-3


def test_append_reports_a_value_wait_that_gave_up(monkeypatch):
    """The value codec's waves wait for each other with a bounded number of polls. Forced from the
    host to give up at once (OKVQ_CODEC_SPIN_LIMIT=0, no poll), every kernel still ends normally and
    the append marks the cache's status word; a normal append leaves it at zero. (The tile launch
    holds the only such wait: the test forces it for these medium-sized appends.)"""
    import torch

    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    wl = workload("omni7b_32k")
    lens = [700, 300]
    lay = gen_layer(wl, 0, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :2].copy(), lay["v"][:, :2].copy()
    cache = gh.new_cache(2, 2, 14, 1024, lay["signs"], lay["rot"])
    monkeypatch.setenv("OKVQ_APPEND_PATH", "tile")
    print("[gpu-case] append, normal wait", flush=True)
    gh.append_chunks(cache, k, v, lay["modality"], lens, [[256, 256]])
    assert okvq.okvq_cache_status(cache) == 0
    monkeypatch.setenv("OKVQ_CODEC_SPIN_LIMIT", "0")
    print("[gpu-case] append, wait bound 0", flush=True)
    cur = gh.append_chunks_from(cache, k, v, lay["modality"], [256, 256], [444, 44])
    torch.cuda.synchronize()
    assert list(cur) == lens
    assert cache.views()["seq_lens"].cpu().tolist() == lens      # the lengths still advanced
    assert okvq.okvq_cache_status(cache) == 1
    assert int(cache["seq_lens"][2].item()) == 0                 # the work-group counter is back at zero
