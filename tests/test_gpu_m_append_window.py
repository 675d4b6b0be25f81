"""GPU: the window-parallel append (one launch over the key windows an append touches, with the
residual rings and the length update) writes the bytes of the tile launch, for every chunking:
fp16 window metadata and TurboQuant keys, per-modality and single global rotations, with and
without the fp16 residual, ragged batches with empty and one-token sequences, zero-norm rows and a
zero-range window. The final cache also equals the stateless (one-shot) calls."""

import numpy as np
import pytest

from synth import gen_layer, workload

pytestmark = pytest.mark.gpu

LENS = [1000, 333, 64, 0, 31, 1]
PLANS = {
    "single_tokens_then_bulk": [[1] * 6] * 40 + [[1000] * 6],
    "ragged_chunks": [[7, 1, 31, 0, 5, 1], [1, 40, 2, 0, 26, 0], [100, 3, 5, 0, 0, 0], [31, 200, 26, 0, 0, 0],
                      [900, 100, 0, 0, 0, 0]],
    "stream_512": [[488, 45, 64, 0, 31, 1]] + [[512, 288, 0, 0, 0, 0]],
    "window_crossing": [[33, 64, 1, 0, 30, 1], [64, 65, 63, 0, 1, 0], [95, 204, 0, 0, 0, 0], [808, 0, 0, 0, 0, 0]],
}


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _layer(seed):
    wl = workload("omni3b_b4_64k_stream")
    lay = gen_layer(wl, seed, lengths=np.asarray(LENS, np.int32), n_tokens=max(LENS))
    k, v, mod = lay["k"][:, :2].copy(), lay["v"][:, :2].copy(), lay["modality"].copy()
    k[0, 0, 5] = 0                       # zero-norm key
    v[0, 1, 9] = 0                       # zero-norm value
    k[1, 0, 64:96, :] = np.float16(60000)  # saturated norm, zero-range window
    mod[4, 3] = 2                        # a text token among audio-visual ones
    return k, v, mod, lay["signs"], lay["rot"]


def _appended(monkeypatch, path, meta, plan, residual=0, flags=0, seed=2, timed=None):
    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    import torch
    k, v, mod, signs, rot = _layer(seed)
    monkeypatch.setenv("OKVQ_APPEND_PATH", path)
    cache = okvq.KVCache(len(LENS), 2, 16, 1024, torch.from_numpy(np.asarray(signs, np.int8)),
                         torch.from_numpy(np.asarray(rot, np.float32)), key_meta=meta, residual=residual)
    done = gh.append_chunks(cache, k, v, mod, LENS, plan, flags=flags, timed=timed)
    assert list(done) == LENS
    out = gh.cache_to_numpy(cache)
    out["ticket"] = int(cache.buffers["seq_lens"][len(LENS)].item())
    return out, (k, v, mod, signs, rot)


def _same(a, b, name):
    a, b = np.asarray(a), np.asarray(b)
    if a.dtype == np.float16:
        a, b = a.view(np.uint16), b.view(np.uint16)
    mism = np.argwhere(a != b)
    assert len(mism) == 0, f"{name}: {len(mism)} mismatches, first at {mism[:5].tolist()}"


@pytest.mark.parametrize("plan_name", list(PLANS))
@pytest.mark.parametrize("meta", ["fp16", "turboquant"])
def test_window_path_equals_tile_path(meta, plan_name, monkeypatch):
    import gpu_helpers as gh
    _announce(f"append window vs tile {meta} plan={plan_name}")
    win, (k, v, mod, signs, rot) = _appended(monkeypatch, "window", meta, PLANS[plan_name])
    tile, _ = _appended(monkeypatch, "tile", meta, PLANS[plan_name])
    for name in tile:
        if name != "ticket":
            _same(win[name], tile[name], name)
    assert win["ticket"] == 0
    assert np.array_equal(win["seq_lens"], np.asarray(LENS, np.int32))
    st = gh.quantize_stateless(k, v, mod, LENS, signs, rot, 1024, 16, key_meta=meta)
    for name in st:
        _same(win[name], st[name], name)


@pytest.mark.parametrize("plan_name", ["single_tokens_then_bulk", "window_crossing"])
def test_window_path_residual_rings(plan_name, monkeypatch):
    """With the captioning protocol's fp16 residual the window launch also fills the rings."""
    _announce(f"append window vs tile, residual, plan={plan_name}")
    win, _ = _appended(monkeypatch, "window", "fp16", PLANS[plan_name], residual=128, seed=4)
    tile, _ = _appended(monkeypatch, "tile", "fp16", PLANS[plan_name], residual=128, seed=4)
    for name in tile:
        _same(win[name], tile[name], name)
    assert "k_res" in win and "v_res" in win


def test_window_path_global_rotation(monkeypatch):
    import paper_2609_11582_amd as okvq
    _announce("append window vs tile, global rotation")
    g = okvq.okvq.OKVQ_GLOBAL_ROTATION
    win, _ = _appended(monkeypatch, "window", "fp16", PLANS["ragged_chunks"], flags=g, seed=6)
    tile, _ = _appended(monkeypatch, "tile", "fp16", PLANS["ragged_chunks"], flags=g, seed=6)
    for name in tile:
        _same(win[name], tile[name], name)


@pytest.mark.parametrize("path,plan_name,meta", [("window", "ragged_chunks", "fp16"), ("tile", "stream_512", "fp16"),
                                                ("window", "window_crossing", "turboquant")])
def test_timed_append_writes_the_same_bytes(path, plan_name, meta, monkeypatch):
    """okvq_append_timed (events bound to the codec launch) writes the bytes of okvq_append and
    gives one positive duration per step."""
    _announce(f"timed append {path} {meta} plan={plan_name}")
    ms = []
    timed, _ = _appended(monkeypatch, path, meta, PLANS[plan_name], seed=8, timed=ms)
    plain, _ = _appended(monkeypatch, path, meta, PLANS[plan_name], seed=8)
    for name in plain:
        _same(timed[name], plain[name], name)
    assert len(ms) > 0 and all(0.0 < x < 100.0 for x in ms), ms
