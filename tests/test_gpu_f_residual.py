"""GPU parity of the captioning protocol's fp16 residual (Sec. 3.1): keys quantized per completed
128-token block, the last 128 values in fp16.

* the rings hold the raw key and value rows of the last min(L, 128) tokens, bit for bit;
* the quantized buffers are byte-identical to those of a cache without the residual;
* decode after every streamed append matches the oracle's mixed-cache attention
  (``oracle.residual.decode_residual``) within 2e-3 of the output norm, at lengths on both sides
  of the 128-token boundaries, with GQA 4 / 7 / 8, ragged batches, an empty sequence, MXFP4 key
  metadata and exact-mode values.
"""

import math

import numpy as np
import pytest

from oracle.residual import decode_layer_residual, residual_boundaries
from synth import gen_layer, gen_queries, workload

pytestmark = pytest.mark.gpu
TOL = 2e-3
SM = 1 / math.sqrt(128)
R = 128


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _layer(wl_name, lens, H=None, layer=0):
    wl = workload(wl_name)
    n = max(max(lens), 1)
    lay = gen_layer(wl, layer, lengths=np.asarray(lens, np.int32), n_tokens=n)
    k, v = lay["k"], lay["v"]
    if H is not None:
        k, v = k[:, :H].copy(), v[:, :H].copy()
    return wl, lay, k, v


def _new_cache(B, H, Hq, cap, lay, key_meta="fp16", residual=R):
    import torch

    import paper_2609_11582_amd as okvq
    return okvq.KVCache(B, H, Hq, cap, torch.from_numpy(np.asarray(lay["signs"], np.int8)),
                        torch.from_numpy(np.asarray(lay["rot"], np.float32)), key_meta=key_meta, residual=residual)


def _check_rings(arrays, k, v, lens):
    for b, L in enumerate(lens):
        for i in range(max(L - R, 0), L):
            np.testing.assert_array_equal(arrays["k_res"][:, :, i % R][b].view(np.uint16), k[b, :, i].view(np.uint16))
            np.testing.assert_array_equal(arrays["v_res"][:, :, i % R][b].view(np.uint16), v[b, :, i].view(np.uint16))


def _stream_and_decode(wl_name, lens, steps, H=None, Hq=None, key_meta="fp16", exact=False, check_rings=True):
    """Append each sequence in the chunks of `steps`; after every append decode and compare with
    the oracle. Returns the worst error ratio."""
    import gpu_helpers as gh
    wl, lay, k, v = _layer(wl_name, lens, H)
    B, Hkv = k.shape[0], k.shape[1]
    Hq = Hq or wl.group * Hkv
    q = gen_queries(wl.wid, 0, B, Hq)
    cap = max(32, -(-max(lens) // 32) * 32)
    cache = _new_cache(B, Hkv, Hq, cap, lay, key_meta=key_meta)
    cur = np.zeros(B, np.int64)
    worst = 0.0
    for si, step in enumerate(steps):
        target = np.minimum(cur + np.asarray(step), np.asarray(lens))
        _announce(f"residual {wl_name} {key_meta} exact={exact} step {si}: lengths {cur.tolist()} -> "
                  f"{target.tolist()} H={Hkv} Hq={Hq}")
        chunk = (target - cur).tolist()
        done = gh.append_chunks_from(cache, k, v, lay["modality"], cur, chunk, exact=exact)
        cur = done
        out = gh.decode(cache, q, cur.tolist())
        arrays = gh.cache_to_numpy(cache)
        np.testing.assert_array_equal(arrays["seq_lens"], cur.astype(np.int32))
        if check_rings:
            _check_rings(arrays, k, v, cur.tolist())
        ref = decode_layer_residual(arrays, k, v, q, cur, lay["signs"], lay["rot"], SM)
        for b, L in enumerate(cur.tolist()):
            if L == 0:
                assert np.all(out[b] == 0)
        live = [b for b, L in enumerate(cur.tolist()) if L > 0]
        r = gh.attention_close(out[live], ref[live])
        kq = [residual_boundaries(L) for L in cur.tolist()]
        print(f"  lengths {cur.tolist()} (Kq, Vq) {kq}: worst err / norm = {r:.2e}", flush=True)
        assert r <= TOL, (cur.tolist(), r)
        worst = max(worst, r)
    return worst


def test_residual_tiny_streaming_across_block_boundaries():
    """Lengths 1, 77, 127, 128, 129, 200, 255, 256, 300, 1000, 1024 (GQA 4)."""
    steps = [[1], [76], [50], [1], [1], [71], [55], [1], [44], [700], [24]]
    _stream_and_decode("tiny_1k", [1024], steps)


def test_residual_ragged_gqa7_with_empty_sequence():
    lens = [1000, 129, 0, 128, 2049, 300]
    steps = [[64, 64, 0, 64, 64, 64], [100, 1, 0, 64, 1000, 100], [836, 64, 0, 0, 985, 136]]
    _stream_and_decode("omni7b_32k", lens, steps, H=2, Hq=14)


def test_residual_mxfp4_gqa8():
    lens = [700, 255]
    steps = [[130, 127], [300, 1], [270, 127]]
    _stream_and_decode("omni3b_b4_64k_stream", lens, steps, H=2, Hq=16, key_meta="mxfp4")


def test_residual_exact_values():
    lens = [333]
    steps = [[200], [5], [128]]
    _stream_and_decode("tiny_1k", lens, steps, exact=True)


def test_residual_codes_match_plain_cache():
    """The residual changes what decode reads, not what append writes: every quantized byte equals
    that of a cache without it, after the same appends."""
    import gpu_helpers as gh
    lens = [777, 300]
    wl, lay, k, v = _layer("omni7b_32k", lens, H=2)
    caches = []
    for residual in (R, 0):
        c = _new_cache(2, 2, 14, 800, lay, residual=residual)
        _announce(f"residual codes vs plain: residual={residual}")
        gh.append_chunks_from(c, k, v, lay["modality"], np.zeros(2, np.int64), [500, 300])
        gh.append_chunks_from(c, k, v, lay["modality"], np.array([500, 300]), [277, 0])
        caches.append(gh.cache_to_numpy(c))
    for name in ("k_codes", "v_codes", "k_norm", "v_norm", "k_min", "k_step", "modality", "k_stage", "seq_lens"):
        np.testing.assert_array_equal(caches[0][name], caches[1][name], err_msg=name)
    _check_rings(caches[0], k, v, lens)
