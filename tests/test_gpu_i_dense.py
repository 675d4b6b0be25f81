"""GPU parity of the dense fp16 decode-attention baseline (Eq. 1 over an unquantized cache) against
float64 attention over the same fp16 keys and values (oracle.attention.decode_dense), within 2e-3
of the output norm: one and several splits, ragged lengths with an empty sequence, GQA groups
1 / 7 / 8, unused capacity rows holding NaN, a softmax maximum that grows along the sequence (the
lazily moved reference), the timed entry point, and the 131072-token layer of the 30B-like
workload on every row."""

import math

import numpy as np
import pytest

from oracle.cache import decode_layer_dense
from synth import gen_layer, gen_queries, workload

pytestmark = pytest.mark.gpu
TOL = 2e-3
SM = 1 / math.sqrt(128)


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _dense(k, v, q, lens, cap=None, events=None, fill_nan=False):
    """k, v [B][H][N][128] fp16 (numpy) -> the library's dense decode output [B][Hq][128]."""
    import torch

    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    B, H, N, _ = k.shape
    Hq = q.shape[1]
    cap = cap or -(-max(max(lens), 1) // 32) * 32
    kk = np.zeros((B, H, cap, 128), np.float16)
    vv = np.zeros((B, H, cap, 128), np.float16)
    if fill_nan:
        kk[:] = np.float16(np.nan)
        vv[:] = np.float16(np.nan)
    for b, L in enumerate(lens):
        kk[b, :, :L] = k[b, :, :L]
        vv[b, :, :L] = v[b, :, :L]
    dims = okvq.make_dims(B, H, Hq, cap)
    ws = okvq.dense_workspace(dims, max(lens))
    out = torch.full((B, Hq, 128), float("nan"), dtype=torch.float32, device="cuda")
    seq = gh.dev(np.asarray(lens, np.int32))
    okvq.okvq_decode_attention_dense(dims, gh.f16dev(kk), gh.f16dev(vv), seq, list(lens), gh.f16dev(q), SM, out, ws,
                                     events=events)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def _check(out, k, v, q, lens, tag):
    import gpu_helpers as gh
    ref = decode_layer_dense(k, v, q, np.asarray(lens), SM)
    for b, L in enumerate(lens):
        if L == 0:
            assert np.all(out[b] == 0), f"{tag}: sequence {b} of length 0 must give zeros"
    live = [b for b, L in enumerate(lens) if L > 0]
    r = gh.attention_close(out[live], ref[live])
    print(f"{tag}: worst err / norm = {r:.2e}", flush=True)
    assert r <= TOL


@pytest.mark.parametrize("case", ["tiny_1k", "ragged_gqa7", "gqa8_splits", "gqa1"])
def test_dense_decode(case):
    if case == "tiny_1k":
        wl, lens, H, Hq = workload("tiny_1k"), [1024], None, None
    elif case == "ragged_gqa7":
        wl, lens, H, Hq = workload("omni7b_32k"), [1000, 517, 33, 1, 0, 2049, 256, 257], 2, 14
    elif case == "gqa8_splits":
        wl, lens, H, Hq = workload("omni3b_b4_64k_stream"), [20000, 7777], 2, 16
    else:
        wl, lens, H, Hq = workload("omni7b_32k"), [3000], 4, 4
    lay = gen_layer(wl, 2, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"], lay["v"]
    if H is not None:
        k, v = k[:, :H].copy(), v[:, :H].copy()
    Hq = Hq or wl.num_q_heads
    q = gen_queries(wl.wid, 2, len(lens), Hq)
    _announce(f"dense decode {case} lens={lens} H={k.shape[1]} Hq={Hq}")
    out = _dense(k, v, q, lens)
    _check(out, k, v, q, lens, case)


def test_dense_decode_ignores_unused_rows():
    """Rows at and beyond a sequence's length hold NaN: they must not reach the output."""
    wl = workload("omni7b_32k")
    lens = [77, 300, 1]
    lay = gen_layer(wl, 4, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :1].copy(), lay["v"][:, :1].copy()
    q = gen_queries(wl.wid, 4, len(lens), 7)
    _announce("dense decode, NaN beyond the lengths")
    out = _dense(k, v, q, lens, cap=512, fill_nan=True)
    assert np.all(np.isfinite(out))
    _check(out, k, v, q, lens, "nan_padding")


def test_dense_decode_growing_maximum():
    """Scores that grow along the sequence move each wave's softmax reference many times."""
    L, G = 4096, 8
    t = np.arange(L, dtype=np.float64)
    q = np.ones((1, G, 128), np.float16)
    q[0, 1::2] *= -1                                  # half the heads see the scores fall instead
    k = np.tile((4.0 * t / L)[:, None], (1, 128)).astype(np.float16)[None, None]
    rng = np.random.default_rng(5)
    v = rng.standard_normal((1, 1, L, 128)).astype(np.float16)
    _announce("dense decode, growing softmax maximum")
    out = _dense(k, v, q, [L])
    _check(out, k, v, q, [L], "growing_max")


def test_dense_decode_timed_equals_untimed():
    import torch
    wl = workload("omni7b_32k")
    lens = [5000, 3001]
    lay = gen_layer(wl, 1, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :2].copy(), lay["v"][:, :2].copy()
    q = gen_queries(wl.wid, 1, 2, 14)
    events = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in events:
        e.record()
    _announce("dense decode, timed entry point")
    a = _dense(k, v, q, lens)
    b = _dense(k, v, q, lens, events=events)
    np.testing.assert_array_equal(a, b)
    assert events[0].elapsed_time(events[1]) > 0 and events[2].elapsed_time(events[3]) > 0


def test_dense_decode_full_size_layer():
    """The 30B-like layer: 4 KV heads, 32 query heads, 131072 tokens, every output row."""
    wl = workload("omni30b_128k_48layer")
    lay = gen_layer(wl, 0)
    lens = [int(x) for x in lay["lens"]]
    q = gen_queries(wl.wid, 0, len(lens), wl.num_q_heads)
    _announce(f"dense decode omni30b layer lens={lens}")
    out = _dense(lay["k"], lay["v"], q, lens)
    _check(out, lay["k"], lay["v"], q, lens, "omni30b_layer")
