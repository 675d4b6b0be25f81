"""Full-size parity at the batch-16 ragged, streaming 3B-like and 128k 30B-like workload shapes.

Each workload runs at its real size through the same entry points the benchmark times (one prefill
append, then decode with the default split plan). The oracle checks sampled outputs one by one:
whole (sequence, KV head) decode rows against the float64 oracle on the GPU-written cache, and
sampled 32-token windows of the codec (key fields and value norms bit-exact, value codes by the
band rule, padded slots zero).
"""

import math

import numpy as np
import pytest

from oracle.cache import decode_layer
from oracle.hadamard import randomized_hadamard
from synth import S_SIGN, gen_layer, gen_queries, gen_stream_layer, rng_for, workload

pytestmark = pytest.mark.gpu
TOL = 2e-3
SM = 1 / math.sqrt(128)


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _prefill(lay, Hq, capacity, n_prefill=None):
    """Cache holding the first n_prefill tokens (default: each sequence's length) from one append."""
    import torch

    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    k, v, mod = lay["k"], lay["v"], lay["modality"]
    B, H = k.shape[:2]
    lens = np.asarray(lay["lens"] if n_prefill is None else np.full(B, n_prefill), np.int32)
    n_max = int(lens.max())
    cache = gh.new_cache(B, H, Hq, capacity, lay["signs"], lay["rot"])
    okvq.okvq_append(cache, [0] * B, gh.f16dev(k[:, :, :n_max]), gh.f16dev(v[:, :, :n_max]),
                     gh.dev(np.ascontiguousarray(mod[:, :n_max])), lens.tolist(), gh.dev(lens), n_max)
    torch.cuda.synchronize()
    return cache, lens


def _check_decode(out, arrays, q, lens, lay, pairs):
    import gpu_helpers as gh
    ref = decode_layer(arrays, q, lens, lay["signs"], lay["rot"], SM, heads=set(pairs))
    r = gh.attention_close(out, ref)
    print(f"decode worst err / norm over {len(pairs)} (b, h) rows = {r:.2e}")
    assert r <= TOL
    return r


def _check_windows(arrays, lay, pairs, lens, per_pair=4, seed=0):
    import gpu_helpers as gh
    rng = np.random.default_rng(seed)
    for b, h in pairs:
        L = int(lens[b])
        last = (L - 1) // 32
        wins = {0, last} | set(rng.integers(0, last + 1, per_pair).tolist())
        for w in sorted(wins):
            gh.check_window(arrays, lay["k"][b, h], lay["v"][b, h], lay["modality"][b], lay["signs"], lay["rot"],
                            b, h, w, L)


def test_b16_ragged16k_full_size():
    """16 sequences, lengths U{8192..16384} (partial last windows), 4 KV heads, 28 query heads."""
    import gpu_helpers as gh
    wl = workload("omni7b_b16_ragged16k")
    lay = gen_layer(wl, 0)
    lens = lay["lens"]
    _announce(f"b16 ragged lens={lens.tolist()}")
    cache, _ = _prefill(lay, wl.num_q_heads, wl.capacity)
    assert np.any(lens % 32 != 0)
    out = gh.decode(cache, lay["q"], lens)
    assert np.all(np.isfinite(out))
    arrays = gh.cache_to_numpy(cache)
    bs = sorted({int(np.argmin(lens)), int(np.argmax(lens)), 5, 11})
    pairs = [(b, h) for b in bs for h in range(wl.num_kv_heads)]
    _check_decode(out, arrays, lay["q"], lens, lay, pairs)
    _check_windows(arrays, lay, [(b, b % wl.num_kv_heads) for b in bs], lens)


def test_omni3b_streaming_full_size():
    """B4 x 65536-token prefill (2 KV heads, 16 query heads), then 16 steps of 512-token audio-visual
    appends, each followed by a decode; oracle rows on the first, a middle and the last step."""
    import torch

    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    wl = workload("omni3b_b4_64k_stream")
    lay = gen_stream_layer(wl, 0)
    pre, step = lay["prefill"], wl.stream_tokens
    _announce(f"omni3b stream prefill={pre} steps={wl.stream_steps}x{step}")
    cache, _ = _prefill(lay, wl.num_q_heads, wl.capacity, n_prefill=pre)
    B = wl.batch
    cur = pre
    pairs = [(0, 0), (3, 1)]
    for s in range(wl.stream_steps):
        sl = slice(cur, cur + step)
        n = np.full(B, step, np.int32)
        okvq.okvq_append(cache, [cur] * B, gh.f16dev(lay["k"][:, :, sl]), gh.f16dev(lay["v"][:, :, sl]),
                         gh.dev(np.ascontiguousarray(lay["modality"][:, sl])), n.tolist(), gh.dev(n), step)
        cur += step
        lens = np.full(B, cur, np.int32)
        q = gen_queries(wl.wid, 0, B, wl.num_q_heads, step=s + 1)
        out = gh.decode(cache, q, lens)
        assert np.all(np.isfinite(out)), f"step {s}"
        if s in (0, 7, wl.stream_steps - 1):
            torch.cuda.synchronize()
            _announce(f"omni3b stream step {s} len={cur}")
            _check_decode(out, gh.cache_to_numpy(cache), q, lens, lay, pairs)
    arrays = gh.cache_to_numpy(cache)
    assert np.array_equal(arrays["seq_lens"], np.full(B, cur, np.int32))
    assert int(cache.buffers["seq_lens"][-1].item()) == 0  # append's work-group counter
    _check_windows(arrays, lay, pairs, np.full(B, cur), per_pair=6, seed=1)
    # the windows either side of the prefill / stream boundary
    for b, h in pairs:
        for w in (pre // 32 - 1, pre // 32):
            gh.check_window(arrays, lay["k"][b, h], lay["v"][b, h], lay["modality"][b], lay["signs"], lay["rot"],
                            b, h, w, cur)


def _omni30b_layer(layer, global_rotation):
    import gpu_helpers as gh
    wl = workload("omni30b_128k_48layer")
    lay = gen_layer(wl, layer)
    if global_rotation:
        # single randomized-Hadamard value rotation with its own signs, shared by all modalities
        s = np.where(rng_for(wl.wid, layer, S_SIGN, 1, 0).integers(0, 2, 128) == 1, 1, -1).astype(np.int8)
        lay["rot"] = np.stack([randomized_hadamard(s)] * 3).astype(np.float32)
    _announce(f"omni30b layer {layer} global_rotation={global_rotation}")
    cache, lens = _prefill(lay, wl.num_q_heads, wl.capacity)
    out = gh.decode(cache, lay["q"], lens)
    assert np.all(np.isfinite(out))
    arrays = gh.cache_to_numpy(cache)
    return wl, lay, lens, out, arrays


def test_omni30b_128k_layer_full_size():
    """One layer at 131072 tokens, 4 KV heads, 32 query heads (group 8), per-modality rotations."""
    wl, lay, lens, out, arrays = _omni30b_layer(3, False)
    _check_decode(out, arrays, lay["q"], lens, lay, [(0, 0), (0, 3)])
    _check_windows(arrays, lay, [(0, h) for h in range(wl.num_kv_heads)], lens, per_pair=3, seed=2)


def test_omni30b_128k_global_rotation_variant():
    """The single-global-rotation variant (R_m = one randomized Hadamard for every m) at 131072 tokens."""
    wl, lay, lens, out, arrays = _omni30b_layer(4, True)
    _check_decode(out, arrays, lay["q"], lens, lay, [(0, 1)])
    _check_windows(arrays, lay, [(0, 2)], lens, per_pair=3, seed=3)
