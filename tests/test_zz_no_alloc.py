"""The allocation-free decode entry point (okvq_decode_attention_noalloc): split records in the
library's static per-GPU array instead of a caller workspace. Checked through the C ABI against
okvq_decode_attention on the same cache (same kernels and plan: identical bits) and against the
float64 oracle at the 2e-3 tolerance, on two calls in a row -- the second with a smaller input, so
the array still holds the first call's records -- and on a ladder-layout cache."""

import math

import numpy as np
import pytest

from oracle.cache import decode_layer
from oracle.ladder import decode_layer_bits
from synth import gen_layer, gen_queries, workload

pytestmark = pytest.mark.gpu
TOL = 2e-3
SM = 1 / math.sqrt(128)


def _both(cache, q, lens):
    import torch

    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    B, Hq, D = q.shape
    qd = gh.f16dev(q)
    ws = okvq.decode_workspace(cache.dims, int(max(lens)))
    ref = torch.full((B, Hq, D), float("nan"), dtype=torch.float32, device="cuda")
    okvq.okvq_decode_attention(cache, list(lens), qd, SM, ref, ws)
    got = torch.full((B, Hq, D), float("nan"), dtype=torch.float32, device="cuda")
    okvq.okvq_decode_attention_noalloc(cache, list(lens), qd, SM, got)
    torch.cuda.synchronize()
    return got.cpu().numpy().astype(np.float64), ref.cpu().numpy().astype(np.float64)


def test_noalloc_decode_equals_workspace_decode_on_two_calls():
    import gpu_helpers as gh
    wl = workload("omni7b_32k")
    for lens, H, Hq in (([5000, 3000], 4, 28), ([700], 2, 14)):
        print(f"[gpu-case] noalloc decode lens={lens} H={H} Hq={Hq}", flush=True)
        lay = gen_layer(wl, 0, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
        k, v = lay["k"][:, :H].copy(), lay["v"][:, :H].copy()
        q = gen_queries(wl.wid, 0, len(lens), Hq)
        cap = -(-max(lens) // 32) * 32
        cache = gh.new_cache(len(lens), H, Hq, cap, lay["signs"], lay["rot"])
        gh.append_chunks(cache, k, v, lay["modality"], lens, [list(lens)])
        got, ref = _both(cache, q, lens)
        assert np.array_equal(got, ref)
        oracle = decode_layer(gh.cache_to_numpy(cache), q, np.asarray(lens), lay["signs"], lay["rot"], SM)
        assert gh.attention_close(got, oracle) <= TOL


def test_noalloc_decode_ladder_layout():
    import gpu_helpers as gh
    wl = workload("omni7b_32k")
    lens = [3000, 1]
    lay = gen_layer(wl, 1, lengths=np.asarray(lens, np.int32), n_tokens=max(lens))
    k, v = lay["k"][:, :2].copy(), lay["v"][:, :2].copy()
    q = gen_queries(wl.wid, 1, 2, 14)
    print("[gpu-case] noalloc decode, ladder K3V3", flush=True)
    cache = gh.ladder_cache(k, v, lay["modality"], lens, lay["signs"], lay["rot"], 3008, 14, 3, 3, "fp16")
    got, ref = _both(cache, q, lens)
    assert np.array_equal(got, ref)
    arrays = {n: t.cpu().numpy() for n, t in cache.views().items() if n != "seq_lens"}
    assert gh.attention_close(got, decode_layer_bits(arrays, q, lens, lay["signs"], lay["rot"], SM, 3, 3)) <= TOL
