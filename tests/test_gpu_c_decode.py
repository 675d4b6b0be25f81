"""GPU parity of fused decode attention against the float64 oracle (tolerance 2e-3 of the output norm)."""

import math

import numpy as np
import pytest

from oracle.cache import decode_layer, quantize_layer
from synth import gen_layer, gen_queries, workload

pytestmark = pytest.mark.gpu
TOL = 2e-3
SM = 1 / math.sqrt(128)


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _run(wl_name, lens, n_tokens=None, layer=0, Hq=None, H=None, heads=None):
    import gpu_helpers as gh
    wl = workload(wl_name)
    lay = gen_layer(wl, layer, lengths=np.asarray(lens, np.int32), n_tokens=n_tokens or max(max(lens), 1))
    k, v = lay["k"], lay["v"]
    if H is not None:
        k, v = k[:, :H].copy(), v[:, :H].copy()
    Hkv = k.shape[1]
    Hq = Hq or wl.num_q_heads * Hkv // wl.num_kv_heads
    q = gen_queries(wl.wid, layer, len(lens), Hq)
    cap = max(32, -(-max(lens) // 32) * 32)
    cache = gh.new_cache(len(lens), Hkv, Hq, cap, lay["signs"], lay["rot"])
    _announce(f"decode {wl_name} lens={list(lens)[:6]} H={Hkv} Hq={Hq}")
    gh.append_chunks(cache, k, v, lay["modality"], lens, [list(lens)])
    out = gh.decode(cache, q, lens)
    arrays = gh.cache_to_numpy(cache)
    ref = decode_layer(arrays, q, np.asarray(lens), lay["signs"], lay["rot"], SM, heads=heads)
    return out, ref, dict(lay=lay, q=q, cache=cache, arrays=arrays, k=k, v=v)


def test_decode_tiny_config():
    out, ref, _ = _run("tiny_1k", [1024])
    import gpu_helpers as gh
    r = gh.attention_close(out, ref)
    print(f"tiny worst err / norm = {r:.2e}")
    assert r <= TOL


def test_decode_ragged_gqa7_multi_split():
    lens = [1000, 517, 33, 1, 64, 2049]
    out, ref, _ = _run("omni7b_32k", lens, H=2, Hq=14)
    import gpu_helpers as gh
    r = gh.attention_close(out, ref)
    print(f"ragged worst err / norm = {r:.2e}")
    assert r <= TOL


def test_decode_empty_sequence_gives_zeros():
    import gpu_helpers as gh
    out, ref, _ = _run("tiny_1k", [100, 0, 40])
    assert np.all(out[1] == 0)
    assert gh.attention_close(out[[0, 2]], ref[[0, 2]]) <= TOL


def test_decode_end_to_end_against_oracle_cache():
    """Oracle-quantized cache decoded by the oracle vs GPU-quantized cache decoded by the GPU."""
    import gpu_helpers as gh
    lens = [1024, 700]
    out, _, ctx = _run("omni3b_b4_64k_stream", lens, H=2, Hq=16)
    lay = ctx["lay"]
    oc = quantize_layer(ctx["k"], ctx["v"], lay["modality"], np.asarray(lens), lay["signs"], lay["rot"], 1024)
    ref = decode_layer(oc, ctx["q"], np.asarray(lens), lay["signs"], lay["rot"], SM)
    r = gh.attention_close(out, ref)
    print(f"end-to-end worst err / norm = {r:.2e}")
    assert r <= TOL


def test_decode_deterministic_and_split_plan_invariant(monkeypatch):
    """Two decodes under one plan are bit-identical; under a different split plan (one work-group
    for the whole sequence instead of six) the result moves only by rounding."""
    import gpu_helpers as gh
    lens = [3000]
    out, ref, ctx = _run("omni7b_32k", lens, H=1, Hq=7)
    out2 = gh.decode(ctx["cache"], ctx["q"], lens)
    assert np.array_equal(out, out2)
    assert gh.attention_close(out, ref) <= TOL
    monkeypatch.setenv("OKVQ_DECODE_GROUPS", "1")
    _announce("decode, one split")
    out3 = gh.decode(ctx["cache"], ctx["q"], lens)
    assert not np.array_equal(out3, out)  # the plan really changed (different rounding points)
    assert gh.attention_close(out3, ref) <= TOL
    assert gh.attention_close(out3, out) <= 5e-4


def test_decode_full_size_omni7b_32k():
    """The benchmark's workload (B1, H4, Hq28, 32768 tokens): every head against the oracle."""
    import gpu_helpers as gh
    wl = workload("omni7b_32k")
    out, ref, _ = _run("omni7b_32k", [wl.seq_len])
    r = gh.attention_close(out, ref)
    print(f"omni7b_32k worst err / norm = {r:.2e}")
    assert r <= TOL


def test_decode_workspace_reused_across_plans():
    """One workspace (never cleared) for consecutive calls whose split plans differ."""
    import torch

    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    out_a, ref_a, ctx_a = _run("omni7b_32k", [3000, 129], H=2, Hq=14)
    out_b, ref_b, ctx_b = _run("omni7b_32k", [40], H=2, Hq=14)
    dims = ctx_a["cache"].dims
    ws = okvq.decode_workspace(dims, 3000)
    ws.fill_(float("nan"))  # stale contents must not leak into the result
    for cache, q, lens, ref in ((ctx_a["cache"], ctx_a["q"], [3000, 129], ref_a),
                                (ctx_b["cache"], ctx_b["q"], [40], ref_b),
                                (ctx_a["cache"], ctx_a["q"], [3000, 129], ref_a)):
        _announce(f"decode reuse lens={lens}")
        out = torch.full((len(lens), 14, 128), float("nan"), dtype=torch.float32, device="cuda")
        okvq.okvq_decode_attention(cache, lens, gh.f16dev(q), SM, out, ws)
        torch.cuda.synchronize()
        assert gh.attention_close(out.cpu().numpy().astype(np.float64), ref) <= TOL


def test_decode_split_count_changes_only_rounding(monkeypatch):
    """Fewer and more work-groups than the default plan: the log-sum-exp merge gives the same answer
    up to the fp16 operands (p n_v, and each split's merged rows before the inverse rotation), whose
    rounding points move with the split boundaries: a few 2^-12 relative steps of the output norm."""
    import gpu_helpers as gh
    lens = [5000, 2100]
    out, ref, ctx = _run("omni7b_32k", lens, H=2, Hq=14)
    for groups in ("2", "8", "24"):  # 1, 2 and 6 splits per sequence and head instead of 10
        monkeypatch.setenv("OKVQ_DECODE_GROUPS", groups)
        _announce(f"decode groups={groups}")
        o2 = gh.decode(ctx["cache"], ctx["q"], lens)
        assert gh.attention_close(o2, ref) <= TOL
        assert gh.attention_close(o2, out) <= 5e-4


def test_prepare_rotation_tables():
    """Inverse table = fp16 transpose; forward fragments = fp16 hi / lo split in the operand layout."""
    import torch

    import paper_2609_11582_amd as okvq
    from synth import gen_rotations
    rot = gen_rotations(2, 3)
    rot[1, 5, 7] = 1.0 / 3.0            # a value that is not exact in fp16 (rounds to nearest even)
    rot[2, 0, 0] = 2.0 ** -25 * 1.5     # an fp16 subnormal after rounding
    want = np.ascontiguousarray(rot.transpose(2, 0, 1)).astype(np.float16).reshape(-1)
    hi = rot.astype(np.float16)
    lo = (rot - hi.astype(np.float32)).astype(np.float16)
    # block ((m 8 + nb) 4 + kk) 2 + part, row l, element e <- R_m[16 nb + l % 16][32 kk + 8 (l / 16) + e]
    lane = np.arange(64)
    frag = np.empty((3, 8, 4, 2, 64, 8), np.float16)
    for m in range(3):
        for nb in range(8):
            for kk in range(4):
                rows = 16 * nb + lane % 16
                cols = 32 * kk + 8 * (lane // 16)
                idx = cols[:, None] + np.arange(8)[None, :]
                frag[m, nb, kk, 0] = hi[m][rows[:, None], idx]
                frag[m, nb, kk, 1] = lo[m][rows[:, None], idx]
    r_dev = torch.from_numpy(rot).cuda()
    got = torch.full((okvq.okvq.ROTATION_TABLE_BYTES // 2,), float("nan"), dtype=torch.float16, device="cuda")
    _announce("prepare_rotation")
    okvq.okvq_prepare_rotation(r_dev, got)
    torch.cuda.synchronize()
    g = got.cpu().numpy().view(np.uint16)
    assert np.array_equal(g[:want.size], want.view(np.uint16))
    assert np.array_equal(g[want.size:], frag.reshape(-1).view(np.uint16))


def test_timed_decode_matches_untimed_and_reports_durations():
    import torch

    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    lens = [2000]
    out, ref, ctx = _run("omni7b_32k", lens, H=2, Hq=14)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in evs:
        e.record()
    ws = okvq.decode_workspace(ctx["cache"].dims, 2000)
    o2 = torch.full((1, 14, 128), float("nan"), dtype=torch.float32, device="cuda")
    _announce("decode timed")
    okvq.okvq_decode_attention_timed(ctx["cache"], lens, gh.f16dev(ctx["q"]), SM, o2, ws, evs)
    torch.cuda.synchronize()
    assert np.array_equal(o2.cpu().numpy().astype(np.float64), out)
    t_split, t_merge = evs[0].elapsed_time(evs[1]), evs[2].elapsed_time(evs[3])
    print(f"split {t_split * 1e3:.2f} us, merge {t_merge * 1e3:.2f} us")
    assert 0.0 < t_split < 1000.0 and 0.0 < t_merge < 1000.0
