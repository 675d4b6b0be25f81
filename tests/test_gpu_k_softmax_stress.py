"""GPU parity of decode attention where small softmax weights matter (Eq. 1).

The workload generators make attention nearly one-hot, which hides how the kernels carry weights far
below the running maximum: each wave keeps a lazily moved softmax reference and feeds p n_v to the
matrix cores as fp16. These cases put many tokens 10-30 log2 units below a dominant one (their
values along one channel, so a dropped or biased weight shows up in full in one output channel),
make the maximum grow or fall along the sequence, and make the value norms grow from 1e-3 to 6e4.
Each runs at the default split plan and at plans where a wave takes hundreds of windows
(OKVQ_DECODE_GROUPS / OKVQ_LADDER_GROUPS), against float64 attention over the GPU-written cache,
at the 2e-3 tolerance. A fixed 2^-8 scale of p n_v (no norm-dependent scale) fails the dominant
case at 3e-3 under OKVQ_DECODE_GROUPS=1."""

import math

import numpy as np
import pytest

from oracle.cache import decode_layer, unpacked_fields
from oracle.hadamard import randomized_hadamard
from oracle.keys import dequantize_directions
from oracle.ladder import decode_layer_bits
from synth.stress import dominant_layer, growing_layer, norm_ramp_layer

pytestmark = pytest.mark.gpu
TOL = 2e-3
SM = 1 / math.sqrt(128)
SCALES = [0.6, 0.8, 1.0, 1.1, 1.2, 1.3, 1.5, 1.8]   # score gaps of about 10 to 30 log2 units


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _score_gaps(arrays, q, L, signs, h=0):
    """log2-unit gap between the largest and the median score of every query head of KV head h."""
    kc, m16, st16, nk, _, _, _ = unpacked_fields(arrays, 0, h)
    zhat = dequantize_directions(kc[:L], m16, st16)
    hm = randomized_hadamard(signs)
    G = q.shape[1] // arrays["k_codes"].shape[1]
    gaps = []
    for j in range(h * G, (h + 1) * G):
        s = SM * nk[:L].astype(np.float64) * (zhat @ (hm @ q[0, j].astype(np.float64))) / math.log(2)
        gaps.append(float(s.max() - np.median(s)))
    return np.array(gaps)


def _packed(lay, key_meta="fp16"):
    import gpu_helpers as gh
    L = int(lay["lens"][0])
    H = lay["k"].shape[1]
    Hq = lay["q"].shape[1]
    cap = -(-L // 32) * 32
    cache = gh.new_cache(1, H, Hq, cap, lay["signs"], lay["rot"], key_meta=key_meta)
    gh.append_chunks(cache, lay["k"], lay["v"], lay["modality"], [L], [[L]])
    return cache, gh.cache_to_numpy(cache)


@pytest.mark.parametrize("groups", [None, "2", "1"])
def test_packed_decode_dominant_tokens_over_flat_background(groups, monkeypatch):
    import gpu_helpers as gh
    lay = dominant_layer(16384, 1, 8, SCALES, period=2048)
    cache, arrays = _packed(lay)
    gaps = _score_gaps(arrays, lay["q"], 16384, lay["signs"])
    assert gaps.min() < 12 and gaps.max() > 25 and np.any((gaps > 16) & (gaps < 21)), gaps
    ref = decode_layer(arrays, lay["q"], lay["lens"], lay["signs"], lay["rot"], SM)
    if groups:
        monkeypatch.setenv("OKVQ_DECODE_GROUPS", groups)
    _announce(f"packed decode, dominant tokens, groups={groups}")
    out = gh.decode(cache, lay["q"], [16384])
    r = gh.attention_close(out, ref)
    print(f"dominant groups={groups} gaps={np.round(gaps, 1).tolist()} worst err / norm = {r:.2e}")
    assert r <= TOL


@pytest.mark.parametrize("key_meta", ["mxfp4", "turboquant"])
def test_packed_decode_dominant_tokens_other_key_formats(key_meta, monkeypatch):
    import gpu_helpers as gh
    lay = dominant_layer(16384, 1, 8, SCALES, period=2048, seed=1)
    cache, arrays = _packed(lay, key_meta)
    ref = decode_layer(arrays, lay["q"], lay["lens"], lay["signs"], lay["rot"], SM)
    monkeypatch.setenv("OKVQ_DECODE_GROUPS", "1")
    _announce(f"packed decode, dominant tokens, {key_meta}, groups=1")
    out = gh.decode(cache, lay["q"], [16384])
    r = gh.attention_close(out, ref)
    print(f"dominant {key_meta} worst err / norm = {r:.2e}")
    assert r <= TOL


@pytest.mark.parametrize("groups", [None, "1"])
@pytest.mark.parametrize("kind", ["growing", "norm_ramp"])
def test_packed_decode_moving_maximum_and_norm_scale(kind, groups, monkeypatch):
    import gpu_helpers as gh
    lay = growing_layer(8192, 1, 8) if kind == "growing" else norm_ramp_layer(8192, 1, 8)
    cache, arrays = _packed(lay)
    ref = decode_layer(arrays, lay["q"], lay["lens"], lay["signs"], lay["rot"], SM)
    if groups:
        monkeypatch.setenv("OKVQ_DECODE_GROUPS", groups)
    _announce(f"packed decode, {kind}, groups={groups}")
    out = gh.decode(cache, lay["q"], [8192])
    assert np.all(np.isfinite(out))
    r = gh.attention_close(out, ref)
    print(f"{kind} groups={groups} worst err / norm = {r:.2e}")
    assert r <= TOL


def test_packed_decode_dominant_tokens_full_layer():
    """The 30B-like layer's shape (4 KV heads, 32 query heads, 131072 tokens) at the default plan,
    where every wave takes four window pairs."""
    import gpu_helpers as gh
    lay = dominant_layer(131072, 4, 8, SCALES, period=2048, seed=2)
    cache, arrays = _packed(lay)
    ref = decode_layer(arrays, lay["q"], lay["lens"], lay["signs"], lay["rot"], SM)
    _announce("packed decode, dominant tokens, 131072-token layer")
    out = gh.decode(cache, lay["q"], [131072])
    r = gh.attention_close(out, ref)
    print(f"dominant 131072 worst err / norm = {r:.2e}")
    assert r <= TOL


@pytest.mark.parametrize("groups", [None, "1"])
@pytest.mark.parametrize("kb,vb,meta", [(2, 2, "fp16"), (4, 4, "fp16"), (3, 2, "turboquant")])
def test_ladder_decode_dominant_and_moving(kb, vb, meta, groups, monkeypatch):
    import gpu_helpers as gh
    for name, lay in (("dominant", dominant_layer(16384, 1, 8, SCALES, period=2048, seed=3)),
                      ("growing", growing_layer(8192, 1, 8, seed=3)),
                      ("norm_ramp", norm_ramp_layer(8192, 1, 8, seed=3))):
        L = int(lay["lens"][0])
        cache = gh.ladder_cache(lay["k"], lay["v"], lay["modality"], [L], lay["signs"], lay["rot"], L, 8, kb, vb,
                                meta)
        arrays = {n: t.cpu().numpy() for n, t in cache.views().items() if n != "seq_lens"}
        ref = decode_layer_bits(arrays, lay["q"], [L], lay["signs"], lay["rot"], SM, kb, vb)
        if groups:
            monkeypatch.setenv("OKVQ_LADDER_GROUPS", groups)
        _announce(f"ladder decode K{kb}V{vb} {meta}, {name}, groups={groups}")
        out = gh.decode(cache, lay["q"], [L])
        monkeypatch.delenv("OKVQ_LADDER_GROUPS", raising=False)
        r = gh.attention_close(out, ref)
        print(f"ladder K{kb}V{vb} {meta} {name} groups={groups} worst err / norm = {r:.2e}")
        assert r <= TOL
