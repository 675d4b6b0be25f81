"""Benchmark of the 2-bit KV-cache hot path on one MI355X.

A step is the paper's multiple-choice protocol on one batch (Sec. 3.1): append the whole prefill
(keys quantized per 32-token window after the Hadamard rotation, values rotated per modality and
coded) into an empty cache, then one decode-attention step over the packed cache.

Workload: the Qwen2.5-Omni-7B-like layer -- batch 1, 4 KV heads, 28 query heads (GQA 7), head
dim 128, 32768 cached tokens in 2-second audio-visual chunks (150 video + 25 audio tokens) and a
256-token text prompt; synthetic keys with temporal drift and outlier channels, values from
per-modality subspaces (seeded generators, no dataset).

Reported (one JSON line):
  value           decode-attention effective GB/s = algorithmic decode bytes / decode time (both
                  launches, back to back), with the cache cold in HBM (the decode cycles through
                  >= 1 GB of cache replicas)
  ms_per_step     one step (append prefill + decode), mean over the timed steps
  roofline        the split-K decode kernel (k_decode, the dominant decode launch) against the HBM
                  peak: algorithmic bytes / its mean duration, timed with HIP events bound to its
                  dispatch; traffic = HBM bytes per launch from the committed rocprofv3 counter
                  summary while the kernel sources are unchanged, else null;
                  roofline_append: the whole append call (the fused codec launch and the length
                  update)
  kernels_us      mean duration of each launch, from the same events
  codec_split     the prefill's keys and values quantized by separate stateless calls
  cpu_baseline    the CPU oracle on this host: its float64 decode of the same cache on all cores (value)
                  and single-threaded, and its fp32-order quantization of the prefill
  mxfp4           the same workload with MXFP4 key window metadata (72.25 instead of 84 bytes per
                  token and KV head): append, decode and split-K kernel time, effective GB/s
  turboquant      the same workload with TurboQuant keys (Eq. 2: Gaussian codebook after the Hadamard
                  rotation, no window metadata, 68 bytes per token and KV head) and the single value
                  rotation R_m = H: the K2/V2 baseline's append and decode
  residual        the same workload in the captioning protocol (fp16 rings of the last 128 keys and
                  values): prefill and one-token append, decode, split-K and merge-with-tail times
  ladder          the same layer at other bit widths (K2V2 .. K4V4, TurboQuant K3V2 / K4V4, Tab. 3 and
                  Tab. 5) in the bit-stream layout: stateless key and value quantization, decode
  omni30b_48layer the 30B-like workload with all 48 layers' caches resident (131072 tokens, 4 KV heads,
                  32 query heads): one decode step per layer over the packed caches, over packed
                  caches with the single global value rotation, and with the dense fp16 baseline
                  kernel over the same fp16 K and V (12.9 GB resident); per-layer append
  stream          the streaming workload (batch 4 x 65536, 2 KV heads, 16 query heads): 16 steps of a
                  512-token append per sequence then a decode, each timed
  calibration     the value-rotation calibration (Eq. 5) on a 4096-token calibration sequence at the
                  same head shapes: attention weights (against the fp16 matrix-core peak), weighted
                  covariance, host eigensolver

--profile-pass runs a short fixed sequence for rocprofv3 counter collection: a 256 MiB device
copy (calibrates FETCH_SIZE / WRITE_SIZE against a known byte count), 8 decode calls on cold
cache replicas and 2 prefill appends, the same with MXFP4 key metadata, 8 decode calls with the
fp16 residual, 8 decode calls and 2 appends with TurboQuant keys, and 4 dense fp16 decode calls at
the 30B-like layer shape.

--shape-scan times decode alone at the other workload shapes (batch 16 with ragged lengths up to
16384, batch 4 x 65536 with 2 KV heads and 16 query heads, 131072 tokens with 32 query heads, and
batch 32 x 32768), with fp16 and MXFP4 key metadata and with TurboQuant keys, one JSON line each, on
caches filled with random codes and metadata and the workload's modality layout (the kernel's work does not depend on the values).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attn effective KV GB/s vs HBM peak; µs/step at 32k ctx, 2-bit"
HBM_PEAK_GBPS = 8000.0
WORKLOAD = "omni7b_32k"
DECODE_BYTES_PER_WINDOW_HEAD = 2 * 1024 + 2 * 64 + 2 * 256   # codes K, V + norms K, V + min/step
APPEND_BYTES_PER_TOKEN_HEAD = 2 * 256 + 84                   # read K, V fp16; write the packed cache
MX_RECORD = 136                                              # MXFP4 min/step record of one window
DECODE_BYTES_PER_WINDOW_HEAD_MX = 2 * 1024 + 2 * 64 + MX_RECORD
APPEND_BYTES_PER_TOKEN_HEAD_MX = 2 * 256 + 68 + MX_RECORD / 32
DECODE_BYTES_PER_WINDOW_HEAD_TQ = 2 * 1024 + 2 * 64                # TurboQuant keys: no window metadata
APPEND_BYTES_PER_TOKEN_HEAD_TQ = 2 * 256 + 68
DECODE_BYTES_PER_WINDOW = {"fp16": DECODE_BYTES_PER_WINDOW_HEAD, "mxfp4": DECODE_BYTES_PER_WINDOW_HEAD_MX,
                           "turboquant": DECODE_BYTES_PER_WINDOW_HEAD_TQ}
APPEND_BYTES_PER_TOKEN = {"fp16": APPEND_BYTES_PER_TOKEN_HEAD, "mxfp4": APPEND_BYTES_PER_TOKEN_HEAD_MX,
                          "turboquant": APPEND_BYTES_PER_TOKEN_HEAD_TQ}
CACHE_BYTES_PER_TOKEN_HEAD = {"fp16": 84, "mxfp4": 72.25, "turboquant": 68}
PROFILE_COUNTERS = os.path.join(ROOT, "profiles", "hbm_counters.json")
CALIBRATION_COPY_BYTES = 256 << 20
KERNEL_SOURCES = ("codec_kernels.hip", "codec_fused.hip", "decode_kernels.hip", "key_quant.hpp", "value_quant.hpp",
                  "okvq_device.hpp", "launch.hpp", "calib_kernels.hip", "dense_decode.hip", "ladder_codec.hip",
                  "ladder_decode.hip", "append_window.hip", "lane_quant.hpp")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_11582_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def decode_algorithmic_bytes(B, H, Hq, lens, with_output=True, key_meta="fp16"):
    nwin = sum(-(-int(L) // 32) for L in lens)
    per_win = DECODE_BYTES_PER_WINDOW[key_meta]
    return (nwin * H * per_win + nwin * 32                            # cache + modality map
            + B * Hq * 128 * (2 + (4 if with_output else 0))          # q in, out
            + 3 * 128 * 128 * 4)                                      # rotations


def append_algorithmic_bytes(B, H, lens, key_meta="fp16"):
    n = sum(int(L) for L in lens)
    per_tok = APPEND_BYTES_PER_TOKEN[key_meta]
    return int(n * H * per_tok) + 2 * n + 3 * 128 * 128 * 4 + 128


def residual_decode_algorithmic_bytes(B, H, Hq, lens, residual=128):
    """Decode bytes with the fp16 residual of the captioning protocol: the quantized windows of the
    tokens below L - 128 (as for plain decode), the tail's quantized keys below 128 floor(L / 128)
    (codes, norm and their windows' metadata not already counted), its fp16 keys and values
    (256 B each), the modality map of the quantized part, q, out and R."""
    total = B * Hq * 128 * (2 + 4) + 3 * 128 * 128 * 4
    for L in lens:
        L = int(L)
        t0, kq = max(L - residual, 0), residual * (L // residual)
        nwm = -(-t0 // 32)                          # windows read by the split-K kernel
        nwk = -(-kq // 32)                          # windows holding quantized keys
        total += nwm * 32 + H * nwm * DECODE_BYTES_PER_WINDOW_HEAD
        total += H * (max(kq - t0, 0) * 34 + max(nwk - nwm, 0) * 512)
        total += H * ((L - max(kq, t0)) * 256 + (L - t0) * 256)
    return total


def measured_traffic(kernel_key):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if the kernels are unchanged."""
    try:
        with open(PROFILE_COUNTERS) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    entry = rec.get(kernel_key)
    return None if entry is None else entry.get("bytes_per_launch")


def cpu_baseline(cache_np, q, lens, signs, rot, bytes_per_call, prefill=None, append_bytes=None,
                 decode_seconds=8.0, single_seconds=4.0):
    """The CPU oracle as it stands, timed on this host: the float64 decode of the layer (all KV heads)
    on every core the BLAS pool uses and single-threaded, and the fp32-order (FMT) quantization of
    the prefill (all 32768 tokens and KV heads; one KV head single-threaded)."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle.cache import decode_layer, quantize_layer

    def decode_rate(min_seconds):
        t0 = time.perf_counter()
        calls = 0
        while True:
            decode_layer(cache_np, q, lens, signs, rot, 1 / math.sqrt(128))
            calls += 1
            el = time.perf_counter() - t0
            if el >= min_seconds or calls >= 200:
                return calls, el

    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    calls, el = decode_rate(decode_seconds)
    res = dict(value=round(bytes_per_call * calls / el / 1e9, 4), unit="GB/s", cores=int(threads), kind="oracle",
               sample=f"{calls} full decode steps of the {WORKLOAD} layer (4 KV heads, 28 query heads, 32768 "
                      f"tokens), float64, {el:.1f} s")
    with threadpool_limits(1):
        c1, e1 = decode_rate(single_seconds)
    res["single_thread"] = dict(value=round(bytes_per_call * c1 / e1 / 1e9, 4), unit="GB/s", cores=1,
                                sample=f"{c1} decode steps, {e1:.1f} s")
    if prefill is not None:
        k, v, mod = prefill
        t0 = time.perf_counter()
        quantize_layer(k, v, mod, lens, signs, rot, k.shape[2])
        eq = time.perf_counter() - t0
        with threadpool_limits(1):
            t0 = time.perf_counter()
            quantize_layer(k[:, :1], v[:, :1], mod, lens, signs, rot, k.shape[2])
            eq1 = time.perf_counter() - t0
        res["quantize"] = dict(value=round(append_bytes / eq / 1e9, 4), unit="GB/s", cores=int(threads),
                               sample=f"the whole prefill (32768 tokens, 4 KV heads) quantized once, fp32 order, "
                                      f"{eq:.1f} s",
                               single_thread=dict(value=round(append_bytes / k.shape[1] / eq1 / 1e9, 4), unit="GB/s",
                                                  cores=1, sample=f"one KV head of the prefill, {eq1:.1f} s"))
    res["host"] = dict(cpu_count=os.cpu_count(), affinity=len(os.sched_getaffinity(0)), blas_threads=int(threads),
                       numpy=np.__version__)
    return res


def _scan_case(okvq, torch, name, B, lens, H, Hq, key_meta, wl):
    """Decode alone on random caches of one shape: per-call time over cycled replicas, effective GB/s.
    Codes, norms and metadata are random (the kernel's work does not depend on them); the modality
    map is the workload's token stream (audio-visual chunks, then the text prompt), which does
    decide the work (a pair with text runs a second value product)."""
    import numpy as np
    dev = torch.device("cuda:0")
    sm = 1 / math.sqrt(128)
    cap = (max(lens) + 31) // 32 * 32
    dims = okvq.make_dims(B, H, Hq, cap, key_meta=key_meta)
    per_cache = sum(okvq.okvq_buffer_bytes(dims, i) for i in range(10))
    reps = max(2, min(16, int(math.ceil(1.05e9 / per_cache))))
    g = torch.Generator(device=dev).manual_seed(7)
    from synth import modality_layout
    mm = np.zeros((B, cap), np.uint8)
    for b, L in enumerate(lens):
        mm[b, :L] = modality_layout(int(L), wl.video_per_chunk, wl.audio_per_chunk, wl.text_tail)
    mod_map = torch.from_numpy(mm.reshape(-1)).to(dev)
    caches = []
    for r in range(reps):
        c = okvq.KVCache(B, H, Hq, cap, torch.ones(128, dtype=torch.int8), torch.eye(128).repeat(3, 1, 1), device=dev,
                         key_meta=key_meta)
        for n, t in c.buffers.items():
            if n == "seq_lens":
                t[:B].copy_(torch.tensor(lens, dtype=torch.int32))
            elif n == "modality":
                t.copy_(mod_map)
            elif t.dtype == torch.float16:
                t.copy_((torch.rand(t.shape, device=dev, generator=g) * 0.5 + 0.1).half())
            elif t.dtype == torch.uint8:
                t.random_(0, 256, generator=g)
        if key_meta == "mxfp4":  # block scales of ordinary key statistics (2^-4)
            c.views()["k_mx"][..., 128:].fill_(123)
        caches.append(c)
    q = torch.randn(B, Hq, 128, device=dev, generator=g).half()
    ws = okvq.decode_workspace(caches[0].dims, max(lens), device=dev)
    out = torch.empty(B, Hq, 128, device=dev)
    for i in range(10):
        okvq.okvq_decode_attention(caches[i % reps], lens, q, sm, out, ws)
    torch.cuda.synchronize()
    n = 100
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(n):
        okvq.okvq_decode_attention(caches[i % reps], lens, q, sm, out, ws)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / n
    nbytes = decode_algorithmic_bytes(B, H, Hq, lens, key_meta=key_meta)
    print(json.dumps({"shape_scan": name, "key_meta": key_meta, "batch": B, "kv_heads": H, "q_heads": Hq,
                      "max_len": max(lens), "decode_us": round(us, 2), "algorithmic_MB": round(nbytes / 1e6, 2),
                      "GBps": round(nbytes / us / 1e3, 1), "frac": round(nbytes / us / 1e3 / HBM_PEAK_GBPS, 4)}),
          flush=True)


def shape_scan(okvq, torch, workload, gen_lengths):
    """Decode alone at the other workload shapes, with fp16 and MXFP4 key metadata and TurboQuant keys."""
    cases = [("omni7b_b16_ragged16k", None), ("omni3b_b4_64k_stream", None), ("omni30b_128k_48layer", None),
             ("omni7b_32k", 32)]
    for name, batch in cases:
        wl = workload(name)
        B = batch or wl.batch
        lens = [int(x) for x in gen_lengths(wl)] if batch is None else [wl.seq_len] * B
        for km in ("fp16", "mxfp4", "turboquant"):
            _scan_case(okvq, torch, name, B, lens, wl.num_kv_heads, wl.num_q_heads, km, wl)


def sylvester_hadamard(signs):
    """Orthonormal randomized Hadamard matrix H diag(signs) of order 128 (Sylvester construction):
    the single value rotation of the TurboQuant baseline."""
    import numpy as np
    h = np.ones((1, 1))
    while h.shape[0] < 128:
        h = np.block([[h, h], [h, -h]])
    return (h * np.asarray(signs, np.float64)[None, :] / math.sqrt(128)).astype(np.float32)


def key_meta_measurement(okvq, torch, np, wl, lens, k_in, v_in, m0, n_new_dev, q, stream, decode_iters,
                         key_meta, signs=None, rot=None, flags=0):
    """The benchmark workload with another key storage: MXFP4 window metadata (the paper's default)
    or TurboQuant keys (no window metadata). Prefill append into an empty cache, decode over >= 1 GB
    of cold cache replicas, and the split-K kernel's duration from events bound to its dispatch."""
    B, H, Hq, N = wl.batch, wl.num_kv_heads, wl.num_q_heads, wl.seq_len
    dev = q.device
    sm = 1 / math.sqrt(128)
    dims = okvq.make_dims(B, H, Hq, wl.capacity, key_meta=key_meta)
    per_cache = sum(okvq.okvq_buffer_bytes(dims, i) for i in range(10))
    n_cache = max(16, int(math.ceil(1.05e9 / per_cache)))
    signs = torch.ones(128, dtype=torch.int8) if signs is None else signs
    rot = torch.eye(128).repeat(3, 1, 1) if rot is None else rot
    caches = [okvq.KVCache(B, H, Hq, wl.capacity, signs, rot, device=dev, key_meta=key_meta)
              for _ in range(n_cache)]
    okvq.okvq_append(caches[0], [0] * B, k_in[0], v_in[0], m0, lens, n_new_dev, N, flags=flags, stream=stream)
    torch.cuda.synchronize()
    for c in caches[1:]:
        for name in c.buffers:
            c.buffers[name].copy_(caches[0].buffers[name])
    ws = okvq.decode_workspace(dims, max(lens), device=dev)
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
    # appends (prefill into an emptied replica, inputs cycled)
    app = []
    for i in range(12):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c = caches[(i + 1) % n_cache]
        c.buffers["seq_lens"].zero_()
        e0.record(stream)
        okvq.okvq_append(c, [0] * B, k_in[i % len(k_in)], v_in[i % len(v_in)], m0, lens, n_new_dev, N, flags=flags,
                         stream=stream)
        e1.record(stream)
        app.append((e0, e1))
    torch.cuda.synchronize()
    append_us = float(np.mean([a.elapsed_time(b) for a, b in app[2:]])) * 1e3
    reps = []
    for rep in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for i in range(20):
            okvq.okvq_decode_attention(caches[i % n_cache], lens, q, sm, out, ws, flags=flags, stream=stream)
        e0.record(stream)
        for i in range(decode_iters):
            okvq.okvq_decode_attention(caches[(i * 7 + rep) % n_cache], lens, q, sm, out, ws, flags=flags,
                                       stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        reps.append(e0.elapsed_time(e1) * 1e3 / decode_iters)
    decode_us, decode_us_min = float(np.median(reps)), float(np.min(reps))
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(decode_iters)]
    for e4 in evs:
        for e in e4:
            e.record(stream)
    torch.cuda.synchronize()
    for i in range(decode_iters):
        okvq.okvq_decode_attention_timed(caches[(i * 7 + 5) % n_cache], lens, q, sm, out, ws, evs[i], flags=flags,
                                         stream=stream)
    torch.cuda.synchronize()
    split_us = float(np.mean([e[0].elapsed_time(e[1]) for e in evs])) * 1e3
    dbytes = decode_algorithmic_bytes(B, H, Hq, lens, key_meta=key_meta)
    sbytes = decode_algorithmic_bytes(B, H, Hq, lens, with_output=False, key_meta=key_meta)
    abytes = append_algorithmic_bytes(B, H, lens, key_meta=key_meta)
    del caches
    tag = {"mxfp4": "mx", "turboquant": "tq"}[key_meta]
    return {"bytes_per_token_head": CACHE_BYTES_PER_TOKEN_HEAD[key_meta], "decode_us": round(decode_us, 3),
            "decode_us_min": round(decode_us_min, 3),
            "decode_GBps": round(dbytes / decode_us / 1e3, 2),
            "k_decode_us": round(split_us, 3), "k_decode_GBps": round(sbytes / split_us / 1e3, 2),
            "k_decode_frac": round(sbytes / split_us / 1e3 / HBM_PEAK_GBPS, 4),
            "traffic": measured_traffic(f"k_decode_{tag}"), "append_traffic": measured_traffic(f"k_codec_{tag}"),
            "append_us": round(append_us, 3), "append_GBps": round(abytes / append_us / 1e3, 2),
            "append_frac": round(abytes / append_us / 1e3 / HBM_PEAK_GBPS, 4), "algorithmic_bytes": dbytes,
            "replicas": n_cache}


def codec_split_measurement(okvq, torch, np, wl, lens, k_in, v_in, m0, signs, rot, stream, iters=12):
    """The prefill's keys and values quantized separately by the stateless calls (each its own
    launch of the codec, one role): okvq_quantize_keys (K rows in; codes, norms, window minimum and
    step out: 306 B per token and KV head) and okvq_quantize_values (V rows and the modality map in;
    codes and norms out: 290 B, with R_m read as fp32 rather than as prepared fragments)."""
    B, H, Hq, N = wl.batch, wl.num_kv_heads, wl.num_q_heads, wl.seq_len
    dev = k_in[0].device
    c = okvq.KVCache(B, H, Hq, wl.capacity, signs, rot, device=dev)
    vw = c.views()
    sdev, rdev = c.key_signs, c.v_rot
    ntok = sum(int(L) for L in lens)

    def timed(fn):
        ev = []
        for i in range(iters):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn(i % len(k_in))
            e1.record(stream)
            ev.append((e0, e1))
        torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in ev[2:]])) * 1e3

    ku = timed(lambda i: okvq.okvq_quantize_keys(c.dims, k_in[i], N, lens, sdev, vw["k_codes"], vw["k_min"],
                                                 vw["k_step"], vw["k_norm"], stream=stream))
    vu = timed(lambda i: okvq.okvq_quantize_values(c.dims, v_in[i], m0, N, lens, rdev, 0, vw["v_codes"],
                                                   vw["v_norm"], stream=stream))
    kb = ntok * H * (256 + 32 + 2 + 16)
    vb = ntok * H * (256 + 32 + 2) + ntok + 3 * 128 * 128 * 4
    return {"keys_us": round(ku, 3), "keys_GBps": round(kb / ku / 1e3, 2), "keys_frac": round(kb / ku / 1e3 / HBM_PEAK_GBPS, 4),
            "values_us": round(vu, 3), "values_GBps": round(vb / vu / 1e3, 2),
            "values_frac": round(vb / vu / 1e3 / HBM_PEAK_GBPS, 4)}


LADDER_CASES = ((2, 2, "fp16"), (3, 3, "fp16"), (4, 4, "fp16"), (3, 2, "turboquant"), (4, 4, "turboquant"))


def ladder_bytes_per_token_head(kb, vb, meta):
    return 16 * kb + 16 * vb + 4 + (16 if meta == "fp16" else 0)


def ladder_measurement(okvq, torch, np, wl, lens, k_in, v_in, m0, q, signs, rot, stream, decode_iters):
    """The benchmark layer at other bit widths (the bit-width ladder, token-major bit-stream layout):
    the stateless key and value codecs over the prefill, then decode over >= 1 GB of cold replicas,
    for the method's keys (fp16 window metadata) and TurboQuant keys."""
    B, H, Hq, N = wl.batch, wl.num_kv_heads, wl.num_q_heads, wl.seq_len
    dev = q.device
    sm = 1 / math.sqrt(128)
    ntok = sum(int(L) for L in lens)
    res = {}
    for kb, vb, meta in LADDER_CASES:
        base = okvq.KVCache(B, H, Hq, wl.capacity, signs, rot, device=dev, key_meta=meta, key_bits=kb, value_bits=vb)
        vw = base.views()
        ev = []
        for i in range(8):
            e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            e0.record(stream)
            if meta == "fp16":
                okvq.okvq_quantize_keys(base.dims, k_in[i % len(k_in)], N, lens, base.key_signs, vw["k_codes"],
                                        vw["k_min"], vw["k_step"], vw["k_norm"], stream=stream)
            else:
                okvq.okvq_quantize_keys_tq(base.dims, k_in[i % len(k_in)], N, lens, base.key_signs, vw["k_codes"],
                                           vw["k_norm"], stream=stream)
            e1.record(stream)
            okvq.okvq_quantize_values(base.dims, v_in[i % len(v_in)], m0, N, lens, base.v_rot, 0, vw["v_codes"],
                                      vw["v_norm"], stream=stream)
            e2.record(stream)
            ev.append((e0, e1, e2))
        vw["modality"].copy_(m0)
        vw["seq_lens"].copy_(torch.tensor(lens, dtype=torch.int32))
        torch.cuda.synchronize()
        keys_us = float(np.mean([a.elapsed_time(b) for a, b, _ in ev[2:]])) * 1e3
        vals_us = float(np.mean([b.elapsed_time(c) for _, b, c in ev[2:]])) * 1e3
        exact = []
        for i in range(6):  # the exact fp32 order of the same call
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            okvq.okvq_quantize_values(base.dims, v_in[i % len(v_in)], m0, N, lens, base.v_rot, okvq.okvq.OKVQ_VALUE_EXACT,
                                      vw["v_codes"], vw["v_norm"], stream=stream)
            e1.record(stream)
            exact.append((e0, e1))
        torch.cuda.synchronize()
        vals_exact_us = float(np.mean([a.elapsed_time(b) for a, b in exact[2:]])) * 1e3
        per_cache = sum(okvq.okvq_buffer_bytes(base.dims, i) for i in range(12))
        n_cache = max(16, int(math.ceil(1.05e9 / per_cache)))
        caches = [base] + [okvq.KVCache(B, H, Hq, wl.capacity, signs, rot, device=dev, key_meta=meta, key_bits=kb,
                                        value_bits=vb) for _ in range(n_cache - 1)]
        for c in caches[1:]:
            for name in c.buffers:
                c.buffers[name].copy_(base.buffers[name])
        ws = okvq.decode_workspace(base.dims, max(lens), device=dev)
        out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
        reps = []
        for rep in range(5):
            for i in range(10):
                okvq.okvq_decode_attention(caches[i % n_cache], lens, q, sm, out, ws, stream=stream)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for i in range(decode_iters):
                okvq.okvq_decode_attention(caches[(i * 7 + rep) % n_cache], lens, q, sm, out, ws, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            reps.append(e0.elapsed_time(e1) * 1e3 / decode_iters)
        decode_us, decode_us_min = float(np.median(reps)), float(np.min(reps))
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(decode_iters)]
        for e4 in evs:
            for e in e4:
                e.record(stream)
        torch.cuda.synchronize()
        for i in range(decode_iters):
            okvq.okvq_decode_attention_timed(caches[(i * 7 + 3) % n_cache], lens, q, sm, out, ws, evs[i], stream=stream)
        torch.cuda.synchronize()
        split_us = float(np.mean([e[0].elapsed_time(e[1]) for e in evs])) * 1e3
        bpt = ladder_bytes_per_token_head(kb, vb, meta)
        dbytes = ntok * H * bpt + ntok + B * Hq * 128 * 6 + 3 * 128 * 128 * 2
        sbytes = dbytes - B * Hq * 128 * 4
        kbytes = ntok * H * (256 + 16 * kb + 2 + (16 if meta == "fp16" else 0))
        vbytes = ntok * H * (256 + 16 * vb + 2) + ntok + 3 * 128 * 128 * 4
        res[f"K{kb}V{vb}_{meta}"] = {
            "bits_per_element": round(bpt * 8 / 256, 4), "bytes_per_token_head": bpt,
            "quantize_keys_us": round(keys_us, 2), "quantize_keys_GBps": round(kbytes / keys_us / 1e3, 1),
            "quantize_values_us": round(vals_us, 2), "quantize_values_GBps": round(vbytes / vals_us / 1e3, 1),
            "quantize_values_exact_us": round(vals_exact_us, 2),
            "decode_us": round(decode_us, 3), "decode_us_min": round(decode_us_min, 3),
            "decode_GBps": round(dbytes / decode_us / 1e3, 1),
            "k_ladder_decode_us": round(split_us, 3), "k_ladder_decode_frac": round(sbytes / split_us / 1e3 / HBM_PEAK_GBPS, 4),
            "replicas": n_cache}
        del caches, base
        torch.cuda.empty_cache()
    return res


def stream_measurement(okvq, torch, np, dev, stream):
    """The streaming workload (batch 4 x 65536 tokens, 2 KV heads, 16 query heads, video-heavy): a
    prefill append, then 16 steps of (append 512 audio-visual tokens per sequence, decode). Each
    append and decode is timed with events; the decode reads the cache the step just wrote (warm in
    the Infinity Cache, as in the protocol). Inputs generated on the device (synth.device for the
    prefill; the streamed rows N(0, 1) with the workload's audio-visual pattern -- the append's
    work does not depend on the values)."""
    from synth import stream_chunk_modalities, workload
    from synth.device import gen_layer_device
    wl = workload("omni3b_b4_64k_stream")
    B, H, Hq, N, steps, step = wl.batch, wl.num_kv_heads, wl.num_q_heads, wl.seq_len, wl.stream_steps, wl.stream_tokens
    sm = 1 / math.sqrt(128)
    lay = gen_layer_device(wl, 0, dev)
    c = okvq.KVCache(B, H, Hq, wl.capacity, torch.from_numpy(lay["signs"]), torch.from_numpy(lay["rot"]), device=dev)
    lens = [N] * B
    okvq.okvq_append(c, [0] * B, lay["k"], lay["v"], lay["modality"], lens, torch.tensor(lens, dtype=torch.int32,
                                                                                          device=dev), N, stream=stream)
    g = torch.Generator(device=dev).manual_seed(11)
    kn = [torch.randn(B, H, step, 128, device=dev, generator=g).half() for _ in range(steps)]
    vn = [torch.randn(B, H, step, 128, device=dev, generator=g).half() for _ in range(steps)]
    mods = [torch.from_numpy(np.tile(stream_chunk_modalities(wl, N - wl.text_tail + s * step, step), (B, 1))).to(dev)
            for s in range(steps)]
    nn = torch.tensor([step] * B, dtype=torch.int32, device=dev)
    q = torch.from_numpy(lay["q"]).to(dev)
    ws = okvq.decode_workspace(c.dims, wl.capacity, device=dev)
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    ev = []
    for s in range(steps):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        cur = N + s * step
        e[0].record(stream)
        okvq.okvq_append(c, [cur] * B, kn[s], vn[s], mods[s], [step] * B, nn, step, stream=stream)
        e[1].record(stream)
        okvq.okvq_decode_attention(c, [cur + step] * B, q, sm, out, ws, stream=stream)
        e[2].record(stream)
        ev.append(e)
    torch.cuda.synchronize()
    app = [e[0].elapsed_time(e[1]) * 1e3 for e in ev]
    dec = [e[1].elapsed_time(e[2]) * 1e3 for e in ev]
    # device-side append latency: the GPU is kept busy while the host enqueues each timed append, so
    # that the events bracket the launch alone (the lengths are set back between the calls)
    L0 = N + (steps - 1) * step  # the last chunk again, from the length before it
    back = torch.tensor([L0] * B, dtype=torch.int32, device=dev)
    c.buffers["seq_lens"][:B].copy_(back)
    dev_app = []
    for s in range(10):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(200000)
        e0.record(stream)
        okvq.okvq_append(c, [L0] * B, kn[steps - 1], vn[steps - 1], mods[steps - 1], [step] * B, nn, step,
                         stream=stream)
        e1.record(stream)
        c.buffers["seq_lens"][:B].copy_(back)
        dev_app.append((e0, e1))
    torch.cuda.synchronize()
    dev_app_us = float(np.median([a.elapsed_time(b) for a, b in dev_app[2:]])) * 1e3
    # the append kernel alone: events bound to its dispatch (okvq_append_timed)
    kern = []
    for s in range(10):
        e2 = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        for e in e2:
            e.record(stream)
        okvq.okvq_append_timed(c, [L0] * B, kn[steps - 1], vn[steps - 1], mods[steps - 1], [step] * B, nn, step, e2,
                               stream=stream)
        c.buffers["seq_lens"][:B].copy_(back)
        kern.append(e2)
    torch.cuda.synchronize()
    kern_us = float(np.median([a.elapsed_time(b) for a, b in kern[2:]])) * 1e3
    mean_len = N + step * (steps + 1) / 2
    abytes = append_algorithmic_bytes(B, H, [step] * B)
    dbytes = decode_algorithmic_bytes(B, H, Hq, [int(mean_len)] * B)
    res = {"workload": "omni3b_b4_64k_stream", "batch": B, "kv_heads": H, "q_heads": Hq, "prefill": N,
           "steps": steps, "tokens_per_step": step,
           "append_us": round(float(np.mean(app[1:])), 2), "append_GBps": round(abytes / np.mean(app[1:]) / 1e3, 1),
           "append_device_us": round(dev_app_us, 2), "append_kernel_us": round(kern_us, 2),
           "decode_us": round(float(np.mean(dec[1:])), 2), "decode_GBps_warm": round(dbytes / np.mean(dec[1:]) / 1e3, 1),
           "step_us": round(float(np.mean([a + d for a, d in zip(app[1:], dec[1:])])), 2),
           "append_algorithmic_bytes": abytes}
    del c, kn, vn
    torch.cuda.empty_cache()
    return res


def dense_decode_bytes(B, H, Hq, lens):
    """Dense fp16 decode: K and V rows (512 B per token and KV head), q in, out."""
    return sum(int(L) for L in lens) * H * 512 + B * Hq * 128 * (2 + 4)


def layers48_measurement(okvq, torch, np, dev, stream, reps=5):
    """The 30B-like workload: 48 layers of 131072 tokens resident at once (4 KV heads, 32 query
    heads), one decode step per layer. Each layer's inputs are generated on the device with its own
    seed (synth.device) and appended into its own packed cache; the same fp16 K and V stay resident
    for the dense fp16 baseline (12.9 GB), and a second set of packed caches uses the single global
    value rotation R_m = H_v (a randomized Hadamard with its own signs) for every modality."""
    from synth import gen_signs, workload
    from synth.device import gen_layer_device
    wl = workload("omni30b_128k_48layer")
    B, H, Hq, N, nl = wl.batch, wl.num_kv_heads, wl.num_q_heads, wl.seq_len, wl.layers
    sm = 1 / math.sqrt(128)
    lens = [N] * B
    n_new = torch.tensor(lens, dtype=torch.int32, device=dev)
    packed, glob, dk, dv, qs, app = [], [], [], [], [], []
    for layer in range(nl):
        lay = gen_layer_device(wl, layer, dev)
        signs = torch.from_numpy(lay["signs"])
        hv = torch.from_numpy(sylvester_hadamard(gen_signs(wl.wid, 1000 + layer))).repeat(3, 1, 1)
        c = okvq.KVCache(B, H, Hq, wl.capacity, signs, torch.from_numpy(lay["rot"]), device=dev)
        cg = okvq.KVCache(B, H, Hq, wl.capacity, signs, hv, device=dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        okvq.okvq_append(c, [0] * B, lay["k"], lay["v"], lay["modality"], lens, n_new, N, stream=stream)
        e1.record(stream)
        okvq.okvq_append(cg, [0] * B, lay["k"], lay["v"], lay["modality"], lens, n_new, N,
                         flags=okvq.okvq.OKVQ_GLOBAL_ROTATION, stream=stream)
        app.append((e0, e1))
        packed.append(c)
        glob.append(cg)
        dk.append(lay["k"])
        dv.append(lay["v"])
        qs.append(torch.from_numpy(lay["q"]).to(dev))
        torch.cuda.synchronize()
    append_us = float(np.mean([a.elapsed_time(b) for a, b in app[2:]])) * 1e3
    ws = okvq.decode_workspace(packed[0].dims, N, device=dev)
    ddims = okvq.make_dims(B, H, Hq, N)
    dws = okvq.dense_workspace(ddims, N, device=dev)
    seq = torch.tensor(lens, dtype=torch.int32, device=dev)
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)

    def packed_call(layer, caches=packed, events=None, flags=0):
        if events is None:
            okvq.okvq_decode_attention(caches[layer], lens, qs[layer], sm, out, ws, flags=flags, stream=stream)
        else:
            okvq.okvq_decode_attention_timed(caches[layer], lens, qs[layer], sm, out, ws, events, flags=flags,
                                             stream=stream)

    def global_call(layer, events=None):
        packed_call(layer, glob, events, okvq.okvq.OKVQ_GLOBAL_ROTATION)

    def dense_call(layer, events=None):
        okvq.okvq_decode_attention_dense(ddims, dk[layer], dv[layer], seq, lens, qs[layer], sm, out, dws,
                                         events=events, stream=stream)

    def sweep(fn):
        """median µs of one decode step over all 48 layers, back to back"""
        for layer in range(nl):
            fn(layer)
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for layer in range(nl):
                fn(layer)
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3)
        return float(np.median(ts)), float(np.min(ts))

    def kernel_us(fn):
        """mean duration of the split-K kernel and of the merge over one sweep (events bound to them)"""
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(nl)]
        for e4 in evs:
            for e in e4:
                e.record(stream)
        torch.cuda.synchronize()
        for layer in range(nl):
            fn(layer, events=evs[layer])
        torch.cuda.synchronize()
        return (float(np.mean([e[0].elapsed_time(e[1]) for e in evs])) * 1e3,
                float(np.mean([e[2].elapsed_time(e[3]) for e in evs])) * 1e3)

    def latency(fn):
        lat = []
        for i in range(20):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn(i % nl)
            torch.cuda.synchronize()
            lat.append((time.perf_counter() - t0) * 1e6)
        return float(np.median(lat))

    pk = decode_algorithmic_bytes(B, H, Hq, lens)
    pk_split = decode_algorithmic_bytes(B, H, Hq, lens, with_output=False)
    dn = dense_decode_bytes(B, H, Hq, lens)
    dn_split = dn - B * Hq * 128 * 4
    t_packed, t_packed_min = sweep(packed_call)
    t_glob, t_glob_min = sweep(global_call)
    t_dense, t_dense_min = sweep(dense_call)
    ks, km = kernel_us(packed_call)
    gs, gm = kernel_us(global_call)
    ds, dm = kernel_us(dense_call)
    res = {
        "workload": "omni30b_128k_48layer", "layers": nl, "batch": B, "kv_heads": H, "q_heads": Hq, "seq_len": N,
        "data": "synthetic, generated on the device per layer (same recipe, torch generator)",
        "resident_GB": {"packed": round(nl * sum(okvq.okvq_buffer_bytes(packed[0].dims, i) for i in range(10)) / 1e9, 3),
                        "dense_fp16": round(nl * 2 * B * H * N * 256 / 1e9, 3)},
        "packed": {"decode_us_all_layers": round(t_packed, 2), "decode_us_all_layers_min": round(t_packed_min, 2),
                   "decode_us_per_layer": round(t_packed / nl, 3),
                   "GBps": round(pk * nl / t_packed / 1e3, 1), "k_decode_us": round(ks, 3),
                   "k_decode_merge_us": round(km, 3), "k_decode_frac": round(pk_split / ks / 1e3 / HBM_PEAK_GBPS, 4),
                   "latency_us_per_layer": round(latency(packed_call), 2), "append_us_per_layer": round(append_us, 2),
                   "algorithmic_bytes_per_layer": pk},
        "global_rotation": {"flag": "OKVQ_GLOBAL_ROTATION", "decode_us_all_layers": round(t_glob, 2),
                            "decode_us_all_layers_min": round(t_glob_min, 2),
                            "decode_us_per_layer": round(t_glob / nl, 3), "k_decode_us": round(gs, 3),
                            "k_decode_merge_us": round(gm, 3),
                            "k_decode_frac": round(pk_split / gs / 1e3 / HBM_PEAK_GBPS, 4)},
        "dense_fp16": {"decode_us_all_layers": round(t_dense, 2), "decode_us_all_layers_min": round(t_dense_min, 2),
                       "decode_us_per_layer": round(t_dense / nl, 3),
                       "GBps": round(dn * nl / t_dense / 1e3, 1), "k_decode_dense_us": round(ds, 3),
                       "merge_us": round(dm, 3), "k_decode_dense_frac": round(dn_split / ds / 1e3 / HBM_PEAK_GBPS, 4),
                       "latency_us_per_layer": round(latency(dense_call), 2), "algorithmic_bytes_per_layer": dn,
                       "traffic": measured_traffic("k_decode_dense")},
        "speedup_packed_vs_dense": round(t_dense / t_packed, 3),
    }
    del packed, glob, dk, dv
    torch.cuda.empty_cache()
    return res


def ragged_measurement(okvq, torch, np, dev, stream, decode_iters):
    """Batch 16 with ragged lengths U[8192, 16384] at the 7B-like head shapes (4 KV heads, 28 query
    heads): the rows generated on the device from the workload's recipe, each sequence's prefill
    (its own length, its own modality layout ending in the text prompt) appended into an empty
    cache, then decode over >= 1 GB of cold cache replicas, and the split-K kernel's duration from
    events bound to its dispatch."""
    from synth import gen_lengths, gen_queries, modality_layout, workload
    from synth.device import gen_layer_device
    wl = workload("omni7b_b16_ragged16k")
    B, H, Hq = wl.batch, wl.num_kv_heads, wl.num_q_heads
    lens = [int(x) for x in gen_lengths(wl)]
    lay = gen_layer_device(wl, 0, dev)
    N = lay["k"].shape[2]
    mod = np.zeros((B, N), np.uint8)
    for b, L in enumerate(lens):
        mod[b, :L] = modality_layout(L, wl.video_per_chunk, wl.audio_per_chunk, wl.text_tail)
    m_in = torch.from_numpy(mod).to(dev)
    sm = 1 / math.sqrt(128)
    signs = torch.from_numpy(lay["signs"])
    rot = torch.from_numpy(lay["rot"])
    base = okvq.KVCache(B, H, Hq, wl.capacity, signs, rot, device=dev)
    n_new = torch.tensor(lens, dtype=torch.int32, device=dev)
    okvq.okvq_append(base, [0] * B, lay["k"], lay["v"], m_in, lens, n_new, N, stream=stream)
    torch.cuda.synchronize()
    del lay
    per_cache = sum(okvq.okvq_buffer_bytes(base.dims, i) for i in range(10))
    n_cache = max(8, int(math.ceil(1.05e9 / per_cache)))
    caches = [base] + [okvq.KVCache(B, H, Hq, wl.capacity, signs, rot, device=dev) for _ in range(n_cache - 1)]
    for c in caches[1:]:
        for name in c.buffers:
            c.buffers[name].copy_(base.buffers[name])
    q = torch.from_numpy(gen_queries(wl.wid, 0, B, Hq)).to(dev)
    ws = okvq.decode_workspace(base.dims, max(lens), device=dev)
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
    reps = []
    for rep in range(5):
        for i in range(10):
            okvq.okvq_decode_attention(caches[i % n_cache], lens, q, sm, out, ws, stream=stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(decode_iters):
            okvq.okvq_decode_attention(caches[(i * 5 + rep) % n_cache], lens, q, sm, out, ws, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        reps.append(e0.elapsed_time(e1) * 1e3 / decode_iters)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(decode_iters)]
    for e4 in evs:
        for e in e4:
            e.record(stream)
    torch.cuda.synchronize()
    for i in range(decode_iters):
        okvq.okvq_decode_attention_timed(caches[(i * 5 + 3) % n_cache], lens, q, sm, out, ws, evs[i], stream=stream)
    torch.cuda.synchronize()
    split_us = float(np.mean([e[0].elapsed_time(e[1]) for e in evs])) * 1e3
    merge_us = float(np.mean([e[2].elapsed_time(e[3]) for e in evs])) * 1e3
    dbytes = decode_algorithmic_bytes(B, H, Hq, lens)
    sbytes = decode_algorithmic_bytes(B, H, Hq, lens, with_output=False)
    decode_us = float(np.median(reps))
    res = {"workload": wl.name, "batch": B, "kv_heads": H, "q_heads": Hq,
           "lengths_min_max_mean": [min(lens), max(lens), round(float(np.mean(lens)), 1)],
           "algorithmic_bytes": dbytes, "decode_us": round(decode_us, 3),
           "decode_us_min": round(float(np.min(reps)), 3), "decode_GBps": round(dbytes / decode_us / 1e3, 1),
           "k_decode_us": round(split_us, 3), "k_decode_merge_us": round(merge_us, 3),
           "k_decode_GBps": round(sbytes / split_us / 1e3, 1),
           "k_decode_frac": round(sbytes / split_us / 1e3 / HBM_PEAK_GBPS, 4), "replicas": n_cache,
           "replica_GB": round(n_cache * per_cache / 1e9, 2)}
    del caches, base
    torch.cuda.empty_cache()
    return res


def residual_measurement(okvq, torch, np, wl, lens, k_in, v_in, m0, n_new_dev, q, stream, decode_iters):
    """The benchmark workload in the captioning protocol (Sec. 3.1): fp16 rings of the last 128 keys
    and values next to the packed cache. Prefill append, one-token append (a generation step), and
    decode over >= 1 GB of cold cache replicas with the per-launch durations."""
    B, H, Hq, N = wl.batch, wl.num_kv_heads, wl.num_q_heads, wl.seq_len
    dev = q.device
    sm = 1 / math.sqrt(128)
    cap = wl.capacity + 32                                   # room for the generated token
    dims = okvq.make_dims(B, H, Hq, cap, residual=128)
    per_cache = sum(okvq.okvq_buffer_bytes(dims, i) for i in range(12))
    n_cache = max(16, int(math.ceil(1.05e9 / per_cache)))
    mk = lambda: okvq.KVCache(B, H, Hq, cap, torch.ones(128, dtype=torch.int8), torch.eye(128).repeat(3, 1, 1),
                              device=dev, residual=128)
    caches = [mk() for _ in range(n_cache)]
    okvq.okvq_append(caches[0], [0] * B, k_in[0], v_in[0], m0, lens, n_new_dev, N, stream=stream)
    torch.cuda.synchronize()
    for c in caches[1:]:
        for name in c.buffers:
            c.buffers[name].copy_(caches[0].buffers[name])
    ws = okvq.decode_workspace(dims, max(lens), device=dev)
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
    app = []
    for i in range(12):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c = caches[(i + 1) % n_cache]
        c.buffers["seq_lens"].zero_()
        e0.record(stream)
        okvq.okvq_append(c, [0] * B, k_in[i % len(k_in)], v_in[i % len(v_in)], m0, lens, n_new_dev, N, stream=stream)
        e1.record(stream)
        app.append((e0, e1))
    torch.cuda.synchronize()
    append_us = float(np.mean([a.elapsed_time(b) for a, b in app[2:]])) * 1e3
    # one generated token appended at length N (then the length is set back, on the stream)
    k1 = k_in[0][:, :, :1].contiguous()
    v1 = v_in[0][:, :, :1].contiguous()
    m1 = m0[:, :1].contiguous()
    one = torch.ones(B, dtype=torch.int32, device=dev)
    back = torch.tensor(lens, dtype=torch.int32, device=dev)
    app1 = []
    for i in range(40):
        c = caches[(3 * i + 2) % n_cache]
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        okvq.okvq_append(c, lens, k1, v1, m1, [1] * B, one, 1, stream=stream)
        e1.record(stream)
        c.buffers["seq_lens"][:B].copy_(back)
        app1.append((e0, e1))
    torch.cuda.synchronize()
    append1_us = float(np.median([a.elapsed_time(b) for a, b in app1[5:]])) * 1e3
    # the same with the GPU kept busy while the host enqueues the timed append (device-side latency)
    app1d = []
    for i in range(25):
        c = caches[(3 * i + 2) % n_cache]
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(200000)
        e0.record(stream)
        okvq.okvq_append(c, lens, k1, v1, m1, [1] * B, one, 1, stream=stream)
        e1.record(stream)
        c.buffers["seq_lens"][:B].copy_(back)
        app1d.append((e0, e1))
    torch.cuda.synchronize()
    append1_dev_us = float(np.median([a.elapsed_time(b) for a, b in app1d[5:]])) * 1e3
    app1k = []  # the append kernel alone: events bound to its dispatch (okvq_append_timed)
    for i in range(25):
        c = caches[(3 * i + 2) % n_cache]
        e2 = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        for e in e2:
            e.record(stream)
        okvq.okvq_append_timed(c, lens, k1, v1, m1, [1] * B, one, 1, e2, stream=stream)
        c.buffers["seq_lens"][:B].copy_(back)
        app1k.append(e2)
    torch.cuda.synchronize()
    append1_kern_us = float(np.median([a.elapsed_time(b) for a, b in app1k[5:]])) * 1e3
    reps = []
    for rep in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for i in range(20):
            okvq.okvq_decode_attention(caches[i % n_cache], lens, q, sm, out, ws, stream=stream)
        e0.record(stream)
        for i in range(decode_iters):
            okvq.okvq_decode_attention(caches[(i * 7 + rep) % n_cache], lens, q, sm, out, ws, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        reps.append(e0.elapsed_time(e1) * 1e3 / decode_iters)
    decode_us, decode_us_min = float(np.median(reps)), float(np.min(reps))
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(decode_iters)]
    for e4 in evs:
        for e in e4:
            e.record(stream)
    torch.cuda.synchronize()
    for i in range(decode_iters):
        okvq.okvq_decode_attention_timed(caches[(i * 7 + 5) % n_cache], lens, q, sm, out, ws, evs[i], stream=stream)
    torch.cuda.synchronize()
    split_us = float(np.mean([e[0].elapsed_time(e[1]) for e in evs])) * 1e3
    merge_us = float(np.mean([e[2].elapsed_time(e[3]) for e in evs])) * 1e3
    dbytes = residual_decode_algorithmic_bytes(B, H, Hq, lens)
    del caches
    return {"protocol": "captioning: keys quantized per 128-token block, last 128 values fp16",
            "decode_us": round(decode_us, 3), "decode_us_min": round(decode_us_min, 3),
            "decode_GBps": round(dbytes / decode_us / 1e3, 2),
            "k_decode_us": round(split_us, 3), "k_decode_merge_residual_us": round(merge_us, 3),
            "append_prefill_us": round(append_us, 3), "append_one_token_us": round(append1_us, 3),
            "append_one_token_device_us": round(append1_dev_us, 3),
            "append_one_token_kernel_us": round(append1_kern_us, 3),
            "algorithmic_bytes": dbytes, "replicas": n_cache}


CALIB_TOKENS = 4096


def calibration_measurement(okvq, torch, np, wl, dev):
    """Value-rotation calibration (Eq. 5, Eq. 6) at the benchmark layer's head shapes on one
    4096-token calibration sequence: attention weights (row statistics and column sums on the
    matrix cores), weighted covariance, and the host eigensolver."""
    from synth import gen_calibration_queries, gen_layer
    H, Hq, N = wl.num_kv_heads, wl.num_q_heads, CALIB_TOKENS
    lay = gen_layer(wl, 1, lengths=np.array([N], np.int32), n_tokens=N)
    q = torch.from_numpy(gen_calibration_queries(wl.wid, 1, 1, Hq, N)).to(dev)
    k = torch.from_numpy(lay["k"]).to(dev)
    v = torch.from_numpy(lay["v"]).to(dev)
    mod = torch.from_numpy(lay["modality"]).to(dev)
    dims = okvq.make_dims(1, H, Hq, 32)
    ws = okvq.calibration_workspace(dims, N, device=dev)
    w = torch.empty((1, H, N), dtype=torch.float32, device=dev)
    cov = torch.empty((3, 128, 128), dtype=torch.float32, device=dev)
    sm = 1 / math.sqrt(128)
    for _ in range(3):
        okvq.okvq_calibration_weights(dims, q, k, N, [N], sm, w, ws)
        okvq.okvq_value_covariance(dims, v, mod, w, N, [N], cov, ws)
    torch.cuda.synchronize()
    reps = 10
    e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    e[0].record()
    for _ in range(reps):
        okvq.okvq_calibration_weights(dims, q, k, N, [N], sm, w, ws)
    e[1].record()
    for _ in range(reps):
        okvq.okvq_value_covariance(dims, v, mod, w, N, [N], cov, ws)
    e[2].record()
    torch.cuda.synchronize()
    weights_us = e[0].elapsed_time(e[1]) * 1e3 / reps
    cov_us = e[1].elapsed_time(e[2]) * 1e3 / reps
    c_host = cov.cpu().numpy()
    rot = np.zeros((3, 128, 128), np.float32)
    t0 = time.perf_counter()
    okvq.okvq_rotation_from_covariance(c_host, np.ascontiguousarray(lay["signs"], np.int8), rot)
    eig_ms = (time.perf_counter() - t0) * 1e3
    # algorithmic work of the weights: two passes over the causal score triangle of every query head
    flops = 2 * Hq * (N * (N + 1) // 2) * 128 * 2
    tflops = flops / weights_us / 1e6
    return {"tokens": N, "kv_heads": H, "q_heads": Hq, "weights_us": round(weights_us, 2),
            "weights_roofline": {"bound": "mfma", "achieved": round(tflops, 1), "peak": 2500.0, "unit": "TFLOP/s",
                                 "frac": round(tflops / 2500.0, 4), "algorithmic_flops": flops},
            "covariance_us": round(cov_us, 2), "eigensolver_host_ms": round(eig_ms, 1)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--decode-iters", type=int, default=200)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-layers48", action="store_true", help="skip the 48-layer 131072-token measurement")
    ap.add_argument("--profile-pass", action="store_true", help="short fixed sequence for rocprofv3 --pmc runs")
    ap.add_argument("--shape-scan", action="store_true", help="decode throughput at the other workload shapes")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the path shards by KV head "
              "or by whole windows, see the design notes)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_11582_amd as okvq
    from synth import gen_layer, gen_lengths, gen_queries, workload

    if args.shape_scan:
        shape_scan(okvq, torch, workload, gen_lengths)
        return

    wl = workload(WORKLOAD)
    B, H, Hq, N = wl.batch, wl.num_kv_heads, wl.num_q_heads, wl.seq_len
    lay = gen_layer(wl, 0)
    lens = [int(x) for x in lay["lens"]]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    signs = torch.from_numpy(lay["signs"])
    rot = torch.from_numpy(lay["rot"])

    # input replicas (the append reads fp16 K/V that are cold in HBM: 8 x 67 MB)
    n_in = 8
    k0 = torch.from_numpy(lay["k"]).to(dev)
    v0 = torch.from_numpy(lay["v"]).to(dev)
    m0 = torch.from_numpy(lay["modality"]).to(dev)
    k_in = [k0.clone() for _ in range(n_in)]
    v_in = [v0.clone() for _ in range(n_in)]
    n_new_dev = torch.tensor(lens, dtype=torch.int32, device=dev)

    # cache replicas (>= 1 GB of packed caches so that decode reads come from HBM)
    per_cache = sum(okvq.okvq_buffer_bytes(okvq.make_dims(B, H, Hq, wl.capacity), i) for i in range(10))
    n_cache = max(16, int(math.ceil(1.05e9 / per_cache)))
    caches = [okvq.KVCache(B, H, Hq, wl.capacity, signs, rot, device=dev) for _ in range(n_cache)]
    okvq.okvq_append(caches[0], [0] * B, k_in[0], v_in[0], m0, lens, n_new_dev, N)
    torch.cuda.synchronize()
    for c in caches[1:]:
        for name in c.buffers:
            c.buffers[name].copy_(caches[0].buffers[name])
    q = torch.from_numpy(gen_queries(wl.wid, 0, B, Hq)).to(dev)
    ws = okvq.decode_workspace(caches[0].dims, max(lens), device=dev)
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
    sm = 1 / math.sqrt(128)

    def append_into(ci, ii):
        caches[ci].buffers["seq_lens"].zero_()
        okvq.okvq_append(caches[ci], [0] * B, k_in[ii], v_in[ii], m0, lens, n_new_dev, N, stream=stream)

    def decode(ci):
        okvq.okvq_decode_attention(caches[ci], lens, q, sm, out, ws, stream=stream)

    if args.profile_pass:
        src = torch.empty(CALIBRATION_COPY_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)  # one copy kernel of known size: reads and writes CALIBRATION_COPY_BYTES
        torch.cuda.synchronize()
        for i in range(8):
            decode((7 * i + 3) % n_cache)
        torch.cuda.synchronize()
        for i in range(2):
            append_into((i + 1) % n_cache, (i + 1) % n_in)
        torch.cuda.synchronize()
        # the same with MXFP4 key metadata
        mx = [okvq.KVCache(B, H, Hq, wl.capacity, signs, rot, device=dev, key_meta="mxfp4") for _ in range(16)]
        okvq.okvq_append(mx[0], [0] * B, k_in[0], v_in[0], m0, lens, n_new_dev, N, stream=stream)
        torch.cuda.synchronize()
        for c in mx[1:]:
            for name in c.buffers:
                c.buffers[name].copy_(mx[0].buffers[name])
        ws_mx = okvq.decode_workspace(mx[0].dims, max(lens), device=dev)
        torch.cuda.synchronize()
        for i in range(8):
            okvq.okvq_decode_attention(mx[(7 * i + 3) % 16], lens, q, sm, out, ws_mx, stream=stream)
        torch.cuda.synchronize()
        for i in range(2):
            mx[i + 1].buffers["seq_lens"].zero_()
            okvq.okvq_append(mx[i + 1], [0] * B, k_in[i + 1], v_in[i + 1], m0, lens, n_new_dev, N, stream=stream)
        torch.cuda.synchronize()
        del mx
        # the fp16 residual (captioning protocol): 8 decode calls on cold replicas
        res = [okvq.KVCache(B, H, Hq, wl.capacity, signs, rot, device=dev, residual=128) for _ in range(16)]
        okvq.okvq_append(res[0], [0] * B, k_in[0], v_in[0], m0, lens, n_new_dev, N, stream=stream)
        torch.cuda.synchronize()
        for c in res[1:]:
            for name in c.buffers:
                c.buffers[name].copy_(res[0].buffers[name])
        ws_res = okvq.decode_workspace(res[0].dims, max(lens), device=dev)
        torch.cuda.synchronize()
        for i in range(8):
            okvq.okvq_decode_attention(res[(7 * i + 3) % 16], lens, q, sm, out, ws_res, stream=stream)
        torch.cuda.synchronize()
        del res
        # TurboQuant keys (no window metadata)
        tq = [okvq.KVCache(B, H, Hq, wl.capacity, signs, rot, device=dev, key_meta="turboquant") for _ in range(16)]
        okvq.okvq_append(tq[0], [0] * B, k_in[0], v_in[0], m0, lens, n_new_dev, N, stream=stream)
        torch.cuda.synchronize()
        for c in tq[1:]:
            for name in c.buffers:
                c.buffers[name].copy_(tq[0].buffers[name])
        ws_tq = okvq.decode_workspace(tq[0].dims, max(lens), device=dev)
        torch.cuda.synchronize()
        for i in range(8):
            okvq.okvq_decode_attention(tq[(7 * i + 3) % 16], lens, q, sm, out, ws_tq, stream=stream)
        torch.cuda.synchronize()
        for i in range(2):
            tq[i + 1].buffers["seq_lens"].zero_()
            okvq.okvq_append(tq[i + 1], [0] * B, k_in[i + 1], v_in[i + 1], m0, lens, n_new_dev, N, stream=stream)
        torch.cuda.synchronize()
        del tq
        # the dense fp16 baseline at the 30B-like layer shape: 4 calls alternating over two layers' K
        # and V (537 MB, beyond the 256 MB Infinity Cache)
        from synth.device import gen_layer_device
        w5 = workload("omni30b_128k_48layer")
        l5 = [gen_layer_device(w5, i, dev) for i in range(2)]
        d5 = okvq.make_dims(w5.batch, w5.num_kv_heads, w5.num_q_heads, w5.seq_len)
        lens5 = [w5.seq_len] * w5.batch
        ws5 = okvq.dense_workspace(d5, w5.seq_len, device=dev)
        q5 = torch.from_numpy(l5[0]["q"]).to(dev)
        s5 = torch.tensor(lens5, dtype=torch.int32, device=dev)
        o5 = torch.empty((w5.batch, w5.num_q_heads, 128), dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        for i in range(4):
            okvq.okvq_decode_attention_dense(d5, l5[i % 2]["k"], l5[i % 2]["v"], s5, lens5, q5, sm, o5, ws5,
                                             stream=stream)
        torch.cuda.synchronize()
        # the prefill's keys and values through the stateless codec calls (one role per launch), twice
        # each, and 8 one-token appends through the window-parallel launch (lengths set to N - 1 first)
        c0 = caches[0]
        v0w = c0.views()
        for i in range(2):
            okvq.okvq_quantize_keys(c0.dims, k_in[i], N, lens, c0.key_signs, v0w["k_codes"], v0w["k_min"],
                                    v0w["k_step"], v0w["k_norm"], stream=stream)
            okvq.okvq_quantize_values(c0.dims, v_in[i], m0, N, lens, c0.v_rot, 0, v0w["v_codes"], v0w["v_norm"],
                                      stream=stream)
        torch.cuda.synchronize()
        k1 = k_in[0][:, :, :1].contiguous()
        v1 = v_in[0][:, :, :1].contiguous()
        m1 = m0[:, :1].contiguous()
        one = torch.ones(B, dtype=torch.int32, device=dev)
        short = torch.tensor([L - 1 for L in lens], dtype=torch.int32, device=dev)
        for i in range(8):
            c = caches[(5 * i + 1) % n_cache]
            c.buffers["seq_lens"][:B].copy_(short)
            okvq.okvq_append(c, [L - 1 for L in lens], k1, v1, m1, [1] * B, one, 1, stream=stream)
        torch.cuda.synchronize()
        print(json.dumps({"profile_pass": True, "copy_bytes": CALIBRATION_COPY_BYTES, "decode_calls": 8,
                          "append_calls": 2, "stateless_key_calls": 2, "stateless_value_calls": 2,
                          "one_token_append_calls": 8, "decode_algorithmic_bytes": decode_algorithmic_bytes(B, H, Hq, lens),
                          "append_algorithmic_bytes": append_algorithmic_bytes(B, H, lens),
                          "mxfp4_decode_calls": 8, "mxfp4_append_calls": 2, "residual_decode_calls": 8,
                          "turboquant_decode_calls": 8, "turboquant_append_calls": 2, "dense_decode_calls": 4,
                          "dense_decode_algorithmic_bytes": dense_decode_bytes(1, 4, 32, [131072]),
                          "residual_decode_algorithmic_bytes": residual_decode_algorithmic_bytes(B, H, Hq, lens)}),
              flush=True)
        return

    # ---- steps: append the prefill into cache replica s, decode a cold replica ----
    for s in range(args.warmup):
        append_into(s % n_cache, s % n_in)
        decode((s + n_cache // 2) % n_cache)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for s in range(args.steps):
        i = s + args.warmup
        ev[s][0].record(stream)
        append_into(i % n_cache, i % n_in)
        ev[s][1].record(stream)
        decode((i + n_cache // 2) % n_cache)
        ev[s][2].record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_wall) * 1e3
    append_ms = [ev[s][0].elapsed_time(ev[s][1]) for s in range(args.steps)]
    decode_step_ms = [ev[s][1].elapsed_time(ev[s][2]) for s in range(args.steps)]
    step_ms = [ev[s][0].elapsed_time(ev[s][2]) for s in range(args.steps)]

    # ---- steady-state decode over cold replicas (median of 5 repetitions) ----
    reps = []
    for rep in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for i in range(20):
            decode(i % n_cache)
        e0.record(stream)
        for i in range(args.decode_iters):
            decode((i * 7 + rep) % n_cache)
        e1.record(stream)
        torch.cuda.synchronize()
        reps.append(e0.elapsed_time(e1) * 1e3 / args.decode_iters)
    decode_us, decode_us_min = float(np.median(reps)), float(np.min(reps))

    # per-launch durations: HIP events bound to the split-K and merge dispatches (start and end of
    # each kernel's execution, as the profiler sees them), over cold replicas
    n_ev = args.decode_iters
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(n_ev)]
    for e3 in evs:
        for e in e3:
            e.record(stream)  # creates the event handle
    torch.cuda.synchronize()
    for i in range(n_ev):
        okvq.okvq_decode_attention_timed(caches[(i * 7 + 5) % n_cache], lens, q, sm, out, ws, evs[i], stream=stream)
    torch.cuda.synchronize()
    split_us = float(np.mean([evs[i][0].elapsed_time(evs[i][1]) for i in range(n_ev)])) * 1e3
    merge_us = float(np.mean([evs[i][2].elapsed_time(evs[i][3]) for i in range(n_ev)])) * 1e3

    # single-call latency including dispatch
    lat = []
    for i in range(30):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        decode(i % n_cache)
        torch.cuda.synchronize()
        lat.append((time.perf_counter() - t0) * 1e6)

    dbytes = decode_algorithmic_bytes(B, H, Hq, lens)
    split_bytes = decode_algorithmic_bytes(B, H, Hq, lens, with_output=False)  # the merge writes the output
    split_gbps = split_bytes / (split_us * 1e-6) / 1e9
    abytes = append_algorithmic_bytes(B, H, lens)
    decode_gbps = dbytes / (decode_us * 1e-6) / 1e9
    append_us = float(np.mean(append_ms)) * 1e3
    append_gbps = abytes / (append_us * 1e-6) / 1e9

    line = {
        "metric": METRIC,
        "value": round(decode_gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(float(np.mean(step_ms)), 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "batch": B, "kv_heads": H, "q_heads": Hq, "head_dim": 128,
                   "seq_len": N, "key_window": 32, "bits": 2, "modalities": "150 video + 25 audio per chunk, "
                   "256 text"},
        "decode_us": round(decode_us, 3),
        "decode_us_min": round(decode_us_min, 3),
        "decode_us_in_step": round(float(np.mean(decode_step_ms)) * 1e3, 3),
        "decode_latency_us": round(float(np.median(lat)), 2),
        "append_us": round(append_us, 3),
        "append_GBps": round(append_gbps, 2),
        "wall_ms_timed_steps": round(wall_ms, 3),
        "roofline": {"bound": "hbm", "achieved": round(split_gbps, 2), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(split_gbps / HBM_PEAK_GBPS, 4), "traffic": measured_traffic("k_decode"),
                     "kernel": "k_decode (split-K decode attention with per-split inverse rotation)",
                     "algorithmic_bytes": split_bytes, "avg_launch_us": round(split_us, 3)},
        "kernels_us": {"k_decode": round(split_us, 3), "k_decode_merge": round(merge_us, 3)},
        "roofline_append": {"bound": "hbm", "achieved": round(append_gbps, 2), "peak": HBM_PEAK_GBPS,
                            "unit": "GB/s", "frac": round(append_gbps / HBM_PEAK_GBPS, 4),
                            "traffic": None,
                            "kernel": "okvq_append (fused key + value codec launch, length update)",
                            "algorithmic_bytes": abytes},
        "cache_replicas": n_cache,
    }
    line["codec_split"] = codec_split_measurement(okvq, torch, np, wl, lens, k_in, v_in, m0, signs, rot, stream)
    line["mxfp4"] = key_meta_measurement(okvq, torch, np, wl, lens, k_in, v_in, m0, n_new_dev, q, stream,
                                         args.decode_iters, "mxfp4")
    line["turboquant"] = key_meta_measurement(okvq, torch, np, wl, lens, k_in, v_in, m0, n_new_dev, q, stream,
                                              args.decode_iters, "turboquant", signs,
                                              torch.from_numpy(sylvester_hadamard(lay["signs"])).repeat(3, 1, 1),
                                              flags=okvq.okvq.OKVQ_GLOBAL_ROTATION)
    line["ladder"] = ladder_measurement(okvq, torch, np, wl, lens, k_in, v_in, m0, q, signs, rot, stream,
                                        args.decode_iters)
    line["calibration"] = calibration_measurement(okvq, torch, np, wl, dev)
    if not args.no_layers48:
        line["omni30b_48layer"] = layers48_measurement(okvq, torch, np, dev, stream)
    line["b16_ragged"] = ragged_measurement(okvq, torch, np, dev, stream, args.decode_iters)
    line["stream"] = stream_measurement(okvq, torch, np, dev, stream)
    line["residual"] = residual_measurement(okvq, torch, np, wl, lens, k_in, v_in, m0, n_new_dev, q, stream,
                                            args.decode_iters)
    if not args.no_cpu_baseline:
        cache_np = {n: t.cpu().numpy() for n, t in caches[0].views().items()}
        line["cpu_baseline"] = cpu_baseline(cache_np, q.cpu().numpy(), np.asarray(lens), lay["signs"], lay["rot"],
                                            dbytes, prefill=(lay["k"], lay["v"], lay["modality"]),
                                            append_bytes=abytes)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
