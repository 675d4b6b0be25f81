"""Run the HIP library on numpy inputs and bring results back as numpy (for the GPU tests)."""

from __future__ import annotations

import math

import numpy as np
import torch

import paper_2609_11582_amd as okvq


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.view(dtype) if t.element_size() == torch.tensor([], dtype=dtype).element_size() else t.to(dtype)
    return t.cuda()


def f16dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float16)).cuda()


def host(t, np_dtype=None):
    a = t.cpu().numpy()
    return a if np_dtype is None else a.view(np_dtype)


def quantize_stateless(k, v, modality, lens, signs, rot, capacity, num_q_heads, exact=False):
    """Stateless key + value calls on dense blocks -> dict of numpy arrays in cache layout."""
    B, H, N, D = k.shape
    dims = okvq.make_dims(B, H, num_q_heads, capacity)
    out = dict(
        k_codes=torch.zeros((B, H, capacity, 32), dtype=torch.uint8, device="cuda"),
        v_codes=torch.zeros((B, H, capacity // 32, 1024), dtype=torch.uint8, device="cuda"),
        k_norm=torch.zeros((B, H, capacity), dtype=torch.float16, device="cuda"),
        v_norm=torch.zeros((B, H, capacity), dtype=torch.float16, device="cuda"),
        k_min=torch.zeros((B, H, capacity // 32, 128), dtype=torch.float16, device="cuda"),
        k_step=torch.zeros((B, H, capacity // 32, 128), dtype=torch.float16, device="cuda"),
    )
    kd, vd = f16dev(k), f16dev(v)
    md = dev(np.ascontiguousarray(modality, np.uint8))
    sd = dev(np.ascontiguousarray(signs, np.int8))
    rd = dev(np.ascontiguousarray(rot, np.float32))
    okvq.okvq_quantize_keys(dims, kd, N, list(lens), sd, out["k_codes"], out["k_min"], out["k_step"], out["k_norm"])
    okvq.okvq_quantize_values(dims, vd, md, N, list(lens), rd, okvq.okvq.OKVQ_VALUE_EXACT if exact else 0,
                              out["v_codes"], out["v_norm"])
    torch.cuda.synchronize()
    res = {n: t.cpu().numpy() for n, t in out.items()}
    mod = np.zeros((B, capacity), np.uint8)
    for b in range(B):
        mod[b, :lens[b]] = modality[b, :lens[b]]
    res["modality"] = mod
    return res


def new_cache(B, H, Hq, capacity, signs, rot):
    return okvq.KVCache(B, H, Hq, capacity, torch.from_numpy(np.asarray(signs, np.int8)),
                        torch.from_numpy(np.asarray(rot, np.float32)))


def append_chunks(cache, k, v, modality, lens, chunk_plan, exact=False):
    """Append each sequence in the given chunks. chunk_plan: list of per-step token counts [B]."""
    B, H, N, D = k.shape
    cur = np.zeros(B, np.int64)
    for step in chunk_plan:
        n_new = np.minimum(np.asarray(step), np.asarray(lens) - cur).clip(0)
        n_max = max(int(n_new.max()), 1)
        kn = np.zeros((B, H, n_max, D), np.float16)
        vn = np.zeros((B, H, n_max, D), np.float16)
        mn = np.zeros((B, n_max), np.uint8)
        for b in range(B):
            a, c = int(cur[b]), int(cur[b] + n_new[b])
            kn[b, :, :c - a] = k[b, :, a:c]
            vn[b, :, :c - a] = v[b, :, a:c]
            mn[b, :c - a] = modality[b, a:c]
        nd = dev(n_new.astype(np.int32))
        okvq.okvq_append(cache, cur.astype(np.int32).tolist(), f16dev(kn), f16dev(vn), dev(mn),
                         n_new.astype(np.int32).tolist(), nd, n_max, okvq.okvq.OKVQ_VALUE_EXACT if exact else 0)
        torch.cuda.synchronize()
        cur = cur + n_new
    return cur


def cache_to_numpy(cache):
    return {n: t.cpu().numpy() for n, t in cache.views().items()}


def decode(cache, q, lens, sm_scale=1 / math.sqrt(128)):
    B, Hq, D = q.shape
    ws = okvq.decode_workspace(cache.dims, int(max(lens)))
    out = torch.full((B, Hq, D), float("nan"), dtype=torch.float32, device="cuda")
    okvq.okvq_decode_attention(cache, list(lens), f16dev(q), sm_scale, out, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def load_cache(cache, arrays, lens):
    """Copy numpy cache arrays (oracle layout) into a KVCache's device buffers."""
    views = cache.views()
    for name in ("k_codes", "v_codes", "k_norm", "v_norm", "k_min", "k_step", "modality"):
        views[name].copy_(torch.from_numpy(np.ascontiguousarray(arrays[name])).to(views[name].dtype).cuda()
                          if arrays[name].dtype != np.float16 else torch.from_numpy(arrays[name]).cuda())
    views["seq_lens"].copy_(torch.from_numpy(np.asarray(lens, np.int32)).cuda())
    torch.cuda.synchronize()


def attention_close(out, ref, tol=2e-3):
    """max_c |out - ref| <= tol * ||ref||_2 for every (b, head); returns the worst ratio."""
    err = np.abs(out - ref).max(-1)
    nrm = np.linalg.norm(ref, axis=-1)
    ratio = err / np.maximum(nrm, 1e-30)
    return float(np.nanmax(ratio))
