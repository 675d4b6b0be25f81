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


def quantize_stateless(k, v, modality, lens, signs, rot, capacity, num_q_heads, exact=False, key_meta="fp16"):
    """Stateless key + value calls on dense blocks -> dict of numpy arrays in cache layout."""
    B, H, N, D = k.shape
    dims = okvq.make_dims(B, H, num_q_heads, capacity, key_meta=key_meta)
    out = dict(
        k_codes=torch.zeros((B, H, capacity, 32), dtype=torch.uint8, device="cuda"),
        v_codes=torch.zeros((B, H, capacity // 32, 1024), dtype=torch.uint8, device="cuda"),
        k_norm=torch.zeros((B, H, capacity), dtype=torch.float16, device="cuda"),
        v_norm=torch.zeros((B, H, capacity), dtype=torch.float16, device="cuda"),
    )
    if key_meta == "fp16":
        out["k_min"] = torch.zeros((B, H, capacity // 32, 128), dtype=torch.float16, device="cuda")
        out["k_step"] = torch.zeros((B, H, capacity // 32, 128), dtype=torch.float16, device="cuda")
    elif key_meta == "mxfp4":
        out["k_mx"] = torch.zeros((B, H, capacity // 32, 136), dtype=torch.uint8, device="cuda")
    kd, vd = f16dev(k), f16dev(v)
    md = dev(np.ascontiguousarray(modality, np.uint8))
    sd = dev(np.ascontiguousarray(signs, np.int8))
    rd = dev(np.ascontiguousarray(rot, np.float32))
    if key_meta == "fp16":
        okvq.okvq_quantize_keys(dims, kd, N, list(lens), sd, out["k_codes"], out["k_min"], out["k_step"],
                                out["k_norm"])
    elif key_meta == "mxfp4":
        okvq.okvq_quantize_keys_mx(dims, kd, N, list(lens), sd, out["k_codes"], out["k_mx"], out["k_norm"])
    else:
        okvq.okvq_quantize_keys_tq(dims, kd, N, list(lens), sd, out["k_codes"], out["k_norm"])
    okvq.okvq_quantize_values(dims, vd, md, N, list(lens), rd, okvq.okvq.OKVQ_VALUE_EXACT if exact else 0,
                              out["v_codes"], out["v_norm"])
    torch.cuda.synchronize()
    res = {n: t.cpu().numpy() for n, t in out.items()}
    mod = np.zeros((B, capacity), np.uint8)
    for b in range(B):
        mod[b, :lens[b]] = modality[b, :lens[b]]
    res["modality"] = mod
    return res


def new_cache(B, H, Hq, capacity, signs, rot, key_meta="fp16"):
    return okvq.KVCache(B, H, Hq, capacity, torch.from_numpy(np.asarray(signs, np.int8)),
                        torch.from_numpy(np.asarray(rot, np.float32)), key_meta=key_meta)


def append_chunks(cache, k, v, modality, lens, chunk_plan, exact=False, flags=0, timed=None):
    """Append each sequence in the given chunks. chunk_plan: list of per-step token counts [B].
    flags: more append flags (OKVQ_GLOBAL_ROTATION). timed: a list that receives the codec launch's
    duration (ms) of every step, through okvq_append_timed."""
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
        fl = (okvq.okvq.OKVQ_VALUE_EXACT if exact else 0) | flags
        if timed is not None and n_new.sum() > 0:
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            for e in ev:
                e.record()
            torch.cuda.synchronize()
            okvq.okvq_append_timed(cache, cur.astype(np.int32).tolist(), f16dev(kn), f16dev(vn), dev(mn),
                                   n_new.astype(np.int32).tolist(), nd, n_max, ev, fl)
            torch.cuda.synchronize()
            timed.append(ev[0].elapsed_time(ev[1]))
        else:
            okvq.okvq_append(cache, cur.astype(np.int32).tolist(), f16dev(kn), f16dev(vn), dev(mn),
                             n_new.astype(np.int32).tolist(), nd, n_max, fl)
        torch.cuda.synchronize()
        cur = cur + n_new
    return cur


def append_chunks_from(cache, k, v, modality, cur, n_new, exact=False):
    """One append of n_new[b] tokens per sequence, continuing from the current lengths cur [B]
    (the inputs k, v [B][H][N][D], modality [B][N] are the whole sequences). Returns the new lengths."""
    B, H, N, D = k.shape
    cur = np.asarray(cur, np.int64)
    n_new = np.asarray(n_new, np.int64)
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
    return cur + n_new


def cache_to_numpy(cache):
    return {n: t.cpu().numpy() for n, t in cache.views().items()}


def decode(cache, q, lens, sm_scale=1 / math.sqrt(128), flags=0):
    B, Hq, D = q.shape
    ws = okvq.decode_workspace(cache.dims, int(max(lens)))
    out = torch.full((B, Hq, D), float("nan"), dtype=torch.float32, device="cuda")
    okvq.okvq_decode_attention(cache, list(lens), f16dev(q), sm_scale, out, ws, flags=flags)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def load_cache(cache, arrays, lens):
    """Copy numpy cache arrays (oracle layout) into a KVCache's device buffers."""
    views = cache.views()
    meta = ("k_mx",) if "k_mx" in views else ("k_min", "k_step") if "k_min" in views else ()
    for name in ("k_codes", "v_codes", "k_norm", "v_norm", "modality") + meta:
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


def band_compare(gpu_vcodes, v16, modality, rot, length):
    """MFMA-mode value codes equal the exact order except where y is within the band of a threshold.

    Returns (codes that differ, codes in the band)."""
    from oracle.layout import unpack_values
    from oracle.values import quantize_values_fmt, rotation_error_bound
    ref = quantize_values_fmt(v16, modality, rot, length)
    got = unpack_values(gpu_vcodes)[:length]
    eps = rotation_error_bound(v16[:length], modality[:length], rot)
    dist = np.abs(ref["y"][:, :, None].astype(np.float64) - ref["thr"][:, None, :].astype(np.float64)).min(-1)
    in_band = dist <= eps
    diff = got != ref["codes"]
    assert not np.any(diff & ~in_band), f"{int((diff & ~in_band).sum())} codes differ outside the band"
    assert np.all(np.abs(got.astype(int) - ref["codes"].astype(int)) <= 1)
    return int(diff.sum()), int(in_band.sum())


def check_window(arrays, k16, v16, modality, signs, rot, b, h, w, length):
    """One 32-token window of a GPU-written cache against the oracle: key fields bit-exact, value
    norms bit-exact, value codes by the band rule, padded slots zero. ``length`` is the sequence
    length; k16 / v16 / modality are the sequence's full inputs."""
    from oracle.keys import quantize_keys_fmt, quantize_keys_mx_fmt
    from oracle.layout import pack_keys, pack_mx_meta, unpack_values
    from oracle.values import quantize_values_fmt
    a = 32 * w
    n = min(32, length - a)
    assert n > 0
    if "k_mx" in arrays:
        kq = quantize_keys_mx_fmt(k16[a:a + n], n, signs)
        np.testing.assert_array_equal(arrays["k_mx"][b, h, w],
                                      pack_mx_meta(kq["m_codes"], kq["s_codes"], kq["m_scale"], kq["s_scale"])[0])
    else:
        kq = quantize_keys_fmt(k16[a:a + n], n, signs)
        np.testing.assert_array_equal(arrays["k_min"][b, h, w].view(np.uint16), kq["m16"][0].view(np.uint16))
        np.testing.assert_array_equal(arrays["k_step"][b, h, w].view(np.uint16), kq["step16"][0].view(np.uint16))
    np.testing.assert_array_equal(arrays["k_norm"][b, h, a:a + n].view(np.uint16), kq["n16"][:n].view(np.uint16))
    np.testing.assert_array_equal(arrays["k_codes"][b, h, a:a + n], pack_keys(kq["codes"][:n]))
    vq = quantize_values_fmt(v16[a:a + n], modality[a:a + n], rot, n)
    np.testing.assert_array_equal(arrays["v_norm"][b, h, a:a + n].view(np.uint16), vq["n16"].view(np.uint16))
    band_compare(arrays["v_codes"][b, h, w:w + 1], v16[a:a + n], modality[a:a + n], rot, n)
    np.testing.assert_array_equal(arrays["modality"][b, a:a + n], modality[a:a + n])
    if n < 32:
        assert not np.any(arrays["k_codes"][b, h, a + n:a + 32])
        assert not np.any(unpack_values(arrays["v_codes"][b, h, w:w + 1])[n:])


def band_compare_bits(gpu_vcodes, v16, modality, rot, length, bits):
    """b-bit MFMA-mode value codes (one (sequence, head) of the ladder layout, [cap][16 b] bytes)
    equal the exact order except where y is within the band of a threshold, and never by more than
    one level. Returns (codes that differ, codes in the band)."""
    from oracle.ladder import quantize_values_bits_fmt, unpack_bits
    from oracle.values import rotation_error_bound
    ref = quantize_values_bits_fmt(v16, modality, rot, length, bits)
    got = unpack_bits(np.asarray(gpu_vcodes)[:length], bits)
    eps = rotation_error_bound(v16[:length], modality[:length], rot)
    dist = np.abs(ref["y"][:, :, None].astype(np.float64) - ref["thr"][:, None, :].astype(np.float64)).min(-1)
    in_band = dist <= eps
    diff = got != ref["codes"]
    assert not np.any(diff & ~in_band), f"{int((diff & ~in_band).sum())} codes differ outside the band"
    assert np.all(np.abs(got.astype(int) - ref["codes"].astype(int)) <= 1)
    return int(diff.sum()), int(in_band.sum())


def ladder_cache(k, v, modality, lens, signs, rot, capacity, num_q_heads, key_bits, value_bits, key_meta="fp16",
                 value_flags=None):
    """A bit-width-ladder cache filled by the stateless codec calls (keys, values), with the
    modality map and the device lengths copied in. Values take the exact order unless
    ``value_flags`` says otherwise (0: the matrix-core mode)."""
    B, H, N, D = k.shape
    cache = okvq.KVCache(B, H, num_q_heads, capacity, torch.from_numpy(np.ascontiguousarray(signs)),
                         torch.from_numpy(np.ascontiguousarray(rot, np.float32)), key_meta=key_meta,
                         key_bits=key_bits, value_bits=value_bits)
    vw = cache.views()
    kd, vd = f16dev(k), f16dev(v)
    md = dev(np.ascontiguousarray(modality, np.uint8))
    if key_meta == "fp16":
        okvq.okvq_quantize_keys(cache.dims, kd, N, list(lens), cache.key_signs, vw["k_codes"], vw["k_min"],
                                vw["k_step"], vw["k_norm"])
    else:
        okvq.okvq_quantize_keys_tq(cache.dims, kd, N, list(lens), cache.key_signs, vw["k_codes"], vw["k_norm"])
    flags = okvq.okvq.OKVQ_VALUE_EXACT if value_flags is None else value_flags
    okvq.okvq_quantize_values(cache.dims, vd, md, N, list(lens), cache.v_rot, flags, vw["v_codes"], vw["v_norm"])
    mod = np.zeros((B, capacity), np.uint8)
    for b in range(B):
        mod[b, :lens[b]] = modality[b, :lens[b]]
    vw["modality"].copy_(dev(mod))
    vw["seq_lens"].copy_(torch.tensor(list(lens), dtype=torch.int32))
    torch.cuda.synchronize()
    return cache
