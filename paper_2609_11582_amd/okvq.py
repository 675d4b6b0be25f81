"""ctypes binding of libokvq.so (include/okvq.h): argument marshalling only.

Every function here forwards to the C ABI function of the same name. Tensors are passed as
device pointers (``data_ptr()``), host integer arrays as ctypes arrays, and the stream is
torch's current HIP stream unless one is given. PyTorch provides device memory and streams;
every step of the computation runs in the library's HIP kernels. There is no fallback: if the
library is missing, importing the binding fails loudly.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libokvq.so")

OKVQ_OK = 0
OKVQ_VALUE_EXACT = 1
OKVQ_GLOBAL_ROTATION = 2  # R_0 rotates the values of every modality (the single global rotation)
OKVQ_KEY_META_FP16 = 0
OKVQ_KEY_META_MXFP4 = 1
OKVQ_KEY_META_TURBOQUANT = 2
KEY_META = {"fp16": OKVQ_KEY_META_FP16, "mxfp4": OKVQ_KEY_META_MXFP4, "turboquant": OKVQ_KEY_META_TURBOQUANT}
ROTATION_TABLE_BYTES = 294912  # OKVQ_ROTATION_TABLE_BYTES
MX_RECORD_BYTES = 136  # one MXFP4 key-metadata record per 32-token window
RESIDUAL_TOKENS = 128  # OKVQ_RESIDUAL_TOKENS: fp16 window of the captioning protocol
NOALLOC_SCRATCH_BYTES = 4 << 20  # OKVQ_NOALLOC_SCRATCH_BYTES: split records of the allocation-free decode
# buffer ids 0..11 of okvq_buffer_bytes (OKVQ_BUF_*)
BUFFERS = ("k_codes", "v_codes", "k_norm", "v_norm", "k_min", "k_step", "modality", "k_stage", "seq_lens", "k_mx",
           "k_res", "v_res")


class OkvqError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_string(status)} ({status})")
        self.status = status


class Dims(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("window", ctypes.c_int32), ("capacity", ctypes.c_int32),
                ("key_meta", ctypes.c_int32), ("residual", ctypes.c_int32), ("key_bits", ctypes.c_int32),
                ("value_bits", ctypes.c_int32)]


class CacheStruct(ctypes.Structure):
    _fields_ = [("dims", Dims)] + [(n, ctypes.c_void_p) for n in BUFFERS[:9]] + [
        ("key_signs", ctypes.c_void_p), ("v_rot", ctypes.c_void_p), ("v_rot16", ctypes.c_void_p),
        ("k_mx", ctypes.c_void_p), ("k_res", ctypes.c_void_p), ("v_res", ctypes.c_void_p)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, u32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_size_t
        P = ctypes.POINTER
        L.okvq_version.restype = i32
        L.okvq_status_string.restype = ctypes.c_char_p
        L.okvq_status_string.argtypes = [i32]
        L.okvq_buffer_bytes.restype = sz
        L.okvq_buffer_bytes.argtypes = [P(Dims), i32]
        L.okvq_codebook.restype = i32
        L.okvq_codebook.argtypes = [P(ctypes.c_float), P(ctypes.c_float)]
        L.okvq_codebook_bits.restype = i32
        L.okvq_codebook_bits.argtypes = [i32, P(ctypes.c_float), P(ctypes.c_float)]
        L.okvq_quantize_keys.restype = i32
        L.okvq_quantize_keys.argtypes = [P(Dims), vp, i32, P(i32), vp, vp, vp, vp, vp, vp]
        L.okvq_quantize_keys_mx.restype = i32
        L.okvq_quantize_keys_mx.argtypes = [P(Dims), vp, i32, P(i32), vp, vp, vp, vp, vp]
        L.okvq_quantize_keys_tq.restype = i32
        L.okvq_quantize_keys_tq.argtypes = [P(Dims), vp, i32, P(i32), vp, vp, vp, vp]
        L.okvq_quantize_values.restype = i32
        L.okvq_quantize_values.argtypes = [P(Dims), vp, vp, i32, P(i32), vp, u32, vp, vp, vp]
        L.okvq_append.restype = i32
        L.okvq_append.argtypes = [P(CacheStruct), P(i32), vp, vp, vp, P(i32), vp, i32, u32, vp]
        L.okvq_append_timed.restype = i32
        L.okvq_append_timed.argtypes = [P(CacheStruct), P(i32), vp, vp, vp, P(i32), vp, i32, u32, vp, P(vp)]
        L.okvq_cache_status.restype = i32
        L.okvq_cache_status.argtypes = [P(CacheStruct), P(i32), vp]
        L.okvq_prepare_rotation.restype = i32
        L.okvq_prepare_rotation.argtypes = [vp, vp, vp]
        L.okvq_decode_workspace_bytes.restype = sz
        L.okvq_decode_workspace_bytes.argtypes = [P(Dims), i32]
        L.okvq_decode_attention.restype = i32
        L.okvq_decode_attention.argtypes = [P(CacheStruct), P(i32), vp, ctypes.c_float, u32, vp, vp, sz, vp]
        L.okvq_decode_attention_noalloc.restype = i32
        L.okvq_decode_attention_noalloc.argtypes = [P(CacheStruct), P(i32), vp, ctypes.c_float, u32, vp, vp]
        L.okvq_decode_attention_timed.restype = i32
        L.okvq_decode_attention_timed.argtypes = [P(CacheStruct), P(i32), vp, ctypes.c_float, u32, vp, vp, sz, vp,
                                                  P(vp)]
        L.okvq_calibration_workspace_bytes.restype = sz
        L.okvq_calibration_workspace_bytes.argtypes = [P(Dims), i32]
        L.okvq_calibration_weights.restype = i32
        L.okvq_calibration_weights.argtypes = [P(Dims), vp, vp, i32, P(i32), ctypes.c_float, vp, vp, sz, vp]
        L.okvq_value_covariance.restype = i32
        L.okvq_value_covariance.argtypes = [P(Dims), vp, vp, vp, i32, P(i32), vp, vp, sz, vp]
        L.okvq_rotation_from_covariance.restype = i32
        L.okvq_rotation_from_covariance.argtypes = [vp, vp, vp, vp]
        L.okvq_dense_workspace_bytes.restype = sz
        L.okvq_dense_workspace_bytes.argtypes = [P(Dims), i32]
        L.okvq_decode_attention_dense.restype = i32
        L.okvq_decode_attention_dense.argtypes = [P(Dims), vp, vp, vp, P(i32), vp, ctypes.c_float, vp, vp, sz, vp,
                                                  P(vp)]
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().okvq_status_string(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != OKVQ_OK:
        raise OkvqError(status, where)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _need(t: torch.Tensor, nbytes: int, name: str) -> None:
    """The library trusts buffer sizes; check them here so that no kernel reads past a tensor."""
    if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous device tensor")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name}: {have} bytes, at least {nbytes} needed")


def _need_len(xs, n: int, name: str) -> None:
    if len(xs) != n:
        raise ValueError(f"{name}: {len(xs)} entries, expected {n}")


def _i32(xs: Sequence[int]):
    return (ctypes.c_int32 * len(xs))(*[int(x) for x in xs])


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def make_dims(batch, num_kv_heads, num_q_heads, capacity, head_dim=128, window=32, key_meta="fp16",
              residual=0, key_bits=0, value_bits=0) -> Dims:
    """key_bits = value_bits = 0: the 2-bit layout; 2..4 each: the bit-width ladder layout."""
    return Dims(batch, num_kv_heads, num_q_heads, head_dim, window, capacity, KEY_META[key_meta], int(residual),
                int(key_bits), int(value_bits))


def okvq_version() -> int:
    return lib().okvq_version()


def okvq_buffer_bytes(dims: Dims, which: int) -> int:
    return lib().okvq_buffer_bytes(ctypes.byref(dims), which)


def okvq_codebook():
    lv = (ctypes.c_float * 4)()
    th = (ctypes.c_float * 3)()
    _check(lib().okvq_codebook(lv, th), "okvq_codebook")
    return list(lv), list(th)


def okvq_codebook_bits(bits: int):
    """(levels [2^b], thresholds [2^b - 1]) of the b-bit codebook."""
    n = 1 << int(bits)
    lv = (ctypes.c_float * 16)()
    th = (ctypes.c_float * 15)()
    _check(lib().okvq_codebook_bits(int(bits), lv, th), "okvq_codebook_bits")
    return list(lv)[:n], list(th)[:n - 1]


def okvq_quantize_keys(dims, k, n_tokens, lens, key_signs, k_codes, k_min, k_step, k_norm, stream=None,
                       check=True) -> int:
    B, H = dims.batch, dims.num_kv_heads
    _need_len(lens, B, "lens")
    _need(k, B * H * int(n_tokens) * 128 * 2, "k")
    _need(key_signs, 128, "key_signs")
    for i, (name, t) in {0: ("k_codes", k_codes), 2: ("k_norm", k_norm), 4: ("k_min", k_min),
                         5: ("k_step", k_step)}.items():
        _need(t, okvq_buffer_bytes(dims, i), name)
    st = lib().okvq_quantize_keys(ctypes.byref(dims), _ptr(k), int(n_tokens), _i32(lens), _ptr(key_signs),
                                  _ptr(k_codes), _ptr(k_min), _ptr(k_step), _ptr(k_norm), _stream(stream))
    if check:
        _check(st, "okvq_quantize_keys")
    return st


def okvq_quantize_keys_mx(dims, k, n_tokens, lens, key_signs, k_codes, k_mx, k_norm, stream=None,
                          check=True) -> int:
    B, H = dims.batch, dims.num_kv_heads
    _need_len(lens, B, "lens")
    _need(k, B * H * int(n_tokens) * 128 * 2, "k")
    _need(key_signs, 128, "key_signs")
    for i, (name, t) in {0: ("k_codes", k_codes), 2: ("k_norm", k_norm), 9: ("k_mx", k_mx)}.items():
        _need(t, okvq_buffer_bytes(dims, i), name)
    st = lib().okvq_quantize_keys_mx(ctypes.byref(dims), _ptr(k), int(n_tokens), _i32(lens), _ptr(key_signs),
                                     _ptr(k_codes), _ptr(k_mx), _ptr(k_norm), _stream(stream))
    if check:
        _check(st, "okvq_quantize_keys_mx")
    return st


def okvq_quantize_keys_tq(dims, k, n_tokens, lens, key_signs, k_codes, k_norm, stream=None, check=True) -> int:
    B, H = dims.batch, dims.num_kv_heads
    _need_len(lens, B, "lens")
    _need(k, B * H * int(n_tokens) * 128 * 2, "k")
    _need(key_signs, 128, "key_signs")
    for i, (name, t) in {0: ("k_codes", k_codes), 2: ("k_norm", k_norm)}.items():
        _need(t, okvq_buffer_bytes(dims, i), name)
    st = lib().okvq_quantize_keys_tq(ctypes.byref(dims), _ptr(k), int(n_tokens), _i32(lens), _ptr(key_signs),
                                     _ptr(k_codes), _ptr(k_norm), _stream(stream))
    if check:
        _check(st, "okvq_quantize_keys_tq")
    return st


def okvq_quantize_values(dims, v, modality, n_tokens, lens, v_rot, flags, v_codes, v_norm, stream=None,
                         check=True) -> int:
    B, H = dims.batch, dims.num_kv_heads
    _need_len(lens, B, "lens")
    _need(v, B * H * int(n_tokens) * 128 * 2, "v")
    _need(modality, B * int(n_tokens), "modality")
    _need(v_rot, 3 * 128 * 128 * 4, "v_rot")
    _need(v_codes, okvq_buffer_bytes(dims, 1), "v_codes")
    _need(v_norm, okvq_buffer_bytes(dims, 3), "v_norm")
    st = lib().okvq_quantize_values(ctypes.byref(dims), _ptr(v), _ptr(modality), int(n_tokens), _i32(lens),
                                    _ptr(v_rot), int(flags), _ptr(v_codes), _ptr(v_norm), _stream(stream))
    if check:
        _check(st, "okvq_quantize_values")
    return st


def okvq_append(cache: "KVCache", lens, k_new, v_new, mod_new, n_new, n_new_dev, n_max, flags=0, stream=None,
                check=True) -> int:
    B, H = cache.dims.batch, cache.dims.num_kv_heads
    _need_len(lens, B, "lens")
    _need_len(n_new, B, "n_new")
    _need(k_new, B * H * int(n_max) * 128 * 2, "k_new")
    _need(v_new, B * H * int(n_max) * 128 * 2, "v_new")
    _need(mod_new, B * int(n_max), "mod_new")
    _need(n_new_dev, B * 4, "n_new_dev")
    st = lib().okvq_append(ctypes.byref(cache.struct), _i32(lens), _ptr(k_new), _ptr(v_new), _ptr(mod_new),
                           _i32(n_new), _ptr(n_new_dev), int(n_max), int(flags), _stream(stream))
    if check:
        _check(st, "okvq_append")
    return st


def okvq_append_timed(cache: "KVCache", lens, k_new, v_new, mod_new, n_new, n_new_dev, n_max, events, flags=0,
                      stream=None, check=True) -> int:
    """okvq_append that records two torch.cuda.Event objects at the start and end of its codec
    launch (the window-parallel launch, or the fused codec launch)."""
    B, H = cache.dims.batch, cache.dims.num_kv_heads
    _need_len(lens, B, "lens")
    _need_len(n_new, B, "n_new")
    _need(k_new, B * H * int(n_max) * 128 * 2, "k_new")
    _need(v_new, B * H * int(n_max) * 128 * 2, "v_new")
    _need(mod_new, B * int(n_max), "mod_new")
    _need(n_new_dev, B * 4, "n_new_dev")
    _need_len(events, 2, "events")
    handles = (ctypes.c_void_p * 2)(*[ctypes.c_void_p(e.cuda_event) for e in events])
    if not all(handles):
        raise ValueError("events: record each torch.cuda.Event once before passing it (torch creates them lazily)")
    st = lib().okvq_append_timed(ctypes.byref(cache.struct), _i32(lens), _ptr(k_new), _ptr(v_new), _ptr(mod_new),
                                 _i32(n_new), _ptr(n_new_dev), int(n_max), int(flags), _stream(stream), handles)
    if check:
        _check(st, "okvq_append_timed")
    return st


def okvq_cache_status(cache: "KVCache", stream=None) -> int:
    """The cache's status word (seq_lens[B + 1]): 0, or 1 once an append's value codec gave up
    waiting for its partner waves (that append's value codes may be wrong). Synchronizes `stream`."""
    word = ctypes.c_int32(-1)
    _check(lib().okvq_cache_status(ctypes.byref(cache.struct), ctypes.byref(word), _stream(stream)),
           "okvq_cache_status")
    return int(word.value)


def okvq_prepare_rotation(v_rot, v_rot16, stream=None, check=True) -> int:
    _need(v_rot, 3 * 128 * 128 * 4, "v_rot")
    _need(v_rot16, ROTATION_TABLE_BYTES, "v_rot16")
    st = lib().okvq_prepare_rotation(_ptr(v_rot), _ptr(v_rot16), _stream(stream))
    if check:
        _check(st, "okvq_prepare_rotation")
    return st


def okvq_decode_workspace_bytes(dims: Dims, max_seq_len: int) -> int:
    return lib().okvq_decode_workspace_bytes(ctypes.byref(dims), int(max_seq_len))


def decode_workspace(dims: Dims, max_seq_len: int, device="cuda") -> torch.Tensor:
    """A decode workspace of okvq_decode_workspace_bytes bytes (zero-filled, though no contents are needed)."""
    nbytes = max(okvq_decode_workspace_bytes(dims, max_seq_len), 16)
    return torch.zeros((nbytes + 15) // 16 * 4, dtype=torch.float32, device=device)


def okvq_decode_attention(cache: "KVCache", lens, q, sm_scale, out, workspace, workspace_bytes=None, flags=0,
                          stream=None, check=True) -> int:
    B, Hq = cache.dims.batch, cache.dims.num_q_heads
    _need_len(lens, B, "lens")
    _need(q, B * Hq * 128 * 2, "q")
    _need(out, B * Hq * 128 * 4, "out")
    have = workspace.numel() * workspace.element_size()
    nbytes = have if workspace_bytes is None else min(int(workspace_bytes), have)
    st = lib().okvq_decode_attention(ctypes.byref(cache.struct), _i32(lens), _ptr(q), float(sm_scale), int(flags),
                                     _ptr(out), _ptr(workspace), int(nbytes), _stream(stream))
    if check:
        _check(st, "okvq_decode_attention")
    return st


def okvq_decode_attention_noalloc(cache: "KVCache", lens, q, sm_scale, out, flags=0, stream=None, check=True) -> int:
    """okvq_decode_attention with the split records in the library's static per-GPU array
    (NOALLOC_SCRATCH_BYTES): no workspace argument, no allocation in the call."""
    B, Hq = cache.dims.batch, cache.dims.num_q_heads
    _need_len(lens, B, "lens")
    _need(q, B * Hq * 128 * 2, "q")
    _need(out, B * Hq * 128 * 4, "out")
    st = lib().okvq_decode_attention_noalloc(ctypes.byref(cache.struct), _i32(lens), _ptr(q), float(sm_scale),
                                             int(flags), _ptr(out), _stream(stream))
    if check:
        _check(st, "okvq_decode_attention_noalloc")
    return st


def okvq_decode_attention_timed(cache: "KVCache", lens, q, sm_scale, out, workspace, events, workspace_bytes=None,
                                flags=0, stream=None, check=True) -> int:
    """okvq_decode_attention that records four torch.cuda.Event objects at the start and end of
    its split-K kernel and of its merge kernel."""
    B, Hq = cache.dims.batch, cache.dims.num_q_heads
    _need_len(lens, B, "lens")
    _need(q, B * Hq * 128 * 2, "q")
    _need(out, B * Hq * 128 * 4, "out")
    _need_len(events, 4, "events")
    handles = (ctypes.c_void_p * 4)(*[ctypes.c_void_p(e.cuda_event) for e in events])
    if not all(handles):
        raise ValueError("events: record each torch.cuda.Event once before passing it (torch creates them lazily)")
    have = workspace.numel() * workspace.element_size()
    nbytes = have if workspace_bytes is None else min(int(workspace_bytes), have)
    st = lib().okvq_decode_attention_timed(ctypes.byref(cache.struct), _i32(lens), _ptr(q), float(sm_scale), int(flags),
                                           _ptr(out), _ptr(workspace), int(nbytes), _stream(stream), handles)
    if check:
        _check(st, "okvq_decode_attention_timed")
    return st


def okvq_dense_workspace_bytes(dims: Dims, max_seq_len: int) -> int:
    return lib().okvq_dense_workspace_bytes(ctypes.byref(dims), int(max_seq_len))


def dense_workspace(dims: Dims, max_seq_len: int, device="cuda") -> torch.Tensor:
    """A workspace of okvq_dense_workspace_bytes bytes for the dense decode (no contents needed)."""
    nbytes = max(okvq_dense_workspace_bytes(dims, max_seq_len), 16)
    return torch.empty((nbytes + 15) // 16 * 4, dtype=torch.float32, device=device)


def okvq_decode_attention_dense(dims: Dims, k, v, seq_lens, lens, q, sm_scale, out, workspace, events=None,
                                workspace_bytes=None, stream=None, check=True) -> int:
    """Dense fp16 decode attention over k, v [B][H][capacity][128] (the comparison baseline);
    events: None, or four torch.cuda.Event objects (split-K start, end; merge start, end)."""
    B, H, Hq, cap = dims.batch, dims.num_kv_heads, dims.num_q_heads, dims.capacity
    _need_len(lens, B, "lens")
    _need(k, B * H * cap * 128 * 2, "k")
    _need(v, B * H * cap * 128 * 2, "v")
    _need(seq_lens, B * 4, "seq_lens")
    _need(q, B * Hq * 128 * 2, "q")
    _need(out, B * Hq * 128 * 4, "out")
    handles = None
    if events is not None:
        _need_len(events, 4, "events")
        handles = (ctypes.c_void_p * 4)(*[ctypes.c_void_p(e.cuda_event) for e in events])
        if not all(handles):
            raise ValueError("events: record each torch.cuda.Event once before passing it (torch creates them lazily)")
    have = workspace.numel() * workspace.element_size()
    nbytes = have if workspace_bytes is None else min(int(workspace_bytes), have)
    st = lib().okvq_decode_attention_dense(ctypes.byref(dims), _ptr(k), _ptr(v), _ptr(seq_lens), _i32(lens), _ptr(q),
                                           float(sm_scale), _ptr(out), _ptr(workspace), int(nbytes), _stream(stream),
                                           handles)
    if check:
        _check(st, "okvq_decode_attention_dense")
    return st


def okvq_calibration_workspace_bytes(dims: Dims, n_tokens: int) -> int:
    return lib().okvq_calibration_workspace_bytes(ctypes.byref(dims), int(n_tokens))


def calibration_workspace(dims: Dims, n_tokens: int, device="cuda") -> torch.Tensor:
    """A calibration workspace of okvq_calibration_workspace_bytes bytes (no contents needed)."""
    nbytes = max(okvq_calibration_workspace_bytes(dims, n_tokens), 16)
    return torch.empty((nbytes + 15) // 16 * 4, dtype=torch.float32, device=device)


def okvq_calibration_weights(dims, q, k, n_tokens, lens, sm_scale, w, workspace, stream=None, check=True) -> int:
    B, H, Hq = dims.batch, dims.num_kv_heads, dims.num_q_heads
    _need_len(lens, B, "lens")
    _need(q, B * Hq * int(n_tokens) * 128 * 2, "q")
    _need(k, B * H * int(n_tokens) * 128 * 2, "k")
    _need(w, B * H * int(n_tokens) * 4, "w")
    have = workspace.numel() * workspace.element_size()
    st = lib().okvq_calibration_weights(ctypes.byref(dims), _ptr(q), _ptr(k), int(n_tokens), _i32(lens),
                                        float(sm_scale), _ptr(w), _ptr(workspace), int(have), _stream(stream))
    if check:
        _check(st, "okvq_calibration_weights")
    return st


def okvq_value_covariance(dims, v, modality, w, n_tokens, lens, cov, workspace, stream=None, check=True) -> int:
    B, H = dims.batch, dims.num_kv_heads
    _need_len(lens, B, "lens")
    _need(v, B * H * int(n_tokens) * 128 * 2, "v")
    _need(modality, B * int(n_tokens), "modality")
    _need(w, B * H * int(n_tokens) * 4, "w")
    _need(cov, 3 * 128 * 128 * 4, "cov")
    have = workspace.numel() * workspace.element_size()
    st = lib().okvq_value_covariance(ctypes.byref(dims), _ptr(v), _ptr(modality), _ptr(w), int(n_tokens), _i32(lens),
                                     _ptr(cov), _ptr(workspace), int(have), _stream(stream))
    if check:
        _check(st, "okvq_value_covariance")
    return st


def okvq_rotation_from_covariance(cov, signs, rot, eigenvalues=None, check=True) -> int:
    """Host call: cov float32 [3][128][128], signs int8 [128], rot float32 [3][128][128] (output),
    eigenvalues float64 [3][128] (output) or None -- C-contiguous numpy arrays."""
    import numpy as np
    for name, a, dt, n in (("cov", cov, np.float32, 3 * 128 * 128), ("signs", signs, np.int8, 128),
                           ("rot", rot, np.float32, 3 * 128 * 128)):
        if not isinstance(a, np.ndarray) or a.dtype != dt or not a.flags["C_CONTIGUOUS"] or a.size < n:
            raise ValueError(f"{name}: expected a contiguous {np.dtype(dt).name} numpy array of {n} elements")
    if eigenvalues is not None and (eigenvalues.dtype != np.float64 or not eigenvalues.flags["C_CONTIGUOUS"]
                                    or eigenvalues.size < 3 * 128):
        raise ValueError("eigenvalues: expected a contiguous float64 numpy array of 384 elements")
    st = lib().okvq_rotation_from_covariance(cov.ctypes.data, signs.ctypes.data, rot.ctypes.data,
                                             None if eigenvalues is None else eigenvalues.ctypes.data)
    if check:
        _check(st, "okvq_rotation_from_covariance")
    return st


_DTYPES = dict(k_codes=torch.uint8, v_codes=torch.uint8, k_norm=torch.float16, v_norm=torch.float16,
               k_min=torch.float16, k_step=torch.float16, modality=torch.uint8, k_stage=torch.float16,
               seq_lens=torch.int32, k_mx=torch.uint8, k_res=torch.float16, v_res=torch.float16)


class KVCache:
    """Device buffers of one layer's packed cache, sized by okvq_buffer_bytes (torch allocations),
    with the layer's key signs, value rotations and the decode's inverse-rotation table.
    key_meta "fp16" keeps the key window minimum and step in k_min / k_step, "mxfp4" in k_mx;
    "turboquant" stores TurboQuant keys (no window metadata, the paper's baseline).
    residual=RESIDUAL_TOKENS adds the fp16 rings of the captioning protocol (k_res, v_res).
    key_bits, value_bits in 2..4 select the bit-width ladder layout (token-major bit streams; filled
    by okvq_append or the stateless codec calls)."""

    def __init__(self, batch, num_kv_heads, num_q_heads, capacity, key_signs: torch.Tensor, v_rot: torch.Tensor,
                 device="cuda", key_meta="fp16", residual=0, key_bits=0, value_bits=0):
        self.key_meta = key_meta
        self.residual = int(residual)
        self.key_bits, self.value_bits = int(key_bits), int(value_bits)
        self.dims = make_dims(batch, num_kv_heads, num_q_heads, capacity, key_meta=key_meta, residual=residual,
                              key_bits=key_bits, value_bits=value_bits)
        self.key_signs = key_signs.to(device=device, dtype=torch.int8).contiguous()
        self.v_rot = v_rot.to(device=device, dtype=torch.float32).contiguous()
        self.v_rot16 = torch.empty(ROTATION_TABLE_BYTES // 2, dtype=torch.float16, device=device)
        okvq_prepare_rotation(self.v_rot, self.v_rot16)
        self.buffers = {}
        unused = {"fp16": ("k_mx",), "mxfp4": ("k_min", "k_step"), "turboquant": ("k_min", "k_step", "k_mx")}[key_meta]
        if not self.residual:
            unused += ("k_res", "v_res")
        if self.key_bits and key_meta != "fp16":  # ladder: only the method's keys keep a stage
            unused += ("k_stage",)
        for i, name in enumerate(BUFFERS):
            nbytes = okvq_buffer_bytes(self.dims, i)
            if (nbytes == 0) != (name in unused):
                raise OkvqError(-1, f"okvq_buffer_bytes({name}) = {nbytes}")
            if nbytes == 0:
                continue
            dt = _DTYPES[name]
            n = nbytes // torch.tensor([], dtype=dt).element_size()
            self.buffers[name] = torch.zeros(n, dtype=dt, device=device)
        ptr = {n: (t.data_ptr() if n in self.buffers else None) for n, t in
               ((n, self.buffers.get(n)) for n in BUFFERS)}
        self.struct = CacheStruct(self.dims, *[ptr[n] for n in BUFFERS[:9]], self.key_signs.data_ptr(),
                                  self.v_rot.data_ptr(), self.v_rot16.data_ptr(), ptr["k_mx"], ptr["k_res"],
                                  ptr["v_res"])

    def __getitem__(self, name):
        return self.buffers[name]

    def views(self):
        """The buffers reshaped to their documented layouts."""
        d = self.dims
        B, H, cap = d.batch, d.num_kv_heads, d.capacity
        b = self.buffers
        if self.key_bits:  # bit-width ladder: token-major bit streams
            v = dict(k_codes=b["k_codes"].view(B, H, cap, 16 * self.key_bits),
                     v_codes=b["v_codes"].view(B, H, cap, 16 * self.value_bits))
            if "k_stage" in b:
                v.update(k_stage=b["k_stage"].view(B, H, 32, 128))
        else:
            v = dict(k_codes=b["k_codes"].view(B, H, cap, 32), v_codes=b["v_codes"].view(B, H, cap // 32, 1024),
                     k_stage=b["k_stage"].view(B, H, 32, 128))
        v.update(k_norm=b["k_norm"].view(B, H, cap), v_norm=b["v_norm"].view(B, H, cap),
                 modality=b["modality"].view(B, cap), seq_lens=b["seq_lens"][:B])
        if self.key_meta == "fp16":
            v.update(k_min=b["k_min"].view(B, H, cap // 32, 128), k_step=b["k_step"].view(B, H, cap // 32, 128))
        elif self.key_meta == "mxfp4":
            v.update(k_mx=b["k_mx"].view(B, H, cap // 32, MX_RECORD_BYTES))
        if self.residual:
            v.update(k_res=b["k_res"].view(B, H, RESIDUAL_TOKENS, 128), v_res=b["v_res"].view(B, H, RESIDUAL_TOKENS, 128))
        return v
