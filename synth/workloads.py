"""Seeded generators for Omni-LLM-shaped KV caches (inputs only).

The paper evaluates on audio-visual benchmarks whose KV caches come from
Qwen2.5-Omni / Qwen3-Omni (Sec. 3.1). Neither the weights nor the datasets are
available, so these generators stand in for the caches those runs produce:

* token stream: per temporal chunk, video tokens then audio tokens, and a text
  prompt at the end (Sec. 2.1, the ordering [V_1, A_1, ..., V_T, A_T, L]);
* keys: N(0, 1) noise plus a per-64-token mean shift that follows a Gaussian
  random walk (std 0.5 per channel and step), with 4 outlier channels scaled
  by 8 -- the "temporal key drift" of Sec. 2.2 and the large coordinates the
  introduction describes;
* values: per modality, a distinct random rank-16 subspace plus N(0, 0.05^2)
  noise -- the "heterogeneous value geometry" of Sec. 2.2 / Fig. 2;
* value rotations: random orthogonal matrices (QR of a Gaussian) standing in
  for the calibrated R_m of Eq. 6;
* key signs: Rademacher diagonal of the randomized Hadamard transform (Eq. 2);
* queries: N(0, 1).

Every stream has its own numpy PCG64 generator keyed by
``SeedSequence([0x0C7A, workload_id, layer, stream, b, h])``.
"""

from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

MOD_AUDIO, MOD_VIDEO, MOD_TEXT = 0, 1, 2
HEAD_DIM = 128

# stream ids
S_KEY_NOISE, S_DRIFT, S_OUTLIER, S_VBASIS, S_VCOEF, S_VNOISE, S_ROT, S_SIGN, S_QUERY, S_LEN, S_CALQ = range(1, 12)


@dataclasses.dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    batch: int
    num_kv_heads: int
    num_q_heads: int
    seq_len: int              # tokens cached per sequence (the maximum when ragged)
    video_per_chunk: int
    audio_per_chunk: int
    text_tail: int
    layers: int = 1
    ragged_min: Optional[int] = None   # lengths ~ U{ragged_min..seq_len} when set
    stream_steps: int = 0              # append+decode steps after the prefill
    stream_tokens: int = 0             # tokens appended per stream step

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def capacity(self) -> int:
        cap = self.seq_len + self.stream_steps * self.stream_tokens
        return (cap + 31) // 32 * 32


WORKLOADS = {
    "tiny_1k": Workload(1, "tiny_1k", 1, 1, 4, 1024, 128, 64, 64),
    "omni7b_32k": Workload(2, "omni7b_32k", 1, 4, 28, 32768, 150, 25, 256),
    "omni7b_b16_ragged16k": Workload(3, "omni7b_b16_ragged16k", 16, 4, 28, 16384, 150, 25, 256,
                                     ragged_min=8192),
    "omni3b_b4_64k_stream": Workload(4, "omni3b_b4_64k_stream", 4, 2, 16, 65536, 144, 16, 256,
                                     stream_steps=16, stream_tokens=512),
    "omni30b_128k_48layer": Workload(5, "omni30b_128k_48layer", 1, 4, 32, 131072, 150, 25, 256,
                                     layers=48),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def rng_for(wid: int, layer: int, stream: int, b: int = 0, h: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([0x0C7A, wid, layer, stream, b, h])))


def modality_layout(n: int, video: int, audio: int, text_tail: int) -> np.ndarray:
    """[V]*video + [A]*audio repeated and cut to n - text_tail tokens, then text_tail text tokens."""
    n_av = max(n - text_tail, 0)
    chunk = np.concatenate([np.full(video, MOD_VIDEO, np.uint8), np.full(audio, MOD_AUDIO, np.uint8)])
    reps = -(-n_av // len(chunk)) if n_av else 0
    av = np.tile(chunk, reps)[:n_av]
    return np.concatenate([av, np.full(n - n_av, MOD_TEXT, np.uint8)])


def stream_chunk_modalities(wl: Workload, start_chunk_token: int, n: int) -> np.ndarray:
    """Modalities of n streamed tokens that continue the audio-visual chunk pattern.

    ``start_chunk_token`` is the position inside the repeating [V, A] pattern at
    which the streamed tokens begin (the prefill's text tail is not part of it).
    """
    chunk = np.concatenate([np.full(wl.video_per_chunk, MOD_VIDEO, np.uint8),
                            np.full(wl.audio_per_chunk, MOD_AUDIO, np.uint8)])
    idx = (start_chunk_token + np.arange(n)) % len(chunk)
    return chunk[idx]


def gen_keys(wid: int, layer: int, b: int, h: int, n: int, d: int = HEAD_DIM) -> np.ndarray:
    """fp16 keys [n][d]: N(0,1) + random-walk mean per 64 tokens (std 0.5 per step) + 4 channels x8."""
    x = rng_for(wid, layer, S_KEY_NOISE, b, h).standard_normal((n, d))
    n_drift = -(-n // 64)
    steps = 0.5 * rng_for(wid, layer, S_DRIFT, b, h).standard_normal((n_drift, d))
    if n_drift:
        steps[0] = 0.0
    mu = np.cumsum(steps, axis=0)
    k = x + np.repeat(mu, 64, axis=0)[:n]
    outl = rng_for(wid, layer, S_OUTLIER, 0, h).choice(d, size=4, replace=False)
    k[:, outl] *= 8.0
    return k.astype(np.float16)


def value_bases(wid: int, layer: int, h: int, d: int = HEAD_DIM, rank: int = 16) -> np.ndarray:
    """[3][d][rank] the random orthonormal subspace bases of the value generator (audio, video, text)."""
    g = rng_for(wid, layer, S_VBASIS, 0, h)
    return np.stack([np.linalg.qr(g.standard_normal((d, rank)))[0] for _ in (MOD_AUDIO, MOD_VIDEO, MOD_TEXT)])


def gen_values(wid: int, layer: int, b: int, h: int, modality: np.ndarray, d: int = HEAD_DIM,
               rank: int = 16, noise: float = 0.05) -> np.ndarray:
    """fp16 values [n][d]: B_m c + eps, B_m a random orthonormal d x rank basis per (layer, head, modality)."""
    n = len(modality)
    out = np.empty((n, d))
    coef = rng_for(wid, layer, S_VCOEF, b, h).standard_normal((n, rank))
    eps = noise * rng_for(wid, layer, S_VNOISE, b, h).standard_normal((n, d))
    bases = value_bases(wid, layer, h, d, rank)
    for m in (MOD_AUDIO, MOD_VIDEO, MOD_TEXT):
        sel = modality == m
        out[sel] = coef[sel] @ bases[m].T
    out += eps
    return out.astype(np.float16)


def gen_rotations(wid: int, layer: int, d: int = HEAD_DIM, count: int = 3) -> np.ndarray:
    """fp32 [count][d][d] random orthogonal matrices (QR of a Gaussian, sign-fixed), one per modality."""
    g = rng_for(wid, layer, S_ROT)
    rots = []
    for _ in range(count):
        q, r = np.linalg.qr(g.standard_normal((d, d)))
        rots.append(q * np.sign(np.diag(r))[None, :])
    return np.stack(rots).astype(np.float32)


def gen_signs(wid: int, layer: int, d: int = HEAD_DIM) -> np.ndarray:
    """int8 [d] Rademacher signs (+1 / -1)."""
    return np.where(rng_for(wid, layer, S_SIGN).integers(0, 2, d) == 1, 1, -1).astype(np.int8)


def gen_queries(wid: int, layer: int, batch: int, num_q_heads: int, d: int = HEAD_DIM,
                step: int = 0) -> np.ndarray:
    """fp16 queries [batch][num_q_heads][d] ~ N(0, 1)."""
    return rng_for(wid, layer, S_QUERY, step, 0).standard_normal((batch, num_q_heads, d)).astype(np.float16)


def gen_calibration_queries(wid: int, layer: int, batch: int, num_q_heads: int, n: int,
                            d: int = HEAD_DIM) -> np.ndarray:
    """fp16 calibration queries [batch][num_q_heads][n][d] ~ N(0, 1): one per position (the prefill
    queries whose attention weights Eq. 5 sums)."""
    return rng_for(wid, layer, S_CALQ).standard_normal((batch, num_q_heads, n, d)).astype(np.float16)


def gen_lengths(wl: Workload) -> np.ndarray:
    if wl.ragged_min is None:
        return np.full(wl.batch, wl.seq_len, np.int32)
    return rng_for(wl.wid, 0, S_LEN).integers(wl.ragged_min, wl.seq_len + 1, wl.batch).astype(np.int32)


def gen_layer(wl: Workload, layer: int = 0, lengths: Optional[np.ndarray] = None, n_tokens: Optional[int] = None):
    """All inputs of one layer: dict with k, v [B][Hkv][N][D] fp16, modality [B][N] u8, lens, q, rot, signs.

    B is len(lengths) when lengths are given, else the workload's batch. Tokens beyond a sequence's
    length are zero-filled (they are ignored by every consumer).
    """
    if lengths is None:
        lengths = gen_lengths(wl)
    n = int(n_tokens if n_tokens is not None else wl.seq_len)
    B, H = len(lengths), wl.num_kv_heads
    k = np.zeros((B, H, n, HEAD_DIM), np.float16)
    v = np.zeros((B, H, n, HEAD_DIM), np.float16)
    mod = np.zeros((B, n), np.uint8)
    for b in range(B):
        L = int(min(lengths[b], n))
        mod[b, :L] = modality_layout(L, wl.video_per_chunk, wl.audio_per_chunk, min(wl.text_tail, L))
        for h in range(H):
            k[b, h, :L] = gen_keys(wl.wid, layer, b, h, L)
            v[b, h, :L] = gen_values(wl.wid, layer, b, h, mod[b, :L])
    return dict(k=k, v=v, modality=mod, lens=np.asarray(lengths, np.int32),
                q=gen_queries(wl.wid, layer, B, wl.num_q_heads),
                rot=gen_rotations(wl.wid, layer), signs=gen_signs(wl.wid, layer))


def gen_stream_layer(wl: Workload, layer: int = 0):
    """A prefill of wl.seq_len tokens followed by wl.stream_steps chunks of wl.stream_tokens tokens.

    The prefill follows ``modality_layout`` (audio-visual chunks, then the text tail); the streamed
    tokens continue the audio-visual pattern. Keys and values cover all tokens; the key drift walk
    runs on through the streamed part. Returns the ``gen_layer`` fields plus ``prefill``.
    """
    pre = wl.seq_len
    n = pre + wl.stream_steps * wl.stream_tokens
    first = modality_layout(pre, wl.video_per_chunk, wl.audio_per_chunk, wl.text_tail)
    rest = stream_chunk_modalities(wl, max(pre - wl.text_tail, 0), n - pre)
    mod1 = np.concatenate([first, rest])
    B, H = wl.batch, wl.num_kv_heads
    k = np.zeros((B, H, n, HEAD_DIM), np.float16)
    v = np.zeros((B, H, n, HEAD_DIM), np.float16)
    for b in range(B):
        for h in range(H):
            k[b, h] = gen_keys(wl.wid, layer, b, h, n)
            v[b, h] = gen_values(wl.wid, layer, b, h, mod1)
    return dict(k=k, v=v, modality=np.tile(mod1, (B, 1)), lens=np.full(B, n, np.int32), prefill=pre,
                q=gen_queries(wl.wid, layer, B, wl.num_q_heads),
                rot=gen_rotations(wl.wid, layer), signs=gen_signs(wl.wid, layer))
