"""Seeded inputs that stress the softmax of decode attention (inputs only, no method arithmetic).

The workload generators make attention nearly one-hot (drifting keys), which hides how small
softmax weights are carried. These layouts expose it:

* ``dominant_layer`` -- a flat background of small keys and, once per ``period`` tokens, one
  dominant key along the query direction. Query head j is the same direction scaled by
  ``scales[j]``, so the score gap between the dominant tokens and the background grows from head
  to head (about 16 log2 units per unit of scale before quantization). The background values
  lie along one channel and the dominant ones along another (plus noise), so weights that are
  dropped or rounded the same way add up instead of cancelling, in one output channel.
* ``growing_layer`` -- keys of one direction whose norm grows along the sequence: the scores rise
  (or fall, for heads with a negated query) by tens of log2 units, so every running maximum keeps
  moving.
* ``norm_ramp_layer`` -- value norms that grow geometrically along the sequence (from about 1e-3
  to about 6e4, the fp16 maximum), with drifting keys: the largest value norm seen keeps growing.

Every array is fp16 (keys, values, queries), uint8 (modality), fp32 (rotations) or int8 (signs),
drawn from numpy PCG64 generators keyed by ``SeedSequence([0x5745, kind, seed, stream])``.
"""

from __future__ import annotations

import numpy as np

from .workloads import HEAD_DIM, MOD_AUDIO, MOD_TEXT, MOD_VIDEO, modality_layout

_KIND_DOMINANT, _KIND_GROWING, _KIND_RAMP = 1, 2, 3


def _rng(kind: int, seed: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([0x5745, kind, seed, stream])))


def _unit(x: np.ndarray) -> np.ndarray:
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _rotations(kind: int, seed: int) -> np.ndarray:
    g = _rng(kind, seed, 90)
    rots = []
    for _ in range(3):
        q, r = np.linalg.qr(g.standard_normal((HEAD_DIM, HEAD_DIM)))
        rots.append(q * np.sign(np.diag(r))[None, :])
    return np.stack(rots).astype(np.float32)


def _signs(kind: int, seed: int) -> np.ndarray:
    return np.where(_rng(kind, seed, 91).integers(0, 2, HEAD_DIM) == 1, 1, -1).astype(np.int8)


def _modality(n: int) -> np.ndarray:
    """Audio-visual chunks (150 video, 25 audio tokens) and a text tail of 256 tokens."""
    return modality_layout(n, 150, 25, min(256, n))


def dominant_layer(n_tokens: int, num_kv_heads: int, group: int, scales, period: int = 512,
                   background: float = 0.05, seed: int = 0):
    """Dict k, v [1][H][n][128] fp16, q [1][H G][128] fp16, modality [1][n], lens, rot, signs,
    dominant (positions of the dominant tokens)."""
    scales = np.asarray(scales, np.float64)
    assert scales.shape == (group,)
    H, n, d = num_kv_heads, int(n_tokens), HEAD_DIM
    u = _unit(_rng(_KIND_DOMINANT, seed, 1).standard_normal((H, d)))
    k = background * _rng(_KIND_DOMINANT, seed, 2).standard_normal((H, n, d))
    offs = _rng(_KIND_DOMINANT, seed, 3).integers(0, period, -(-n // period))
    pos = np.arange(0, n, period)[:len(offs)] + offs
    pos = pos[pos < n]
    k[:, pos, :] = np.sqrt(d) * u[:, None, :]
    # background values along one channel, dominant values along another: a bias in the weight of
    # either group shows up in full in one output channel
    ch = _rng(_KIND_DOMINANT, seed, 4).choice(d, size=2, replace=False)
    w_bg = np.zeros((H, d))
    w_bg[:, ch[0]] = 1.0
    w_dom = np.zeros((H, d))
    w_dom[:, ch[1]] = 1.0
    v = 4.0 * w_bg[:, None, :] + 0.05 * _rng(_KIND_DOMINANT, seed, 6).standard_normal((H, n, d))
    v[:, pos, :] = 4.0 * w_dom[:, None, :] + 0.05 * _rng(_KIND_DOMINANT, seed, 7).standard_normal((H, len(pos), d))
    q = np.sqrt(d) * scales[None, :, None] * u[:, None, :]          # [H][G][d]
    return dict(k=k[None].astype(np.float16), v=v[None].astype(np.float16),
                q=q.reshape(1, H * group, d).astype(np.float16), modality=_modality(n)[None],
                lens=np.array([n], np.int32), rot=_rotations(_KIND_DOMINANT, seed),
                signs=_signs(_KIND_DOMINANT, seed), dominant=pos)


def growing_layer(n_tokens: int, num_kv_heads: int, group: int, rise: float = 6.0, seed: int = 0):
    """Keys k_i = rise (i / n) sqrt(128) u (one direction u per head) plus small noise; query head j
    is +-u sqrt(128) (odd heads negated: their scores fall along the sequence). Values N(0, 1)."""
    H, n, d = num_kv_heads, int(n_tokens), HEAD_DIM
    u = _unit(_rng(_KIND_GROWING, seed, 1).standard_normal((H, d)))
    t = np.arange(n, dtype=np.float64) / max(n, 1)
    k = rise * np.sqrt(d) * t[None, :, None] * u[:, None, :]
    k += 0.02 * _rng(_KIND_GROWING, seed, 2).standard_normal((H, n, d))
    v = _rng(_KIND_GROWING, seed, 3).standard_normal((H, n, d))
    sign = np.where(np.arange(group) % 2 == 0, 1.0, -1.0)
    q = np.sqrt(d) * sign[None, :, None] * u[:, None, :]
    return dict(k=k[None].astype(np.float16), v=v[None].astype(np.float16),
                q=q.reshape(1, H * group, d).astype(np.float16), modality=_modality(n)[None],
                lens=np.array([n], np.int32), rot=_rotations(_KIND_GROWING, seed), signs=_signs(_KIND_GROWING, seed))


def norm_ramp_layer(n_tokens: int, num_kv_heads: int, group: int, seed: int = 0):
    """Keys N(0, 1) (queries N(0, 1) / 4: a soft attention); values random directions whose norms
    grow geometrically from 1e-3 to 6e4 along the sequence."""
    H, n, d = num_kv_heads, int(n_tokens), HEAD_DIM
    k = _rng(_KIND_RAMP, seed, 1).standard_normal((H, n, d))
    dirs = _unit(_rng(_KIND_RAMP, seed, 2).standard_normal((H, n, d)))
    norms = np.exp(np.linspace(np.log(1e-3), np.log(6.0e4), n))
    v = dirs * norms[None, :, None]
    q = 0.25 * _rng(_KIND_RAMP, seed, 3).standard_normal((1, H * group, d))
    return dict(k=k[None].astype(np.float16), v=v[None].astype(np.float16), q=q.astype(np.float16),
                modality=_modality(n)[None], lens=np.array([n], np.int32), rot=_rotations(_KIND_RAMP, seed),
                signs=_signs(_KIND_RAMP, seed))


__all__ = ["dominant_layer", "growing_layer", "norm_ramp_layer", "MOD_AUDIO", "MOD_VIDEO", "MOD_TEXT"]
