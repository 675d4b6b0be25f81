"""Device-side generation of synthetic layers (torch on the GPU), for benchmark set-ups whose host
generation would take minutes (48 layers of 131072 tokens).

Same recipe as ``synth.workloads.gen_layer`` -- keys N(0, 1) plus a random-walk mean per 64 tokens
(std 0.5 per step and channel) with 4 outlier channels scaled by 8, values B_m c + N(0, 0.05^2) on
the per-(layer, head, modality) rank-16 bases of ``value_bases``, the token stream of
``modality_layout`` -- with the Gaussian draws taken from torch's generator seeded per (workload,
layer) instead of the numpy streams (so not bitwise equal to ``gen_layer``). The bases, outlier
channels, rotations, signs and queries are the numpy ones. Inputs only: no method arithmetic.
"""

from __future__ import annotations

import numpy as np

from .workloads import (HEAD_DIM, MOD_AUDIO, MOD_TEXT, MOD_VIDEO, S_OUTLIER, Workload, gen_queries, gen_rotations,
                        gen_signs, modality_layout, rng_for, value_bases)


def _torch_seed(wid: int, layer: int) -> int:
    return int(np.random.SeedSequence([0x0C7A, wid, layer, 0xDE71]).generate_state(1)[0])


def gen_layer_device(wl: Workload, layer: int, device):
    """dict: k, v [B][Hkv][N][128] fp16 and modality [B][N] u8 as device tensors; modality_np, lens,
    rot, signs, q as numpy (every sequence has the workload's full length)."""
    import torch

    B, H, N, D = wl.batch, wl.num_kv_heads, wl.seq_len, HEAD_DIM
    g = torch.Generator(device=device).manual_seed(_torch_seed(wl.wid, layer))
    mod = modality_layout(N, wl.video_per_chunk, wl.audio_per_chunk, wl.text_tail)
    # keys
    k = torch.randn(B, H, N, D, generator=g, device=device)
    nd = -(-N // 64)
    steps = 0.5 * torch.randn(B, H, nd, D, generator=g, device=device)
    steps[:, :, 0] = 0.0
    k += steps.cumsum(2).repeat_interleave(64, dim=2)[:, :, :N]
    for h in range(H):
        outl = torch.from_numpy(rng_for(wl.wid, layer, S_OUTLIER, 0, h).choice(D, size=4, replace=False)).to(device)
        k[:, h, :, outl] *= 8.0
    k16 = k.half()
    del k, steps
    # values
    mod_dev = torch.from_numpy(mod).to(device)
    v = 0.05 * torch.randn(B, H, N, D, generator=g, device=device)
    coef = torch.randn(B, H, N, 16, generator=g, device=device)
    for h in range(H):
        bases = torch.from_numpy(value_bases(wl.wid, layer, h)).float().to(device)  # [3][D][16]
        for m in (MOD_AUDIO, MOD_VIDEO, MOD_TEXT):
            sel = mod_dev == m
            v[:, h, sel] += coef[:, h, sel] @ bases[m].T
    v16 = v.half()
    del v, coef
    return dict(k=k16, v=v16, modality=mod_dev.unsqueeze(0).repeat(B, 1).contiguous(),
                modality_np=np.tile(mod, (B, 1)), lens=np.full(B, N, np.int32),
                rot=gen_rotations(wl.wid, layer), signs=gen_signs(wl.wid, layer),
                q=gen_queries(wl.wid, layer, B, wl.num_q_heads))
