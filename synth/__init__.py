"""Seeded synthetic inputs for the 2-bit KV-cache hot path.

This package produces *inputs only*: fp16 keys, values and queries, modality
maps, random orthogonal value rotations, Rademacher sign vectors and sequence
lengths. It holds none of the method's arithmetic (no Hadamard transform, no
codebook, no quantizer, no attention), so both the CPU oracle and the GPU path
can draw from it without sharing any computation.
"""

from .workloads import (  # noqa: F401
    MOD_AUDIO, MOD_VIDEO, MOD_TEXT, S_SIGN,
    Workload, WORKLOADS, workload, modality_layout, rng_for,
    gen_keys, gen_values, gen_queries, gen_rotations, gen_signs, gen_lengths, value_bases,
    gen_calibration_queries,
    gen_layer, gen_stream_layer, stream_chunk_modalities,
)
