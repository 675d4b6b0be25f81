"""OmniKVQuant 2-bit KV-cache hot path for AMD MI355X (gfx950).

The computation lives in libokvq.so (hand-written HIP kernels behind the C ABI of
include/okvq.h); ``okvq`` is its ctypes binding.
"""

from . import okvq  # noqa: F401
from .okvq import (KVCache, OkvqError, calibration_workspace, decode_workspace, dense_workspace,  # noqa: F401
                   make_dims, okvq_append, okvq_append_timed, okvq_buffer_bytes, okvq_calibration_weights,
                   okvq_calibration_workspace_bytes, okvq_codebook, okvq_codebook_bits, okvq_decode_attention,
                   okvq_decode_attention_dense, okvq_decode_attention_noalloc, okvq_decode_attention_timed, okvq_decode_workspace_bytes,
                   okvq_dense_workspace_bytes, okvq_cache_status, okvq_prepare_rotation, okvq_quantize_keys,
                   okvq_quantize_keys_mx, okvq_quantize_keys_tq, okvq_quantize_values,
                   okvq_rotation_from_covariance, okvq_value_covariance, okvq_version, status_string)
