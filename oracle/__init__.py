"""CPU oracle for the OmniKVQuant 2-bit KV-cache hot path -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously correct CPU statement of what the hot
path computes, written from the paper (arXiv 2609.11582, "OmniKVQuant: KV Cache
Quantization for Omni-LLMs"). Only the test suite, the graft smoke check and
the CPU-baseline leg of the benchmark may import it; the product library never
does, and it shares no code, tables or constants with the HIP path.

Two arithmetic modes are provided:

* F64 -- the paper's mathematics in float64 (used for invariants and for the
  attention parity check);
* FMT -- a numpy-float32 emulation of the documented operation order (used
  where the GPU must be bit-exact: norms, rotated key directions, window
  minimum / step, codes). numpy float32 element-wise operations are IEEE
  binary32 with round-to-nearest-even and no contraction; sqrt and division
  are correctly rounded, ``np.rint`` rounds half to even and ``astype(float16)``
  rounds to nearest even.

Modules
-------
codebook   Lloyd-Max codebook for N(0, 1/d) (Eq. 3)
hadamard   Sylvester Hadamard matrix, randomized H, fp32 butterfly order (Eq. 2)
keys       key codec: norm split, Hadamard, per-window min/step, codes (Eq. 2, Eq. 4)
mxfp4      MXFP4 (E2M1 elements, E8M0 block scales) storage of the key window metadata
values     value codec with per-modality rotation R_m (Eq. 6, Eq. 3)
layout     packed byte layouts and the bits-per-element accounting (Tab. 3)
attention  decode attention over the quantized cache, two formulations (Eq. 1)
cache      whole-layer quantization into the packed cache buffers
residual   decode over the captioning protocol's mixed cache (fp16 residual)
calibration  modality-aware value-rotation calibration: attention weights, weighted
           covariance, eigenbasis, R_m = H U_m^T (Eq. 5, Eq. 6)
turboquant the TurboQuant key codec (Eq. 2, Eq. 3), the paper's baseline, and decode over it

Parity status: every function is pinned by a ``-m "not gpu"`` test except the
paper's measured error tables (Tab. 1, Tab. 3 error columns, Tab. 6), which
need real model activations: parity unpinned, and not reproduced.
"""
