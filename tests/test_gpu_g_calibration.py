"""GPU parity of the value-rotation calibration (Eq. 5, Eq. 6) against the float64 oracle.

* attention weights w_j = sum_i alpha_ij^2: within 3e-4 of each weight plus 1e-7 of the largest
  (fp16 products are exact on the matrix cores; the fp32 score accumulation over 128 channels,
  the hardware exp2 and the fp32 sums of up to G L squared weights stay far inside that), and the
  closed form of uniform attention (q = 0);
* the weighted covariance, given the same weights: within 1e-5 of sum_t w_t |v_t| |v_t|^T per
  element (w v split into fp16 hi + lo parts: about 2^-22 per term, plus fp32 accumulation);
* the whole calibration: eigenvalues within 1e-4 of the largest, the top eigenvectors (those with a
  relative gap above 1e-2) within 2e-3, R_m orthogonal; a cache built with the calibrated R_m
  decodes within the decode tolerance of the oracle.
"""

import math

import numpy as np
import pytest

from oracle.calibration import attention_weights, rotation_from_covariance, value_covariance
from synth import gen_calibration_queries, gen_layer, gen_queries, workload

pytestmark = pytest.mark.gpu
SM = 1 / math.sqrt(128)


def _announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _inputs(wl_name, lens, H=None, Hq=None, layer=0):
    wl = workload(wl_name)
    N = max(max(lens), 1)
    lay = gen_layer(wl, layer, lengths=np.asarray(lens, np.int32), n_tokens=N)
    k, v = lay["k"], lay["v"]
    if H is not None:
        k, v = k[:, :H].copy(), v[:, :H].copy()
    Hkv = k.shape[1]
    Hq = Hq or wl.group * Hkv
    q = gen_calibration_queries(wl.wid, layer, len(lens), Hq, N)
    return wl, lay, q, k, v, N


def _gpu_weights(q, k, lens, N):
    import torch

    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    B, Hq = q.shape[:2]
    H = k.shape[1]
    dims = okvq.make_dims(B, H, Hq, 32)
    ws = okvq.calibration_workspace(dims, N)
    w = torch.full((B, H, N), float("nan"), dtype=torch.float32, device="cuda")
    okvq.okvq_calibration_weights(dims, gh.f16dev(q), gh.f16dev(k), N, list(lens), SM, w, ws)
    torch.cuda.synchronize()
    return w, ws, dims


def _gpu_cov(dims, v, modality, w, lens, N, ws):
    import torch

    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    cov = torch.full((3, 128, 128), float("nan"), dtype=torch.float32, device="cuda")
    okvq.okvq_value_covariance(dims, gh.f16dev(v), gh.dev(np.ascontiguousarray(modality, np.uint8)), w, N, list(lens),
                               cov, ws)
    torch.cuda.synchronize()
    return cov.cpu().numpy()


def _check_weights(got, ref, tag):
    bound = 3e-4 * ref + 1e-7 * ref.max()
    err = np.abs(got - ref)
    print(f"{tag}: weights max rel err {float((err / np.maximum(ref, 1e-30)).max()):.2e}, "
          f"worst / bound {float((err / bound).max()):.3f}", flush=True)
    assert np.all(err <= bound)


@pytest.mark.parametrize("case", ["tiny_513", "ragged_gqa7", "gqa8_long"])
def test_attention_weights(case):
    if case == "tiny_513":
        wl, lay, q, k, v, N = _inputs("tiny_1k", [513])
        lens = [513]
    elif case == "ragged_gqa7":
        lens = [300, 77, 1, 0, 160]
        wl, lay, q, k, v, N = _inputs("omni7b_32k", lens, H=2, Hq=14)
    else:
        lens = [1500]
        wl, lay, q, k, v, N = _inputs("omni3b_b4_64k_stream", lens, H=1, Hq=8)
    _announce(f"calibration weights {case} lens={lens} q={q.shape}")
    w, _, _ = _gpu_weights(q, k, lens, N)
    got = w.cpu().numpy().astype(np.float64)
    ref = attention_weights(q, k, lens, SM)
    _check_weights(got, ref, case)


def test_attention_weights_uniform_closed_form():
    """q = 0: w_t = G sum_{i >= t} 1 / (i + 1)^2 (no oracle involved)."""
    L, G = 200, 4
    rng = np.random.default_rng(11)
    q = np.zeros((1, G, L, 128), np.float16)
    k = rng.standard_normal((1, 1, L, 128)).astype(np.float16)
    _announce("calibration weights, uniform attention")
    w, _, _ = _gpu_weights(q, k, [L], L)
    want = np.array([G * sum(1.0 / (i + 1) ** 2 for i in range(t, L)) for t in range(L)])
    np.testing.assert_allclose(w.cpu().numpy()[0, 0], want, rtol=2e-5)


def test_covariance_given_weights():
    lens = [700, 333]
    wl, lay, q, k, v, N = _inputs("omni7b_32k", lens, H=2, Hq=14)
    _announce(f"calibration covariance lens={lens}")
    w, ws, dims = _gpu_weights(q, k, lens, N)
    cov = _gpu_cov(dims, v, lay["modality"], w, lens, N, ws)
    wn = w.cpu().numpy().astype(np.float64)
    ref = value_covariance(v, lay["modality"], wn, lens)
    absv = np.abs(v.astype(np.float64))
    scale = value_covariance(absv, lay["modality"], wn, lens)  # sum_t w_t |v_t| |v_t|^T
    err = np.abs(cov - ref)
    print(f"covariance worst err / scale = {float((err / np.maximum(scale, 1e-30)).max()):.2e}", flush=True)
    assert np.all(err <= 1e-5 * scale + 1e-30)


def test_calibration_end_to_end_and_decode_with_calibrated_rotation():
    import torch

    import gpu_helpers as gh
    import paper_2609_11582_amd as okvq
    from oracle.cache import decode_layer
    lens = [1024]
    wl, lay, q, k, v, N = _inputs("tiny_1k", lens)
    _announce("calibration end to end, then a cache with the calibrated rotations")
    w, ws, dims = _gpu_weights(q, k, lens, N)
    cov = _gpu_cov(dims, v, lay["modality"], w, lens, N, ws)
    rot = np.zeros((3, 128, 128), np.float32)
    ev = np.zeros((3, 128))
    okvq.okvq_rotation_from_covariance(cov, np.ascontiguousarray(lay["signs"], np.int8), rot, ev)
    wr = attention_weights(q, k, lens, SM)
    R_ref, ev_ref, U_ref = rotation_from_covariance(value_covariance(v, lay["modality"], wr, lens), lay["signs"])
    from oracle.hadamard import randomized_hadamard
    Hm = randomized_hadamard(lay["signs"])
    for m in range(3):
        top = ev_ref[m].max()
        np.testing.assert_allclose(ev[m], ev_ref[m], rtol=0, atol=1e-4 * top)
        d = np.abs(ev_ref[m][:, None] - ev_ref[m][None, :]) + np.eye(128) * 1e300
        gap = d.min(axis=1) / top
        sep = np.nonzero(gap > 1e-2)[0]
        U = (Hm.T @ rot[m].astype(np.float64)).T
        err = np.abs(U[:, sep] - U_ref[m][:, sep]).max() if len(sep) else 0.0
        print(f"modality {m}: {len(sep)} separated eigenvectors, max err {err:.2e}", flush=True)
        assert err <= 2e-3
        np.testing.assert_allclose(rot[m].astype(np.float64) @ rot[m].T, np.eye(128), atol=1e-5)
    # the calibrated rotations drive the codec and decode like any orthogonal R_m
    cache = okvq.KVCache(1, 1, 4, 1024, torch.from_numpy(lay["signs"]), torch.from_numpy(rot))
    gh.append_chunks(cache, lay["k"], lay["v"], lay["modality"], lens, [lens])
    qd = gen_queries(wl.wid, 0, 1, 4)
    out = gh.decode(cache, qd, lens)
    arrays = gh.cache_to_numpy(cache)
    ref = decode_layer(arrays, qd, np.asarray(lens), lay["signs"], rot, SM)
    r = gh.attention_close(out, ref)
    print(f"decode with the calibrated rotations: worst err / norm = {r:.2e}", flush=True)
    assert r <= 2e-3
