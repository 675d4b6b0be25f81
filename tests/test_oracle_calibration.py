"""Pins of the value-rotation calibration oracle (Eq. 5, Eq. 6): attention weights against closed
forms of uniform and one-hot causal attention, covariance identities, the PCA special case against an
SVD, the TurboQuant special case R_m = H, the eigenvector conventions, and the recovery of the value
generator's per-modality subspaces."""

import math

import numpy as np
import pytest

from oracle.calibration import (attention_weights, calibrate_rotations, causal_attention_probs,
                                rotation_from_covariance, sorted_eigenbasis, value_covariance)
from oracle.hadamard import randomized_hadamard
from synth import gen_calibration_queries, gen_layer, gen_signs, value_bases, workload

SM = 1 / math.sqrt(128)


def test_uniform_attention_closed_form():
    """q = 0: query i spreads 1/(i+1) over tokens 0..i, so w_t = G sum_{i=t}^{L-1} 1/(i+1)^2."""
    rng = np.random.default_rng(1)
    B, H, G, L, D = 1, 2, 3, 40, 128
    q = np.zeros((B, H * G, L, D), np.float16)
    k = rng.standard_normal((B, H, L, D)).astype(np.float16)
    w = attention_weights(q, k, [L], SM)
    want = np.array([G * sum(1.0 / (i + 1) ** 2 for i in range(t, L)) for t in range(L)])
    for h in range(H):
        np.testing.assert_allclose(w[0, h], want, rtol=1e-13, atol=0)


def test_one_hot_attention_closed_form():
    """Queries and keys on distinct basis vectors, q_i = beta e_i, k_t = e_t: query i scores beta
    on its own token and 0 on the i earlier ones, so alpha_ii = e^b / (e^b + i) and alpha_it =
    1 / (e^b + i) for t < i; w_t = (e^b / (e^b + t))^2 + sum_{i > t} 1 / (e^b + i)^2."""
    L, D, beta = 24, 128, 3.0
    q = np.zeros((1, 1, L, D))
    k = np.zeros((1, 1, L, D))
    for i in range(L):
        q[0, 0, i, i] = beta / SM      # score = SM * q . k = beta on the diagonal
        k[0, 0, i, i] = 1.0
    w = attention_weights(q, k, [L], SM)[0, 0]
    eb = math.exp(beta)
    want = [(eb / (eb + t)) ** 2 + sum(1.0 / (eb + i) ** 2 for i in range(t + 1, L)) for t in range(L)]
    np.testing.assert_allclose(w, want, rtol=1e-12)


def test_probabilities_are_causal_rows():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((30, 128))
    k = rng.standard_normal((30, 128))
    a = causal_attention_probs(q, k, SM)
    np.testing.assert_allclose(a.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    assert np.all(a[np.triu_indices(30, 1)] == 0)
    # row i equals a textbook softmax of the first i + 1 scores
    i = 17
    s = SM * (k[:i + 1] @ q[i])
    np.testing.assert_allclose(a[i, :i + 1], np.exp(s) / np.exp(s).sum(), rtol=1e-13)


def test_weights_ignore_tokens_beyond_length_and_sum_bounds():
    wl = workload("tiny_1k")
    lay = gen_layer(wl, 0, lengths=np.array([200, 77], np.int32), n_tokens=200)
    q = gen_calibration_queries(wl.wid, 0, 2, 4, 200)
    w = attention_weights(q, lay["k"], [200, 77], SM)
    assert np.all(w[1, :, 77:] == 0)
    # each query contributes sum_t alpha^2 in [1 / (i + 1), 1]: bounds on the total
    for b, L in enumerate((200, 77)):
        tot = w[b].sum(axis=-1)
        assert np.all(tot <= 4 * L + 1e-9)
        assert np.all(tot >= 4 * sum(1.0 / (i + 1) for i in range(L)) - 1e-9)
    # the last token is seen by the last query only
    a_last = [causal_attention_probs(q[0, j, :200], lay["k"][0, 0, :200], SM)[199, 199] for j in range(4)]
    np.testing.assert_allclose(w[0, 0, 199], sum(x * x for x in a_last), rtol=1e-12)


def test_covariance_identities():
    rng = np.random.default_rng(3)
    B, H, N, D = 2, 2, 90, 128
    v = rng.standard_normal((B, H, N, D)).astype(np.float16)
    mod = rng.integers(0, 3, (B, N)).astype(np.uint8)
    w = rng.random((B, H, N))
    lens = [90, 61]
    C = value_covariance(v, mod, w, lens)
    for m in range(3):
        np.testing.assert_allclose(C[m], C[m].T, rtol=1e-13, atol=1e-13)
        assert np.linalg.eigvalsh(C[m]).min() > -1e-10
        tr = sum(w[b, h, t] * float(np.sum(v[b, h, t].astype(np.float64) ** 2))
                 for b in range(B) for h in range(H) for t in range(lens[b]) if mod[b, t] == m)
        np.testing.assert_allclose(np.trace(C[m]), tr, rtol=1e-12)
    # a token of another modality, or beyond the length, does not move C_m
    v2 = v.copy()
    t = int(np.nonzero(mod[0, :90] != 0)[0][0])
    v2[0, 0, t] += np.float16(1.0)
    v2[1, 1, 70] += np.float16(1.0)
    C2 = value_covariance(v2, mod, w, lens)
    np.testing.assert_array_equal(C2[0], C[0])


def test_rank_of_noise_free_subspace():
    """Values in a rank-16 subspace give exactly 16 nonzero eigenvalues, spanning that subspace."""
    rng = np.random.default_rng(4)
    basis = np.linalg.qr(rng.standard_normal((128, 16)))[0]
    v = (rng.standard_normal((1, 1, 300, 16)) @ basis.T)
    mod = np.full((1, 300), 1, np.uint8)
    C = value_covariance(v, mod, rng.random((1, 1, 300)) + 0.1, [300])
    ev, U = sorted_eigenbasis(C[1])
    assert ev[15] > 1e-6 * ev[0] and abs(ev[16]) < 1e-10 * ev[0]
    proj = U[:, :16].T @ basis
    np.testing.assert_allclose(np.linalg.svd(proj, compute_uv=False), 1.0, atol=1e-10)


def test_uniform_weights_give_pca():
    """Equal weights: U_m are the right singular vectors of V_m (an SVD, a different routine), and
    the eigenvalues are w times the squared singular values."""
    rng = np.random.default_rng(5)
    v = rng.standard_normal((1, 1, 400, 128)) * np.linspace(3.0, 0.1, 128)
    mod = np.zeros((1, 400), np.uint8)
    C = value_covariance(v, mod, np.full((1, 1, 400), 0.5), [400])
    ev, U = sorted_eigenbasis(C[0])
    _, sv, vt = np.linalg.svd(v[0, 0])
    np.testing.assert_allclose(ev, 0.5 * sv ** 2, rtol=1e-10)
    np.testing.assert_allclose(np.abs(np.sum(U * vt.T, axis=0)), 1.0, atol=1e-8)  # same vectors up to sign


def test_rotation_special_cases_and_conventions():
    signs = gen_signs(7, 0)
    H = randomized_hadamard(signs)
    # C diagonal with decreasing entries: U = I, so R_m = H (the TurboQuant rotation of Eq. 2)
    C = np.stack([np.diag(np.linspace(5.0, 1.0, 128))] * 3)
    R, ev, U = rotation_from_covariance(C, signs)
    np.testing.assert_allclose(U[0], np.eye(128), atol=0)
    np.testing.assert_allclose(R[1], H, atol=1e-15)
    # increasing entries: U is the reversal permutation
    C2 = np.stack([np.diag(np.linspace(1.0, 5.0, 128))] * 3)
    _, _, U2 = rotation_from_covariance(C2, signs)
    np.testing.assert_array_equal(U2[2], np.eye(128)[:, ::-1])
    # a hand example: the pair block [[2, 1], [1, 2]] has eigenvector (1, 1)/sqrt(2) for 3 and
    # (1, -1)/sqrt(2) for 1 -- its largest component (the first, on the tie) made positive
    C3 = np.zeros((1, 128, 128))
    C3[0, :2, :2] = [[2.0, 1.0], [1.0, 2.0]]
    C3[0, 2:, 2:] = np.diag(np.linspace(0.9, 0.1, 126))
    ev3, U3 = sorted_eigenbasis(C3[0])
    np.testing.assert_allclose(ev3[:2], [3.0, 1.0], rtol=1e-14)
    np.testing.assert_allclose(U3[:2, 0], [1 / math.sqrt(2)] * 2, rtol=1e-14)
    np.testing.assert_allclose(U3[:2, 1], [1 / math.sqrt(2), -1 / math.sqrt(2)], rtol=1e-14)
    # R_m is orthogonal and H^T R_m = U_m^T
    rng = np.random.default_rng(6)
    A = rng.standard_normal((3, 128, 128))
    Rr, _, Ur = rotation_from_covariance(A @ A.transpose(0, 2, 1), signs)
    for m in range(3):
        np.testing.assert_allclose(Rr[m] @ Rr[m].T, np.eye(128), atol=1e-12)
        np.testing.assert_allclose(H.T @ Rr[m], Ur[m].T, atol=1e-12)


@pytest.mark.parametrize("modality", [0, 1])
def test_generator_subspaces_recovered(modality):
    """On the synthetic workload the top 16 eigenvectors of C_m span the value generator's rank-16
    basis of modality m (principal-angle cosines near 1: the remaining energy is the 0.05 noise;
    random 16-dimensional subspaces of R^128 would give cosines near 0.35)."""
    wl = workload("tiny_1k")
    L = 1024
    lay = gen_layer(wl, 0, lengths=np.array([L], np.int32), n_tokens=L)
    q = gen_calibration_queries(wl.wid, 0, 1, 4, L)
    R, ev, U, C, w = calibrate_rotations(q, lay["k"], lay["v"], lay["modality"], [L], lay["signs"], SM)
    basis = value_bases(wl.wid, 0, 0)[modality]
    cos = np.linalg.svd(U[modality][:, :16].T @ basis, compute_uv=False)
    assert cos.min() > 0.98, cos.min()
    assert ev[modality][15] > 10 * ev[modality][16]
