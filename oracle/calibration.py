"""Modality-aware value-rotation calibration (Sec. 2.3, Eq. 5 and Eq. 6) -- TEST INFRASTRUCTURE (oracle).

Eq. 5 weights every cached value by how strongly it contributes to the attention output,
w_j = sum_i alpha_{i,j}^2, and forms one weighted second-moment matrix per modality,
C_m = sum_{j in m} w_j v_j^T v_j (v_j a row vector). The basis U_m comes from the
eigendecomposition of C_m, and Eq. 6 replaces the value Hadamard rotation by R_m = H U_m^T.

Readings (the paper gives the formulas and names the calibration set only):
* R25 -- alpha_{i,j} are the causal softmax attention weights of calibration query i over the
  tokens j <= i of the same sequence (scores q_i . k_j times sm_scale); every position i < L is a
  calibration query, and w_j sums over every query head that reads the KV head (GQA group) as
  well as over i;
* R26 -- v_j are the raw fp16 value vectors (not their unit directions), as Eq. 5 writes them;
* R27 -- one C_m per layer and modality: the sums run over the sequences and KV heads of the
  layer, so that one R_m serves every head (R13);
* R28 -- H is the layer's randomized Hadamard H = Had diag(s) / sqrt(d) (R5, the rotation Eq. 6
  replaces), with the signs passed in;
* R15 -- U_m has the eigenvectors as columns in descending eigenvalue order, each with its
  largest-magnitude component positive (the first such component on ties). Eigenvectors of
  (nearly) equal eigenvalues are not unique; comparisons use what is.

Float64 throughout (numpy), no blocking beyond the formulas.
"""

from __future__ import annotations

import numpy as np

from .hadamard import randomized_hadamard


def causal_attention_probs(q: np.ndarray, k: np.ndarray, sm_scale: float) -> np.ndarray:
    """alpha [L][L] float64 for queries q [L][d] over keys k [L][d]: row i is the softmax of
    sm_scale * q_i . k_j over j <= i (zero for j > i)."""
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    L = q.shape[0]
    s = sm_scale * (q @ k.T)
    s[np.triu_indices(L, 1)] = -np.inf
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    return p / p.sum(axis=1, keepdims=True)


def attention_weights(q16: np.ndarray, k16: np.ndarray, lens, sm_scale: float) -> np.ndarray:
    """w [B][H][N] float64 (Eq. 5): w_j = sum over the query heads of KV head h and the queries i
    of alpha_{i,j}^2; zero beyond each sequence's length.

    q16 [B][Hq][N][d] calibration queries, k16 [B][H][N][d] keys, lens [B]."""
    B, Hq, N, _ = q16.shape
    H = k16.shape[1]
    G = Hq // H
    w = np.zeros((B, H, N))
    for b in range(B):
        L = int(lens[b])
        if L == 0:
            continue
        for h in range(H):
            for j in range(h * G, (h + 1) * G):
                a = causal_attention_probs(q16[b, j, :L], k16[b, h, :L], sm_scale)
                w[b, h, :L] += (a * a).sum(axis=0)
    return w


def value_covariance(v16: np.ndarray, modality: np.ndarray, w: np.ndarray, lens, num_modalities: int = 3):
    """C [M][d][d] float64 (Eq. 5): C_m = sum over sequences, KV heads and tokens j < L of
    modality m of w_j v_j^T v_j."""
    B, H, N, D = v16.shape
    C = np.zeros((num_modalities, D, D))
    for b in range(B):
        L = int(lens[b])
        mod = np.asarray(modality[b, :L])
        for h in range(H):
            V = np.asarray(v16[b, h, :L], np.float64)
            wt = np.asarray(w[b, h, :L], np.float64)
            for m in range(num_modalities):
                sel = mod == m
                C[m] += V[sel].T @ (wt[sel, None] * V[sel])
    return C


def sorted_eigenbasis(C: np.ndarray):
    """(eigenvalues descending [d], U [d][d] with the eigenvectors as columns) of a symmetric C,
    signs fixed by R15."""
    evals, U = np.linalg.eigh(np.asarray(C, np.float64))
    order = np.argsort(-evals, kind="stable")
    evals, U = evals[order], U[:, order].copy()
    for c in range(U.shape[1]):
        i = int(np.argmax(np.abs(U[:, c])))
        if U[i, c] < 0:
            U[:, c] = -U[:, c]
    return evals, U


def rotation_from_covariance(C: np.ndarray, signs: np.ndarray):
    """(R [M][d][d], eigenvalues [M][d], U [M][d][d]): R_m = H U_m^T (Eq. 6), H the randomized
    Hadamard of the signs (R28)."""
    H = randomized_hadamard(signs)
    M, D, _ = C.shape
    R = np.zeros((M, D, D))
    ev = np.zeros((M, D))
    Us = np.zeros((M, D, D))
    for m in range(M):
        ev[m], Us[m] = sorted_eigenbasis(C[m])
        R[m] = H @ Us[m].T
    return R, ev, Us


def calibrate_rotations(q16, k16, v16, modality, lens, signs, sm_scale):
    """The whole calibration: weights, covariances and rotations (R, eigenvalues, U, C, w)."""
    w = attention_weights(q16, k16, lens, sm_scale)
    C = value_covariance(v16, modality, w, lens)
    R, ev, U = rotation_from_covariance(C, signs)
    return R, ev, U, C, w
