"""fp64 oracle of WaterKron: two-sided GPTQ with waterfilling scales
(test infrastructure only; never imported by the product path).

* ``rev_cholesky(M)``: the lower-triangular L with positive diagonal and
  L^T L = M (Section 2 notation).
* ``waterfilling_scales(A, B, gamma)``: Corollary 3.2's choice
  alpha_j = sqrt(gamma) |A|^(1/2n) / L^A_jj and beta_i = sqrt(gamma) |B|^(1/2m) / L^B_ii
  with L^A = RevCholesky(A), L^B = RevCholesky(B).
* ``gptq(W, A, alpha, beta)``: Algorithm 1 (input-sided GPTQ): columns in
  order, each rounded on its grid alpha_j beta_i, the error spread over the
  later columns through the column-normalised inverse factor.
* ``two_sided_gptq(W, A, B, alpha, beta)``: Algorithm 2: column j outer, row
  i inner; the error of entry (i, j) is spread with the outer product of the
  normalised inverse factors' columns i (output side) and j (input side).
* ``distortion(V, W, A, B)``: D_{A,B} = (1/(m n)) ||L^B (V - W) (L^A)^T||_F^2.

Rounding is to the nearest integer with ties to even (numpy ``rint``).  The
plain loops are O(m^2 n^2); for small layers only.
"""
from __future__ import annotations

import numpy as np


def rev_cholesky(M):
    """L lower triangular, positive diagonal, L^T L = M (via the reversal
    J: L = J chol(J M J)^T J; the products with the exchange matrix J are
    taken as the row and column reversals they are)."""
    M = np.asarray(M, np.float64)
    C = np.linalg.cholesky(np.ascontiguousarray(M[::-1, ::-1]))      # chol(J M J)
    return np.ascontiguousarray(C.T[::-1, ::-1])                     # J C^T J


def normalised_inverse(M):
    """L^-1 of L = RevCholesky(M), each column divided by its diagonal entry."""
    Lt = np.linalg.inv(rev_cholesky(M))
    return Lt / np.diag(Lt)[None, :]


def waterfilling_scales(A, B, gamma):
    """(alpha, beta) of Corollary 3.2."""
    LA = rev_cholesky(A)
    LB = rev_cholesky(B)
    n, m = LA.shape[0], LB.shape[0]
    gA = np.exp(np.sum(np.log(np.diag(LA))) / n)     # |A|^(1/2n)
    gB = np.exp(np.sum(np.log(np.diag(LB))) / m)
    alpha = np.sqrt(gamma) * gA / np.diag(LA)
    beta = np.sqrt(gamma) * gB / np.diag(LB)
    return alpha, beta


def gptq(W, A, alpha, beta):
    """Algorithm 1. Returns (Z, V)."""
    W = np.array(W, dtype=np.float64)
    m, n = W.shape
    Lt = normalised_inverse(A)
    Z = np.zeros((m, n), dtype=np.int64)
    for j in range(n):
        step = alpha[j] * np.asarray(beta, np.float64)
        Z[:, j] = np.rint(W[:, j] / step).astype(np.int64)
        delta = step * Z[:, j] - W[:, j]
        W += np.outer(delta, Lt[:, j])
    V = np.outer(beta, alpha) * Z
    return Z, V


def two_sided_gptq(W, A, B, alpha, beta):
    """Algorithm 2. Returns (Z, V)."""
    W = np.array(W, dtype=np.float64)
    m, n = W.shape
    LtA = normalised_inverse(A)
    LtB = normalised_inverse(B)
    Z = np.zeros((m, n), dtype=np.int64)
    for j in range(n):
        for i in range(m):
            step = alpha[j] * beta[i]
            Z[i, j] = int(np.rint(W[i, j] / step))
            delta = step * Z[i, j] - W[i, j]
            W += delta * np.outer(LtB[:, i], LtA[:, j])
    V = np.outer(beta, alpha) * Z
    return Z, V


def distortion(V, W, A, B):
    """D_{A,B} of Section 3 (two-sided distortion), with L = RevCholesky."""
    V = np.asarray(V, np.float64)
    W = np.asarray(W, np.float64)
    m, n = W.shape
    X = rev_cholesky(B) @ (V - W) @ rev_cholesky(A).T
    return float(np.sum(X * X) / (m * n))
