"""Kronecker-factor application and the mismatch factor (fp64, test infrastructure).

* ``kron_apply``: with column-major vec (Section 2 notation),
  ``(A (x) B) vec(X) = vec(B X A^T)``; A is symmetric, so the product is
  ``B X A``.  The inverse uses ``(A (x) B)^-1 = A^-1 (x) B^-1``.
* ``mismatch_factor``: Section 4, Phi(H, A (x) B) as the ratio of the
  arithmetic to the geometric mean of the generalised eigenvalues of
  (H, A (x) B); only for tiny m n, where H can be formed explicitly.
"""
from __future__ import annotations

import numpy as np
import scipy.linalg as sla


def kron_apply(A, B, X, inverse=False):
    """Y_b = B X_b A (or B^-1 X_b A^-1) for X of shape (batch, m, n)."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    X = np.asarray(X, np.float64)
    if not inverse:
        return np.einsum("ij,bjk,kl->bil", B, X, A)
    cA = sla.cho_factor(A, lower=True)
    cB = sla.cho_factor(B, lower=True)
    out = np.empty_like(X)
    for b in range(X.shape[0]):
        Y = sla.cho_solve(cB, X[b])                 # B^-1 X
        out[b] = sla.cho_solve(cA, Y.T).T           # (A^-1 Y^T)^T = Y A^-1
    return out


def mismatch_factor(H, A, B):
    """Phi(H, A (x) B) = AM / GM of the generalised eigenvalues of (H, A (x) B)."""
    K = np.kron(np.asarray(A, np.float64), np.asarray(B, np.float64))
    lam = sla.eigh(np.asarray(H, np.float64), K, eigvals_only=True)
    return float(np.mean(lam) / np.exp(np.mean(np.log(lam))))
