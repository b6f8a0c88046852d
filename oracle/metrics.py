"""Comparison metrics between two Kronecker products (fp64, test infrastructure).

The parity measure is the relative Frobenius error of the normalised
product A (x) B.  The mn x mn product is never formed: with dA = A - A*,
dB = B - B*,

    A (x) B - A* (x) B* = dA (x) B + A* (x) dB,

and ||X (x) Y||_F = ||X||_F ||Y||_F, <X1 (x) Y1, X2 (x) Y2> = <X1,X2><Y1,Y2>, so

    ||A(x)B - A*(x)B*||^2 = ||dA||^2 ||B||^2 + ||A*||^2 ||dB||^2
                           + 2 <dA, A*> <B, dB>.

Every term is formed from the differences themselves, so the result has no
cancellation floor (the expanded form ||A||^2||B||^2 - 2<A,A*><B,B*> + ...
loses half the digits).
"""
from __future__ import annotations

import numpy as np


def _f64(X):
    return np.asarray(X, dtype=np.float64)


def kron_rel_error(A, B, A_ref, B_ref) -> float:
    """||A(x)B - A_ref(x)B_ref||_F / ||A_ref(x)B_ref||_F, evaluated in fp64."""
    A, B, A_ref, B_ref = map(_f64, (A, B, A_ref, B_ref))
    dA = A - A_ref
    dB = B - B_ref
    sq = (np.sum(dA * dA) * np.sum(B * B) + np.sum(A_ref * A_ref) * np.sum(dB * dB)
          + 2.0 * np.sum(dA * A_ref) * np.sum(B * dB))
    den = np.sqrt(np.sum(A_ref * A_ref) * np.sum(B_ref * B_ref))
    return float(np.sqrt(max(sq, 0.0)) / den)


def kron_rel_error_scale_free(A, B, A_ref, B_ref) -> float:
    """|| A(x)B / ||A(x)B|| - A_ref(x)B_ref / ||A_ref(x)B_ref|| ||_F: the error
    of the products' directions, blind to an overall scale (the error
    metric's scale-free companion).  Each factor is scaled to unit norm (the
    product then has unit norm) and the stable form above is applied."""
    A, B, A_ref, B_ref = map(_f64, (A, B, A_ref, B_ref))
    unit = lambda X: X / np.sqrt(np.sum(X * X))
    return kron_rel_error(unit(A), unit(B), unit(A_ref), unit(B_ref))


def trace_identity(G, A, B) -> float:
    """(1/(N m n)) sum_i tr(B^-1 G_i A^-1 G_i^T)  (Section 5 trace identity).

    Equals 1 after an exact maximum-likelihood half step.  Computed with
    plain inverses, independently of the solves in the iteration.
    """
    from .flipflop import as_f64_samples
    G = as_f64_samples(G)
    N, m, n = G.shape
    Ai = np.linalg.inv(_f64(A))
    Bi = np.linalg.inv(_f64(B))
    tot = 0.0
    for Gi in G:
        tot += np.sum((Bi @ Gi) * (Gi @ Ai))
    return float(tot / (N * m * n))
