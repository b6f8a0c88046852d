"""The flip-flop iteration in fp64, written out directly.

Paper passages followed (Section 5, "The FlipFlop Hessian Approximation"):

* samples ``G = g x^T`` with ``vec(G) = x (x) g``, so ``H = E[vec G vec G^T]``
  and the Kronecker factors are A (n x n, input side) and B (m x m, output
  side) with ``H ~ A (x) B``;
* for fixed A the best B is proportional to ``S = E[G A^-1 G^T]``, and for
  fixed B the best A is proportional to ``E[G^T B^-1 G]`` (the AM-GM argument);
* alternating the two gives the flip-flop iteration, the matrix-normal
  maximum-likelihood iteration, whose fixed point is unique up to scale when
  H is positive definite;
* Appendix B: A starts at the identity, one iteration updates B and then A,
  and both factors may be damped by a multiple of their mean diagonal,
  including between iterations.

Readings taken where the paper gives the updates only up to a constant factor:

* the expectation is the empirical mean over the N samples;
* B is scaled by 1/(N n) and A by 1/(N m): the maximum-likelihood
  stationarity conditions of the matrix-normal model, so that every half step
  is an exact likelihood maximiser;
* after each full iteration the scale ambiguity is removed by
  ``c = tr(A)/n, A <- A/c, B <- B c`` (A (x) B is unchanged);
* damping, when used, adds ``kappa * tr(X)/dim * I`` right after the update
  of X, before X is used again or normalised;
* no centring of the samples (H is the uncentred second moment).

The computation is the direct form: per sample a Cholesky solve
(``cho_solve``) and a dense product, accumulated in fp64.  It is independent
of the GPU design (whitening with an explicit triangular inverse followed by
a symmetric rank-k product).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import contextlib

import numpy as np
import scipy.linalg as sla
from threadpoolctl import threadpool_info, threadpool_limits

LOG_2PI = float(np.log(2.0 * np.pi))

# threadpoolctl finds the C library once per process, by running `ldconfig` in
# a child process.  Do it when the oracle is imported, so that it never has to
# start a child process later, from a process that already drives a GPU.
threadpool_info()


def blas_threads(m, n):
    """BLAS thread budget: one thread for small factors (per-call overhead
    of a threaded BLAS dominates there), the library default otherwise."""
    if max(m, n) <= 512:
        return threadpool_limits(limits=1, user_api="blas")
    return contextlib.nullcontext()


class NotSPDError(np.linalg.LinAlgError):
    """A factor that must be inverted is not positive definite.

    The paper assumes every PSD matrix it inverts is invertible (Section 2,
    notation) and recommends damping otherwise.
    """

    def __init__(self, msg, iteration):
        super().__init__(msg)
        self.iteration = iteration


def as_f64_samples(G) -> np.ndarray:
    """Samples as fp64 (N, m, n).  uint16 input is read as bf16 bit patterns.

    Both conversions are exact.
    """
    G = np.asarray(G)
    if G.dtype == np.uint16:
        G = (G.astype(np.uint32) << np.uint32(16)).view(np.float32)
    if G.ndim != 3:
        raise ValueError("G must be (N, m, n)")
    return G.astype(np.float64)


def _chol(X, what, iteration):
    if not np.all(np.isfinite(X)):
        raise NotSPDError(f"{what} has non-finite entries", iteration)
    try:
        return sla.cho_factor(X, lower=True, check_finite=False)
    except np.linalg.LinAlgError as e:
        raise NotSPDError(f"{what} is not positive definite: {e}", iteration) from None


def half_step_B(G, A, *, iteration=0):
    """B = (1/(N n)) sum_i G_i A^-1 G_i^T  (Section 5, update of B)."""
    N, m, n = G.shape
    cA = _chol(A, "A", iteration)
    B = np.zeros((m, m))
    for Gi in G:
        B += Gi @ sla.cho_solve(cA, Gi.T, check_finite=False)
    B /= N * n
    return 0.5 * (B + B.T)


def half_step_A(G, B, *, iteration=0):
    """A = (1/(N m)) sum_i G_i^T B^-1 G_i  (Section 5, update of A)."""
    N, m, n = G.shape
    cB = _chol(B, "B", iteration)
    A = np.zeros((n, n))
    for Gi in G:
        A += Gi.T @ sla.cho_solve(cB, Gi, check_finite=False)
    A /= N * m
    return 0.5 * (A + A.T)


def half_step_B_rows(G, A, rows, progress=None):
    """Rows ``rows`` of the B update (1/(N n)) sum_i G_i A^-1 G_i^T
    (Section 5, update of B); A = None means the identity.

    Row r of sample i's term is (A^-1 G_i[r]^T)^T G_i^T, one Cholesky solve
    per selected row.  For large layers: the samples are converted to fp64
    one at a time (uint16 = bf16 bit patterns), so only one sample is held
    in fp64.  ``progress(i)``, if given, is called after sample i.
    """
    G = np.asarray(G)
    N, m, n = G.shape
    rows = np.asarray(rows)
    identity = A is None
    cA = None if identity else _chol(np.asarray(A, np.float64), "A", 0)
    out = np.zeros((len(rows), m))
    for i in range(N):
        Gi = as_f64_samples(G[i:i + 1])[0]
        R = Gi[rows]                                    # (r, n)
        if not identity:
            R = sla.cho_solve(cA, R.T, check_finite=False).T
        out += R @ Gi.T
        if progress is not None:
            progress(i)
    return out / (N * n)


def half_step_A_rows(G, B, rows, progress=None):
    """Rows ``rows`` of the A update (1/(N m)) sum_i G_i^T B^-1 G_i
    (Section 5, update of A); B = None means the identity.

    Row c of sample i's term is (B^-1 G_i[:, c])^T G_i, one Cholesky solve
    per selected column of G_i; samples are converted one at a time.
    ``progress(i)``, if given, is called after sample i.
    """
    G = np.asarray(G)
    N, m, n = G.shape
    rows = np.asarray(rows)
    identity = B is None
    cB = None if identity else _chol(np.asarray(B, np.float64), "B", 0)
    out = np.zeros((len(rows), n))
    for i in range(N):
        Gi = as_f64_samples(G[i:i + 1])[0]
        C = Gi[:, rows]                                 # (m, r)
        if not identity:
            C = sla.cho_solve(cB, C, check_finite=False)
        out += C.T @ Gi
        if progress is not None:
            progress(i)
    return out / (N * m)


def damp(X, kappa):
    """X + kappa * (tr X / dim) I  (Appendix B: damping by the mean diagonal)."""
    if kappa == 0.0:
        return X
    d = X.shape[0]
    return X + (kappa * np.trace(X) / d) * np.eye(d)


def normalise(A, B):
    """Remove the scale ambiguity: tr(A) = n, A (x) B unchanged."""
    c = np.trace(A) / A.shape[0]
    return A / c, B * c


def loglik(G, A, B):
    """Matrix-normal log-likelihood of the samples under Cov(vec G) = A (x) B.

    ``l = -(N/2)(m log|A| + n log|B|) - (1/2) sum_i tr(B^-1 G_i A^-1 G_i^T)
    - (N m n / 2) log 2 pi``; the trace term is the Section 5 trace identity
    and the relation to the mismatch factor is eq. (6) (Section 4).
    """
    G = as_f64_samples(G)
    N, m, n = G.shape
    with blas_threads(m, n):
        return _loglik(G, A, B)


def _loglik(G, A, B):
    N, m, n = G.shape
    cA = _chol(A, "A", -1)
    cB = _chol(B, "B", -1)
    logdetA = 2.0 * np.sum(np.log(np.diag(cA[0])))
    logdetB = 2.0 * np.sum(np.log(np.diag(cB[0])))
    quad = 0.0
    for Gi in G:
        quad += np.trace(sla.cho_solve(cB, Gi @ sla.cho_solve(cA, Gi.T, check_finite=False),
                                       check_finite=False))
    return -0.5 * N * (m * logdetA + n * logdetB) - 0.5 * quad - 0.5 * N * m * n * LOG_2PI


def objective(G, A, B):
    """The mismatch objective of Section 4 without its H-only term.

    With H = (1/N) sum_i vec(G_i) vec(G_i)^T, the mismatch factor is
    Phi(H, A (x) B) = [tr(H (A (x) B)^-1) / mn] / [|H|^(1/mn) |A (x) B|^(-1/mn)];
    tr(H (A (x) B)^-1) = (1/N) sum_i tr(B^-1 G_i A^-1 G_i^T) (column-major vec)
    and |A (x) B|^(1/mn) = |A|^(1/n) |B|^(1/m), so this returns
    psi = log((1/(N m n)) sum_i tr(B^-1 G_i A^-1 G_i^T)) + log|A|/n + log|B|/m
        = log Phi + log|H| / (m n),
    which stays finite when H is singular (N < m n).  Each sample's trace is
    taken directly with two Cholesky solves, as in ``loglik``.
    """
    G = as_f64_samples(G)
    N, m, n = G.shape
    with blas_threads(m, n):
        cA = _chol(A, "A", -1)
        cB = _chol(B, "B", -1)
        logdetA = 2.0 * np.sum(np.log(np.diag(cA[0])))
        logdetB = 2.0 * np.sum(np.log(np.diag(cB[0])))
        quad = 0.0
        for Gi in G:
            quad += np.trace(sla.cho_solve(cB, Gi @ sla.cho_solve(cA, Gi.T, check_finite=False),
                                           check_finite=False))
    return float(np.log(quad / (N * m * n)) + logdetA / n + logdetB / m)


@dataclass
class FlipFlopResult:
    A: np.ndarray
    B: np.ndarray
    iters_done: int
    history: list = field(default_factory=list)   # (A, B) after each full iteration
    half_steps: list = field(default_factory=list)  # ("B"|"A", A, B) after each half step


def flipflop(G, iters, *, order="B_FIRST", damping=0.0, A0=None, B0=None,
             keep_history=False, keep_half_steps=False) -> FlipFlopResult:
    """Run ``iters`` flip-flop iterations on samples G (N, m, n).

    ``order="B_FIRST"`` (Appendix B): start from A0 (default I_n), each
    iteration updates B from A, then A from B.  ``order="A_FIRST"``
    (Section 5 indexing): start from B0 (default I_m), update A then B.
    Every iteration ends with the trace normalisation tr(A) = n.

    Raises NotSPDError (with ``.iteration``, 1-based) if a factor that must
    be inverted is not positive definite.
    """
    G = as_f64_samples(G)
    N, m, n = G.shape
    A = np.eye(n) if A0 is None else np.array(A0, dtype=np.float64)
    B = np.eye(m) if B0 is None else np.array(B0, dtype=np.float64)
    res = FlipFlopResult(A, B, 0)
    with blas_threads(m, n):
        _run(G, A, B, iters, order, damping, keep_history, keep_half_steps, res)
    return res


def _run(G, A, B, iters, order, damping, keep_history, keep_half_steps, res):
    for k in range(1, iters + 1):
        if order == "B_FIRST":
            B = damp(half_step_B(G, A, iteration=k), damping)
            if keep_half_steps:
                res.half_steps.append(("B", A.copy(), B.copy()))
            A = damp(half_step_A(G, B, iteration=k), damping)
            if keep_half_steps:
                res.half_steps.append(("A", A.copy(), B.copy()))
        elif order == "A_FIRST":
            A = damp(half_step_A(G, B, iteration=k), damping)
            if keep_half_steps:
                res.half_steps.append(("A", A.copy(), B.copy()))
            B = damp(half_step_B(G, A, iteration=k), damping)
            if keep_half_steps:
                res.half_steps.append(("B", A.copy(), B.copy()))
        else:
            raise ValueError(f"unknown order {order!r}")
        A, B = normalise(A, B)
        res.A, res.B, res.iters_done = A, B, k
        if keep_history:
            res.history.append((A.copy(), B.copy()))
