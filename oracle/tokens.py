"""fp64 oracle of the per-token (rank-one) flip-flop (test infrastructure).

With samples G_t = g_t x_t^T (output gradient g_t, input x_t of token t),
Section 5 writes the two half steps as weighted second moments:
    A <- E[(g^T B^-1 g) x x^T],    B <- E[(x^T A^-1 x) g g^T].
With the same scalings as the dense form (the maximum-likelihood
stationarity conditions over T samples of m x n),
    B = (1/(T n)) sum_t (x_t^T A^-1 x_t) g_t g_t^T,
    A = (1/(T m)) sum_t (g_t^T B^-1 g_t) x_t x_t^T,
followed, per iteration, by the trace normalisation tr(A) = n and optional
damping by the mean diagonal (Appendix B), exactly as ``flipflop``.  The
weights come from Cholesky solves of all tokens at once; the weighted
moment is one product.  The tests pin this against the dense oracle run on
the materialised G_t.
"""
from __future__ import annotations

import numpy as np
import scipy.linalg as sla

from .flipflop import FlipFlopResult, LOG_2PI, _chol, blas_threads, damp, normalise


def _as_f64(V):
    V = np.asarray(V)
    if V.dtype == np.uint16:                       # bf16 bit patterns
        return (V.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return V.astype(np.float64)


def token_weights(V, F, what="factor", iteration=0):
    """w_t = v_t^T F^-1 v_t for the rows v_t of V (T, dim)."""
    cF = _chol(np.asarray(F, np.float64), what, iteration)
    S = sla.cho_solve(cF, V.T, check_finite=False)      # F^-1 v_t as columns
    return np.einsum("ti,it->t", V, S)


def half_step_B_tokens(x, g, A, *, iteration=0):
    """B = (1/(T n)) sum_t (x_t^T A^-1 x_t) g_t g_t^T."""
    x, g = _as_f64(x), _as_f64(g)
    T, n = x.shape
    w = token_weights(x, A, "A", iteration)
    return (g.T * w) @ g / (T * n)


def half_step_B_tokens_rows(x, g, A, rows, chunk=65536):
    """Rows ``rows`` of the B half step, for large token sets: tokens are
    converted to fp64 a chunk at a time.  A = None means the identity."""
    x = np.asarray(x)
    g = np.asarray(g)
    T, n = x.shape
    rows = np.asarray(rows)
    cA = None if A is None else _chol(np.asarray(A, np.float64), "A", 0)
    out = np.zeros((len(rows), g.shape[1]))
    for t0 in range(0, T, chunk):
        xc = _as_f64(x[t0:t0 + chunk])
        gc = _as_f64(g[t0:t0 + chunk])
        if cA is None:
            w = np.einsum("ti,ti->t", xc, xc)
        else:
            w = np.einsum("ti,it->t", xc, sla.cho_solve(cA, xc.T, check_finite=False))
        out += (gc[:, rows].T * w) @ gc
    return out / (T * n)


def half_step_A_tokens(x, g, B, *, iteration=0):
    """A = (1/(T m)) sum_t (g_t^T B^-1 g_t) x_t x_t^T."""
    x, g = _as_f64(x), _as_f64(g)
    T, m = g.shape
    v = token_weights(g, B, "B", iteration)
    return (x.T * v) @ x / (T * m)


def flipflop_tokens(x, g, iters, *, order="B_FIRST", damping=0.0, A0=None, B0=None,
                    keep_history=False) -> FlipFlopResult:
    """The flip-flop iteration on the tokens; same conventions as ``flipflop``."""
    x, g = _as_f64(x), _as_f64(g)
    T, n = x.shape
    m = g.shape[1]
    A = np.eye(n) if A0 is None else np.array(A0, dtype=np.float64)
    B = np.eye(m) if B0 is None else np.array(B0, dtype=np.float64)
    res = FlipFlopResult(A, B, 0)
    with blas_threads(m, n):
        for k in range(1, iters + 1):
            if order == "B_FIRST":
                B = damp(half_step_B_tokens(x, g, A, iteration=k), damping)
                A = damp(half_step_A_tokens(x, g, B, iteration=k), damping)
            elif order == "A_FIRST":
                A = damp(half_step_A_tokens(x, g, B, iteration=k), damping)
                B = damp(half_step_B_tokens(x, g, A, iteration=k), damping)
            else:
                raise ValueError(f"unknown order {order!r}")
            A, B = normalise(A, B)
            res.A, res.B, res.iters_done = A, B, k
            if keep_history:
                res.history.append((A.copy(), B.copy()))
    return res


def loglik_tokens(x, g, A, B):
    """Matrix-normal log-likelihood of the rank-one samples:
    tr(B^-1 g x^T A^-1 x g^T) = (x^T A^-1 x)(g^T B^-1 g)."""
    x, g = _as_f64(x), _as_f64(g)
    T, n = x.shape
    m = g.shape[1]
    w = token_weights(x, A, "A")
    v = token_weights(g, B, "B")
    ldA = 2.0 * np.sum(np.log(np.diag(np.linalg.cholesky(A))))
    ldB = 2.0 * np.sum(np.log(np.diag(np.linalg.cholesky(B))))
    return float(-0.5 * T * (m * ldA + n * ldB) - 0.5 * np.dot(w, v) - 0.5 * T * m * n * LOG_2PI)


def objective_tokens(x, g, A, B):
    """psi of ``objective`` (Section 4) for the rank-one samples."""
    x, g = _as_f64(x), _as_f64(g)
    T, n = x.shape
    m = g.shape[1]
    w = token_weights(x, A, "A")
    v = token_weights(g, B, "B")
    ldA = 2.0 * np.sum(np.log(np.diag(np.linalg.cholesky(A))))
    ldB = 2.0 * np.sum(np.log(np.diag(np.linalg.cholesky(B))))
    return float(np.log(np.dot(w, v) / (T * m * n)) + ldA / n + ldB / m)


def materialise(x, g):
    """The dense samples G_t = g_t x_t^T (T, m, n), for small T only."""
    x, g = _as_f64(x), _as_f64(g)
    return g[:, :, None] * x[:, None, :]
