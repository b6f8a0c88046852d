"""fp64 oracle of the Hessian approximations of Table 1 other than FlipFlop
(test infrastructure only; never imported by the product path).

For H = E[x x^T (x) g g^T] (x: input, g: output gradient of a token), Table 1
lists
* Input:     A = E[x x^T],             B = I_m   (one-sided GPTQ's Hessian);
* Marginal:  A = E[x x^T],             B = E[g g^T];
* Frobenius: A = E[(g^T B g) x x^T],   B = E[(x^T A x) g g^T], alternating
             from the identity.  Section 5 describes it as the flip-flop
             iteration with A^-1, B^-1 replaced by A, B: a power iteration
             for min ||H - A (x) B||_F.

Readings where the paper gives the updates only up to a constant factor:
* Frobenius keeps every convention of ``flipflop``: B first from A = I_n,
  scalings 1/(N n) for B and 1/(N m) for A, optional damping right after each
  update, trace normalisation tr(A) = n after each iteration.  The two
  iterations differ only in using the factors instead of their inverses.
  For dense samples G_i: B <- (1/(N n)) sum_i G_i A G_i^T and
  A <- (1/(N m)) sum_i G_i^T B G_i.
* Input and Marginal are means over the tokens (they are not functions of
  the samples G_t = g_t x_t^T alone), optionally damped, then normalised the
  same way (the B of Input becomes c I_m).
"""
from __future__ import annotations

import numpy as np

from .flipflop import FlipFlopResult, as_f64_samples, blas_threads, damp, normalise
from .tokens import _as_f64


def frob_half_step_B(G, A):
    """B = (1/(N n)) sum_i G_i A G_i^T."""
    N, m, n = G.shape
    B = np.zeros((m, m))
    for Gi in G:
        B += Gi @ A @ Gi.T
    B /= N * n
    return 0.5 * (B + B.T)


def frob_half_step_A(G, B):
    """A = (1/(N m)) sum_i G_i^T B G_i."""
    N, m, n = G.shape
    A = np.zeros((n, n))
    for Gi in G:
        A += Gi.T @ B @ Gi
    A /= N * m
    return 0.5 * (A + A.T)


def frobenius(G, iters, *, order="B_FIRST", damping=0.0, keep_history=False) -> FlipFlopResult:
    """The Frobenius power iteration on samples G (N, m, n)."""
    G = as_f64_samples(G)
    N, m, n = G.shape
    A, B = np.eye(n), np.eye(m)
    res = FlipFlopResult(A, B, 0)
    with blas_threads(m, n):
        for k in range(1, iters + 1):
            if order == "B_FIRST":
                B = damp(frob_half_step_B(G, A), damping)
                A = damp(frob_half_step_A(G, B), damping)
            elif order == "A_FIRST":
                A = damp(frob_half_step_A(G, B), damping)
                B = damp(frob_half_step_B(G, A), damping)
            else:
                raise ValueError(f"unknown order {order!r}")
            A, B = normalise(A, B)
            res.A, res.B, res.iters_done = A, B, k
            if keep_history:
                res.history.append((A.copy(), B.copy()))
    return res


def frobenius_tokens(x, g, iters, *, order="B_FIRST", damping=0.0) -> FlipFlopResult:
    """The Frobenius iteration on tokens: B <- (1/(T n)) sum_t (x_t^T A x_t) g_t g_t^T,
    A <- (1/(T m)) sum_t (g_t^T B g_t) x_t x_t^T."""
    x, g = _as_f64(x), _as_f64(g)
    T, n = x.shape
    m = g.shape[1]
    A, B = np.eye(n), np.eye(m)

    def upd_B(A):
        w = np.einsum("ti,ij,tj->t", x, A, x)
        return (g.T * w) @ g / (T * n)

    def upd_A(B):
        v = np.einsum("ti,ij,tj->t", g, B, g)
        return (x.T * v) @ x / (T * m)

    res = FlipFlopResult(A, B, 0)
    for k in range(1, iters + 1):
        if order == "B_FIRST":
            B = damp(upd_B(A), damping)
            A = damp(upd_A(B), damping)
        elif order == "A_FIRST":
            A = damp(upd_A(B), damping)
            B = damp(upd_B(A), damping)
        else:
            raise ValueError(f"unknown order {order!r}")
        A, B = normalise(A, B)
        res.A, res.B, res.iters_done = A, B, k
    return res


def marginal_tokens(x, g, *, damping=0.0):
    """(A, B) = (E[x x^T], E[g g^T]) over the tokens, damped, trace-normalised."""
    x, g = _as_f64(x), _as_f64(g)
    T = x.shape[0]
    A = damp(x.T @ x / T, damping)
    B = damp(g.T @ g / T, damping)
    return normalise(A, B)


def input_tokens(x, m, *, damping=0.0):
    """(A, B) = (E[x x^T], I_m), damped, trace-normalised."""
    x = _as_f64(x)
    T = x.shape[0]
    A = damp(x.T @ x / T, damping)
    B = damp(np.eye(m), damping)
    return normalise(A, B)
