"""Seeded per-token workloads (the rank-one sample form G_t = g_t x_t^T).

The paper estimates the Hessian of a linear layer from calibration tokens:
each token contributes an input x_t (n) and an output gradient g_t (m), and
H = E[x x^T (x) g g^T].  Those activations and gradients are not available
here; this generator stands in for them.

Recipe:

* two mixture components c = 0, 1 with equal weight, each with its own
  factor roots S_A^c = Q_A^c diag(sqrt(lambda_A)) and S_B^c (the power-law
  spectra of ``generator.power_law_spectrum``, independent Haar rotations
  drawn from ``default_rng([seed, 0, c])``), so that H = (1/2) sum_c
  A_c (x) B_c is not a Kronecker product;
* token t (in blocks of 4096 tokens, block b drawn from
  ``default_rng([seed, 2, b])``): component c_t ~ Bernoulli(1/2), input
  x_t = S_A^c z_t with z_t iid Student-t(4) scaled to unit variance (heavy
  tailed, like activation outliers), gradient g_t = S_B^c u_t with u_t iid
  N(0, 1);
* storage: the fp64 products rounded to fp32 (RNE) and, for bf16
  workloads, to bf16 (RNE), kept as uint16 bit patterns on the CPU.

Only random numbers and their products live here: no step of the method.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace

import numpy as np

from .generator import BASE_SEED, f32_to_bf16_bits, haar_orthogonal, power_law_spectrum

BLOCK = 4096


@dataclass(frozen=True)
class TokenWorkload:
    name: str
    m: int          # output channels (g_t), B is m x m
    n: int          # input channels (x_t), A is n x n
    T: int          # tokens
    iters: int
    p_A: float
    p_B: float
    dtype: str      # "f32" or "bf16"
    index: int      # seed offset

    @property
    def seed(self) -> int:
        return BASE_SEED + 100 + self.index

    @property
    def flop_per_iter(self) -> float:
        """Whitening norms (T n^2 and T m^2, triangular) and weighted
        symmetric products (T m^2 and T n^2), plus two factorisations."""
        m, n, T = self.m, self.n, self.T
        return 2.0 * T * (m * m + n * n) + (m ** 3 + n ** 3) / 3.0

    def scaled(self, **kw) -> "TokenWorkload":
        return replace(self, **kw)


TOKEN_WORKLOADS = {
    "tokens_tiny": TokenWorkload("tokens-tiny-48x80-T3000", 48, 80, 3000, 10, 1.0, 1.0, "f32", 0),
    # the paper's calibration set, 256 sequences of 2048 tokens, at the
    # attention-layer width
    "tokens_attn": TokenWorkload("tokens-attn-4096x4096-T524288", 4096, 4096, 524288, 10,
                                 1.2, 0.8, "bf16", 1),
}


def token_workload(key: str) -> TokenWorkload:
    return TOKEN_WORKLOADS[key]


def _roots(w: TokenWorkload, seed: int):
    lamA = power_law_spectrum(w.n, w.p_A)
    lamB = power_law_spectrum(w.m, w.p_B)
    out = []
    for c in range(2):
        rng = np.random.default_rng([seed, 0, c])
        QA = haar_orthogonal(w.n, rng)
        QB = haar_orthogonal(w.m, rng)
        out.append((QA * np.sqrt(lamA)[None, :], QB * np.sqrt(lamB)[None, :]))
    return out


def _draw_block(w: TokenWorkload, seed: int, b: int):
    """Component labels, z (t4, unit variance) and u (normal) of block b."""
    t0 = b * BLOCK
    cnt = min(BLOCK, w.T - t0)
    rng = np.random.default_rng([seed, 2, b])
    c = rng.integers(0, 2, size=cnt)
    z = rng.standard_t(4, size=(cnt, w.n)) / np.sqrt(2.0)
    u = rng.standard_normal((cnt, w.m))
    return t0, c, z, u


def _store(X, dtype):
    X32 = X.astype(np.float32)
    return f32_to_bf16_bits(X32) if dtype == "bf16" else X32


@dataclass
class TokenDraw:
    workload: TokenWorkload
    x: object        # (T, n): uint16 bf16 bits / float32 (numpy), or a torch tensor
    g: object        # (T, m)
    A_parts: list    # the two components' n x n factors (fp64)
    B_parts: list


def generate_tokens(w: TokenWorkload, seed: int | None = None,
                    threads: int | None = None) -> TokenDraw:
    """Draw all tokens on the CPU (numpy, fp64 products)."""
    seed = w.seed if seed is None else int(seed)
    roots = _roots(w, seed)
    dt = np.uint16 if w.dtype == "bf16" else np.float32
    x = np.empty((w.T, w.n), dtype=dt)
    g = np.empty((w.T, w.m), dtype=dt)

    def one(b):
        t0, c, z, u = _draw_block(w, seed, b)
        X = np.empty((len(c), w.n))
        Gd = np.empty((len(c), w.m))
        for k in range(2):
            sel = c == k
            X[sel] = z[sel] @ roots[k][0].T
            Gd[sel] = u[sel] @ roots[k][1].T
        x[t0:t0 + len(c)] = _store(X, w.dtype)
        g[t0:t0 + len(c)] = _store(Gd, w.dtype)

    nb = (w.T + BLOCK - 1) // BLOCK
    nthreads = threads or min(8, os.cpu_count() or 1)
    with ThreadPoolExecutor(max(1, nthreads)) as ex:
        list(ex.map(one, range(nb)))
    return TokenDraw(w, x, g, [S @ S.T for S, _ in roots], [S @ S.T for _, S in roots])


def generate_tokens_device(w: TokenWorkload, seed: int | None = None, *, device="cuda",
                           threads: int = 16):
    """Draw the tokens straight into device memory: the same numpy random
    streams, products in fp64 on the device.  Returns torch tensors (x, g)."""
    import torch

    seed = w.seed if seed is None else int(seed)
    dev = torch.device(device)
    roots = [(torch.from_numpy(SA).to(dev), torch.from_numpy(SB).to(dev))
             for SA, SB in _roots(w, seed)]
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    x = torch.empty((w.T, w.n), dtype=tdt, device=dev)
    g = torch.empty((w.T, w.m), dtype=tdt, device=dev)
    nb = (w.T + BLOCK - 1) // BLOCK
    with ThreadPoolExecutor(max(1, threads)) as ex:
        futs = {}
        for b in range(min(nb, 2 * threads)):
            futs[b] = ex.submit(_draw_block, w, seed, b)
        for b in range(nb):
            t0, c, z, u = futs.pop(b).result()
            if b + 2 * threads < nb:
                futs[b + 2 * threads] = ex.submit(_draw_block, w, seed, b + 2 * threads)
            cd = torch.from_numpy(c).to(dev)
            zd = torch.from_numpy(z).to(dev)
            ud = torch.from_numpy(u).to(dev)
            X = torch.empty((len(c), w.n), dtype=torch.float64, device=dev)
            Gd = torch.empty((len(c), w.m), dtype=torch.float64, device=dev)
            for k in range(2):
                sel = cd == k
                X[sel] = zd[sel] @ roots[k][0].T
                Gd[sel] = ud[sel] @ roots[k][1].T
            x[t0:t0 + len(c)] = X.float().to(tdt)
            g[t0:t0 + len(c)] = Gd.float().to(tdt)
    return x, g
