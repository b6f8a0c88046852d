"""Workload table and seeded generators (CPU numpy, or torch on a device).

Recipe (stated once, used by every test and by the benchmark):

* spectra: ``lambda_k = c * k**(-p)``, k = 1..dim, with c chosen so that the
  trace equals ``dim`` (mean eigenvalue 1);
* eigenvectors: Haar orthogonal Q from the QR factorisation of a Gaussian
  matrix with the sign of diag(R) folded into Q;
* square roots: ``S = Q diag(sqrt(lambda))`` so that ``S S^T`` is the true
  factor (any square root gives the same law);
* samples: ``G_i = S_B Z_i S_A^T (+ sigma_p U_i V_i^T)`` with Z_i iid N(0,1)
  (or Student-t(nu) scaled to unit variance) and U_i (m x r), V_i (n x r) iid
  N(0,1); ``sigma_p**2 = rho * tr(A) tr(B) / (m n r)`` makes the expected
  energy of the low-rank term ``rho`` times that of the Kronecker term;
* storage: the fp64 product is rounded to fp32 (RNE) and, for bf16
  workloads, to bf16 (RNE) and kept as uint16 bit patterns;
* seeds: the factors come from ``default_rng([seed, 0])``; sample i draws
  Z_i, then U_i, then V_i from ``default_rng([seed, 1, i])``, so any subset
  of samples can be drawn on its own and in parallel.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace

import numpy as np

BASE_SEED = 20261202


@dataclass(frozen=True)
class Workload:
    name: str
    m: int          # output channels: rows of G, B is m x m
    n: int          # input channels: columns of G, A is n x n
    N: int          # number of samples G_i
    iters: int      # flip-flop iterations the workload is run for
    p_A: float      # power-law exponent of A's spectrum
    p_B: float      # power-law exponent of B's spectrum
    dist: str       # "normal" or "t<nu>"
    rank: int       # rank of the per-sample non-Kronecker term (0 = none)
    rho: float      # its energy relative to the Kronecker term
    dtype: str      # storage / compute path: "f32" or "bf16"
    index: int      # position in the workload table (seed offset)

    @property
    def seed(self) -> int:
        return BASE_SEED + self.index

    @property
    def flop_per_iter(self) -> float:
        """Algorithmic work of one flip-flop iteration.

        Whitening (triangular, N m n^2 and N m^2 n) plus the symmetric
        products (N n m^2 and N m n^2) give 2 N m n (m + n); the two
        Cholesky factorisations add (m^3 + n^3)/3.
        """
        m, n, N = self.m, self.n, self.N
        return 2.0 * N * m * n * (m + n) + (m ** 3 + n ** 3) / 3.0

    def scaled(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    "tiny": Workload("tiny-64x128-N256", 64, 128, 256, 20, 1.0, 1.0, "normal", 0, 0.0, "f32", 0),
    "attn": Workload("attn-4096x4096-N128", 4096, 4096, 128, 10, 1.2, 0.8, "normal", 32, 0.1, "bf16", 1),
    "mlp_up": Workload("mlp-up-11008x4096-N128", 11008, 4096, 128, 10, 1.2, 0.8, "normal", 32, 0.1, "bf16", 2),
    "mlp_down": Workload("mlp-down-4096x11008-N64", 4096, 11008, 64, 10, 1.2, 0.8, "t4", 32, 0.1, "bf16", 3),
    "mlp_large": Workload("mlp-large-8192x28672-N32", 8192, 28672, 32, 8, 1.2, 0.8, "normal", 64, 0.1, "bf16", 4),
}
WORKLOAD_ORDER = ["tiny", "attn", "mlp_up", "mlp_down", "mlp_large"]


def workload(key: str | int) -> Workload:
    if isinstance(key, int):
        key = WORKLOAD_ORDER[key]
    return WORKLOADS[key]


# ---------------------------------------------------------------- primitives

def power_law_spectrum(dim: int, p: float) -> np.ndarray:
    """Eigenvalues c * k^-p, k = 1..dim, scaled to sum to dim."""
    lam = np.arange(1, dim + 1, dtype=np.float64) ** (-float(p))
    return lam * (dim / lam.sum())


def haar_orthogonal(dim: int, rng: np.random.Generator) -> np.ndarray:
    """Haar-distributed orthogonal matrix (QR of a Gaussian, sign-fixed)."""
    X = rng.standard_normal((dim, dim))
    Q, R = np.linalg.qr(X)
    return Q * np.sign(np.diag(R))[None, :]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _factor_roots(w: Workload, seed: int):
    rng = np.random.default_rng([seed, 0])
    QA = haar_orthogonal(w.n, rng)
    QB = haar_orthogonal(w.m, rng)
    lamA = power_law_spectrum(w.n, w.p_A)
    lamB = power_law_spectrum(w.m, w.p_B)
    SA = QA * np.sqrt(lamA)[None, :]
    SB = QB * np.sqrt(lamB)[None, :]
    return SA, SB, lamA, lamB


def _draw_z(w: Workload, rng: np.random.Generator) -> np.ndarray:
    if w.dist == "normal":
        return rng.standard_normal((w.m, w.n), dtype=np.float32)
    if w.dist.startswith("t"):
        nu = float(w.dist[1:])
        z = rng.standard_t(nu, size=(w.m, w.n)).astype(np.float32)
        return z * np.float32(np.sqrt((nu - 2.0) / nu))
    raise ValueError(f"unknown entry law {w.dist!r}")


def _draw_sample_randoms(w: Workload, seed: int, i: int):
    rng = np.random.default_rng([seed, 1, i])
    Z = _draw_z(w, rng)
    if w.rank > 0:
        U = rng.standard_normal((w.m, w.rank), dtype=np.float32)
        V = rng.standard_normal((w.n, w.rank), dtype=np.float32)
    else:
        U = V = None
    return Z, U, V


def _sigma_p(w: Workload, lamA, lamB) -> float:
    if w.rank == 0:
        return 0.0
    return float(np.sqrt(w.rho * lamA.sum() * lamB.sum() / (w.m * w.n * w.rank)))


@dataclass
class Draw:
    workload: Workload
    G: object            # numpy (N, m, n) uint16 bf16 bits / float32, or a torch tensor
    A_true: np.ndarray   # n x n fp64
    B_true: np.ndarray   # m x m fp64
    seed: int


def generate(w: Workload, seed: int | None = None, *, samples=None,
             with_truth: bool = True, threads: int | None = None) -> Draw:
    """Draw the workload on the CPU (numpy, fp64 products).

    ``samples`` selects a subset of sample indices (default: all N).
    Returns G as float32 for f32 workloads and as uint16 bf16 bits for
    bf16 workloads, shaped (len(samples), m, n).
    """
    seed = w.seed if seed is None else int(seed)
    idx = list(range(w.N)) if samples is None else list(samples)
    SA, SB, lamA, lamB = _factor_roots(w, seed)
    sp = _sigma_p(w, lamA, lamB)
    out_dtype = np.uint16 if w.dtype == "bf16" else np.float32
    G = np.empty((len(idx), w.m, w.n), dtype=out_dtype)

    def one(k):
        Z, U, V = _draw_sample_randoms(w, seed, idx[k])
        X = SB @ Z.astype(np.float64) @ SA.T
        if U is not None:
            X += sp * (U.astype(np.float64) @ V.astype(np.float64).T)
        X32 = X.astype(np.float32)
        G[k] = f32_to_bf16_bits(X32) if w.dtype == "bf16" else X32

    nthreads = threads or min(8, os.cpu_count() or 1)
    if len(idx) > 1 and nthreads > 1:
        with ThreadPoolExecutor(nthreads) as ex:
            list(ex.map(one, range(len(idx))))
    else:
        for k in range(len(idx)):
            one(k)
    A_true = SA @ SA.T if with_truth else None
    B_true = SB @ SB.T if with_truth else None
    return Draw(w, G, A_true, B_true, seed)


def generate_device(w: Workload, seed: int | None = None, *, device="cuda",
                    samples=None, threads: int = 16):
    """Draw the workload straight into device memory (torch, fp64 products).

    The random numbers are the same numpy streams as :func:`generate`; the
    products run in fp64 on the device, so the stored bits agree with the
    CPU draw except where an fp64 rounding difference crosses a bf16
    rounding boundary (vanishingly rare).  Returns a contiguous torch tensor
    (N, m, n) of dtype bfloat16 or float32.
    """
    import torch

    seed = w.seed if seed is None else int(seed)
    idx = list(range(w.N)) if samples is None else list(samples)
    rng = np.random.default_rng([seed, 0])
    dev = torch.device(device)
    # Factor roots: Haar Q from a device QR of the same Gaussian draws.
    XA = torch.from_numpy(rng.standard_normal((w.n, w.n))).to(dev)
    XB = torch.from_numpy(rng.standard_normal((w.m, w.m))).to(dev)

    def haar_dev(X):
        Q, R = torch.linalg.qr(X)
        return Q * torch.sign(torch.diagonal(R))[None, :]

    lamA = power_law_spectrum(w.n, w.p_A)
    lamB = power_law_spectrum(w.m, w.p_B)
    SA = haar_dev(XA) * torch.from_numpy(np.sqrt(lamA)).to(dev)[None, :]
    del XA
    SB = haar_dev(XB) * torch.from_numpy(np.sqrt(lamB)).to(dev)[None, :]
    del XB
    SAt = SA.T.contiguous()
    sp = _sigma_p(w, lamA, lamB)
    tdtype = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    G = torch.empty((len(idx), w.m, w.n), dtype=tdtype, device=dev)

    nthr = max(1, threads)
    with ThreadPoolExecutor(nthr) as ex:
        # at most 2 * threads draws in flight: bounded host memory on large layers
        futs = {}
        for k in range(min(len(idx), 2 * nthr)):
            futs[k] = ex.submit(_draw_sample_randoms, w, seed, idx[k])
        for k in range(len(idx)):
            Z, U, V = futs.pop(k).result()
            if k + 2 * nthr < len(idx):
                futs[k + 2 * nthr] = ex.submit(_draw_sample_randoms, w, seed, idx[k + 2 * nthr])
            Zd = torch.from_numpy(Z).to(dev, non_blocking=False).double()
            X = SB @ Zd @ SAt
            del Zd
            if U is not None:
                X += sp * (torch.from_numpy(U).to(dev).double()
                           @ torch.from_numpy(V).to(dev).double().T)
            G[k] = X.float().to(tdtype)
            del X
    return G
