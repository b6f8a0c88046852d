"""Workload table and seeded generators (CPU numpy, or torch on a device).

Recipe (stated once, used by every test and by the benchmark):

* spectra: ``lambda_k = c * k**(-p)``, k = 1..dim, with c chosen so that the
  trace equals ``dim`` (mean eigenvalue 1);
* samples: ``G_i = S_B Z_i S_A^T (+ sigma_p U_i V_i^T)`` with
  ``S = Q diag(sqrt(lambda))``, Z_i iid N(0,1) (or Student-t(nu) scaled to
  unit variance) and U_i (m x r), V_i (n x r) iid N(0,1);
  ``sigma_p**2 = rho * tr(A) tr(B) / (m n r)`` makes the expected energy of
  the low-rank term ``rho`` times that of the Kronecker term;
* eigenvectors Q, by the workload's ``basis``:

  - ``"haar"``: a dense Haar orthogonal matrix, the QR factorisation of a
    Gaussian matrix with the sign of diag(R) folded into Q; the products
    run in fp64 BLAS, so the last bits of G depend on the machine;
  - ``"kron"``: ``Q = P1 (Qa (x) Qb) P2 (Qc (x) Qd)`` with small Haar
    factors (dim = a b, a the largest divisor <= sqrt(dim)) and uniformly
    random permutations P1, P2 (one dense Haar factor when dim has no
    useful split).  Everything is computed in fixed point: the factors,
    the draws and the square roots of the eigenvalues are rounded to
    integers at fixed power-of-two scales, every product is a sum of
    integers whose magnitudes are checked to stay below 2**52 (so any
    summation order, on any CPU or GPU, gives the same exact result) and
    every rescaling is a power of two followed by round-half-even.  The
    bits of G are therefore the same on every machine, which is what lets
    expected values computed on one machine be checked on another.  The
    truth is ``A = Q diag(lambda_q) Q^T`` with ``sqrt(lambda_q)`` the
    rounded square roots;

* storage: the fp64 sample is rounded to fp32 (RNE) and, for bf16
  workloads, to bf16 (RNE) and kept as uint16 bit patterns;
* seeds: the factors come from ``default_rng([seed, 0])``; sample i draws
  Z_i, then U_i, then V_i from ``default_rng([seed, 1, i])``, so any subset
  of samples can be drawn on its own and in parallel.
"""
from __future__ import annotations

import hashlib
import math
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
    basis: str = "haar"  # eigenvector construction: "haar" or "kron" (exact fixed point)

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
    "attn": Workload("attn-4096x4096-N128", 4096, 4096, 128, 10, 1.2, 0.8, "normal", 32, 0.1, "bf16", 1,
                     "kron"),
    "mlp_up": Workload("mlp-up-11008x4096-N128", 11008, 4096, 128, 10, 1.2, 0.8, "normal", 32, 0.1, "bf16",
                       2, "kron"),
    "mlp_down": Workload("mlp-down-4096x11008-N64", 4096, 11008, 64, 10, 1.2, 0.8, "t4", 32, 0.1, "bf16",
                         3, "kron"),
    "mlp_large": Workload("mlp-large-8192x28672-N32", 8192, 28672, 32, 8, 1.2, 0.8, "normal", 64, 0.1,
                          "bf16", 4, "kron"),
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


# ----------------------------------------------- exact fixed-point basis ("kron")

_QS = 15          # orthogonal factors: integers at scale 2**15
_ZS = 12          # Z, U, V: integers at scale 2**12
_LS = 10          # square roots of the eigenvalues: integers at scale 2**10
_LIMIT = 2.0 ** 52  # bound on every partial sum of a product of integers


def _split(dim: int):
    """dim = a b with a the largest divisor <= sqrt(dim); (1, dim) if none > 1."""
    a = 1
    for c in range(int(math.isqrt(dim)), 1, -1):
        if dim % c == 0:
            a = c
            break
    return a, dim // a


@dataclass
class KronBasis:
    """The eigenvector map of one side: x -> P1 K1 P2 K2 x, K = Qa (x) Qb
    acting on x viewed row-major as an a x b matrix (K x = Qa X Qb^T), or
    one dense factor (a = 1).  Factors are integer-valued fp64 at 2**_QS."""
    dim: int
    a: int
    b: int
    stages: list      # [(Qa, Qb) or (None, Qd)] applied last-to-first
    perms: list       # permutation index arrays, one per stage (applied after it)
    root: np.ndarray  # integer-valued fp64 sqrt(lambda) at 2**_LS

    def digest(self) -> str:
        h = hashlib.sha256()
        for Qa, Qb in self.stages:
            for Q in (Qa, Qb):
                if Q is not None:
                    h.update(np.ascontiguousarray(Q).tobytes())
        for p in self.perms:
            h.update(np.ascontiguousarray(p, dtype=np.int64).tobytes())
        h.update(np.ascontiguousarray(self.root).tobytes())
        return h.hexdigest()


def _kron_basis(dim: int, p: float, rng: np.random.Generator) -> KronBasis:
    def q(d):
        return np.rint(haar_orthogonal(d, rng) * 2.0 ** _QS)

    a, b = _split(dim)
    if a == 1:
        if dim > 4096:
            raise ValueError(f"dimension {dim} has no factor split for the fixed-point basis")
        stages = [(None, q(dim))]
        perms = [rng.permutation(dim)]
    else:
        Qa1, Qb1, Qa2, Qb2 = q(a), q(b), q(a), q(b)
        stages = [(Qa1, Qb1), (Qa2, Qb2)]
        perms = [rng.permutation(dim), rng.permutation(dim)]
    root = np.rint(np.sqrt(power_law_spectrum(dim, p)) * 2.0 ** _LS)
    return KronBasis(dim, a, b, stages, perms, root)


def _kron_bases(w: Workload, seed: int):
    rng = np.random.default_rng([seed, 0])
    return _kron_basis(w.n, w.p_A, rng), _kron_basis(w.m, w.p_B, rng)


class _NumpyOps:
    def __init__(self):
        self.xp = np

    def const(self, a):
        return np.asarray(a, dtype=np.float64)

    def index(self, a):
        return np.asarray(a, dtype=np.int64)

    def f64(self, a):
        return np.asarray(a, dtype=np.float64)

    def rint(self, x):
        return np.rint(x)

    def absmax(self, x):
        return float(np.max(np.abs(x))) if x.size else 0.0

    def take(self, x, idx, axis):
        return np.take(x, idx, axis=axis)


class _TorchOps:
    def __init__(self, device):
        import torch
        self.torch = torch
        self.device = device

    def const(self, a):
        return self.torch.as_tensor(np.asarray(a, dtype=np.float64), device=self.device)

    def index(self, a):
        return self.torch.as_tensor(np.asarray(a, dtype=np.int64), device=self.device)

    def f64(self, a):
        return self.torch.as_tensor(a).to(self.device).double()

    def rint(self, x):
        return self.torch.round(x)   # round half to even, like numpy's rint

    def absmax(self, x):
        return float(x.abs().max()) if x.numel() else 0.0

    def take(self, x, idx, axis):
        return self.torch.index_select(x, axis, idx)


def _rowsum(Q) -> float:
    return float(np.max(np.sum(np.abs(Q), axis=1)))


def _fit(ops, X, e, rowsum):
    """Shift X (value X * 2**-e) right until |X| * rowsum < 2**52.

    The shift depends only on max|X|, which is exact on every backend."""
    mx = ops.absmax(X)
    s = 0
    while mx * 2.0 ** -s * rowsum >= _LIMIT * 0.5:
        s += 1
    if s:
        X = ops.rint(X * 2.0 ** -s)
        e -= s
    return X, e


def _contract_last(ops, X, Q, Qc, e):
    """X (..., d) -> X Q^T along the last axis, exact; value scale kept."""
    X, e = _fit(ops, X, e, _rowsum(Q))
    X = ops.rint((X @ Qc.T) * 2.0 ** -_QS)
    return X, e


def _apply_basis(ops, X, e, basis: KronBasis, consts, axis: int):
    """Apply the map of `basis` to every vector of X along `axis` (0 or 1).

    Exact: every product is a sum of integers below 2**52 and every
    rescaling a power of two followed by round-half-even."""
    d = basis.dim
    for (Qa, Qb), (Qac, Qbc), perm in zip(reversed(basis.stages), reversed(consts["Q"]),
                                           reversed(consts["perm"])):
        if axis == 1:
            R = X.shape[0]
            if Qa is None:
                X, e = _contract_last(ops, X, Qb, Qbc, e)
            else:
                X3 = X.reshape(R, basis.a, basis.b)
                X3, e = _contract_last(ops, X3, Qb, Qbc, e)
                X3, e = _fit(ops, X3, e, _rowsum(Qa))
                X3 = ops.rint((Qac @ X3) * 2.0 ** -_QS)
                X = X3.reshape(R, d)
        else:
            C = X.shape[1]
            if Qa is None:
                X, e = _fit(ops, X, e, _rowsum(Qb))
                X = ops.rint((Qbc @ X) * 2.0 ** -_QS)
            else:
                X3 = X.reshape(basis.a, basis.b, C)
                X3, e = _fit(ops, X3, e, _rowsum(Qb))
                X3 = ops.rint((Qbc @ X3) * 2.0 ** -_QS)
                X3, e = _fit(ops, X3, e, _rowsum(Qa))
                X2 = ops.rint((Qac @ X3.reshape(basis.a, basis.b * C)) * 2.0 ** -_QS)
                X = X2.reshape(d, C)
        X = ops.take(X, perm, axis)
    return X, e


def _basis_consts(ops, basis: KronBasis):
    return {"Q": [(None if Qa is None else ops.const(Qa), ops.const(Qb)) for Qa, Qb in basis.stages],
            "perm": [ops.index(p) for p in basis.perms]}


def _exact_sample(ops, w: Workload, bA: KronBasis, bB: KronBasis, cA, cB, rootA, rootB, sp,
                  Z, U, V):
    """One sample G (fp64 on the ops' backend) of a "kron" workload."""
    Zq = ops.rint(ops.f64(Z) * 2.0 ** _ZS)
    mz = ops.absmax(Zq)
    if mz * float(bB.root.max()) * float(bA.root.max()) >= _LIMIT:
        raise OverflowError("sample draw too large for the exact fixed-point product")
    X = (Zq * rootB[:, None]) * rootA[None, :]           # exact integer products
    del Zq
    e = _ZS + 2 * _LS
    X, e = _apply_basis(ops, X, e, bA, cA, axis=1)        # rows:    M Q_A^T
    X, e = _apply_basis(ops, X, e, bB, cB, axis=0)        # columns: Q_B M
    X = X * 2.0 ** -e
    if U is not None:
        Uq = ops.rint(ops.f64(U) * 2.0 ** _ZS)
        Vq = ops.rint(ops.f64(V) * 2.0 ** _ZS)
        if ops.absmax(Uq) * ops.absmax(Vq) * U.shape[1] >= _LIMIT:
            raise OverflowError("low-rank draw too large for the exact fixed-point product")
        X = X + (Uq @ Vq.T) * (sp * 2.0 ** (-2 * _ZS))
    return X


def _kron_truth(basis: KronBasis) -> np.ndarray:
    """Q diag(lambda_q) Q^T of a "kron" basis, Q its map without the roundings."""
    d = basis.dim
    Q = np.eye(d)
    for (Qa, Qb), perm in zip(reversed(basis.stages), reversed(basis.perms)):
        if Qa is None:
            Q = (Qb * 2.0 ** -_QS) @ Q
        else:
            X3 = Q.reshape(basis.a, basis.b, d)
            X3 = (Qb * 2.0 ** -_QS) @ X3
            Q = ((Qa * 2.0 ** -_QS) @ X3.reshape(basis.a, basis.b * d)).reshape(d, d)
        Q = Q[perm, :]
    lam = (basis.root * 2.0 ** -_LS) ** 2
    return (Q * lam[None, :]) @ Q.T


# ------------------------------------------------------------------ draws

def _factor_roots(w: Workload, seed: int):
    rng = np.random.default_rng([seed, 0])
    QA = haar_orthogonal(w.n, rng)
    QB = haar_orthogonal(w.m, rng)
    lamA = power_law_spectrum(w.n, w.p_A)
    lamB = power_law_spectrum(w.m, w.p_B)
    SA = QA * np.sqrt(lamA)[None, :]
    SB = QB * np.sqrt(lamB)[None, :]
    return SA, SB, lamA, lamB


class Draw:
    """Samples of a workload and, on request, the true factors.

    ``A_true`` (n x n) and ``B_true`` (m x m) are computed when first read."""

    def __init__(self, workload: Workload, G, seed: int, truth):
        self.workload = workload
        self.G = G                 # numpy (N, m, n) uint16 bf16 bits / float32, or a torch tensor
        self.seed = seed
        self._truth = truth        # callable -> (A_true, B_true)
        self._cache = None

    def _get(self):
        if self._cache is None:
            self._cache = self._truth()
        return self._cache

    @property
    def A_true(self) -> np.ndarray:
        return self._get()[0]

    @property
    def B_true(self) -> np.ndarray:
        return self._get()[1]


def _spectra(w: Workload):
    return power_law_spectrum(w.n, w.p_A), power_law_spectrum(w.m, w.p_B)


def _kron_sigma_p(w: Workload, bA: KronBasis, bB: KronBasis) -> float:
    lamA = (bA.root * 2.0 ** -_LS) ** 2
    lamB = (bB.root * 2.0 ** -_LS) ** 2
    return _sigma_p(w, lamA, lamB)


def basis_digest(w: Workload, seed: int | None = None) -> str:
    """sha256 of the fixed-point basis of a "kron" workload (factors,
    permutations and square roots of both sides)."""
    seed = w.seed if seed is None else int(seed)
    bA, bB = _kron_bases(w, seed)
    return hashlib.sha256((bA.digest() + bB.digest()).encode()).hexdigest()


def generate(w: Workload, seed: int | None = None, *, samples=None,
             with_truth: bool = True, threads: int | None = None) -> Draw:
    """Draw the workload on the CPU (numpy).

    ``samples`` selects a subset of sample indices (default: all N).
    Returns G as float32 for f32 workloads and as uint16 bf16 bits for
    bf16 workloads, shaped (len(samples), m, n).  ``with_truth`` is kept
    for compatibility: the true factors are computed lazily when read.
    """
    seed = w.seed if seed is None else int(seed)
    idx = list(range(w.N)) if samples is None else list(samples)
    out_dtype = np.uint16 if w.dtype == "bf16" else np.float32
    G = np.empty((len(idx), w.m, w.n), dtype=out_dtype)

    if w.basis == "kron":
        # torch on the CPU: its element-wise passes are vectorised and
        # threaded; every product is exact, so the bits do not depend on the
        # backend (numpy gives the same result, more slowly).
        import torch
        bA, bB = _kron_bases(w, seed)
        sp = _kron_sigma_p(w, bA, bB)
        ops = _TorchOps(torch.device("cpu"))
        cA, cB = _basis_consts(ops, bA), _basis_consts(ops, bB)
        rootA, rootB = ops.const(bA.root), ops.const(bB.root)
        for k, i in enumerate(idx):
            Z, U, V = _draw_sample_randoms(w, seed, i)
            X32 = _exact_sample(ops, w, bA, bB, cA, cB, rootA, rootB, sp, Z, U, V).float()
            if w.dtype == "bf16":
                G[k] = X32.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
            else:
                G[k] = X32.numpy()
        return Draw(w, G, seed, lambda: (_kron_truth(bA), _kron_truth(bB)))

    if w.basis != "haar":
        raise ValueError(f"unknown basis {w.basis!r}")
    SA, SB, lamA, lamB = _factor_roots(w, seed)
    sp = _sigma_p(w, lamA, lamB)

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
    return Draw(w, G, seed, lambda: (SA @ SA.T, SB @ SB.T))


def generate_device(w: Workload, seed: int | None = None, *, device="cuda",
                    samples=None, threads: int = 16):
    """Draw the workload straight into device memory (torch).

    The random numbers are the same numpy streams as :func:`generate`.  For
    a "kron" workload every product is exact, so the stored bits are
    identical to the CPU draw.  For a "haar" workload the products run in
    fp64 on the device and agree with the CPU draw except where an fp64
    rounding difference crosses a bf16 rounding boundary (rare).  Returns a
    contiguous torch tensor (N, m, n) of dtype bfloat16 or float32.
    """
    import torch

    seed = w.seed if seed is None else int(seed)
    idx = list(range(w.N)) if samples is None else list(samples)
    dev = torch.device(device)
    tdtype = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    G = torch.empty((len(idx), w.m, w.n), dtype=tdtype, device=dev)

    if w.basis == "kron":
        bA, bB = _kron_bases(w, seed)
        sp = _kron_sigma_p(w, bA, bB)
        ops = _TorchOps(dev)
        cA, cB = _basis_consts(ops, bA), _basis_consts(ops, bB)
        rootA, rootB = ops.const(bA.root), ops.const(bB.root)

        def make(k, Z, U, V):
            X = _exact_sample(ops, w, bA, bB, cA, cB, rootA, rootB, sp, Z, U, V)
            G[k] = X.float().to(tdtype)
    else:
        rng = np.random.default_rng([seed, 0])
        XA = torch.from_numpy(rng.standard_normal((w.n, w.n))).to(dev)
        XB = torch.from_numpy(rng.standard_normal((w.m, w.m))).to(dev)

        def haar_dev(X):
            Q, R = torch.linalg.qr(X)
            return Q * torch.sign(torch.diagonal(R))[None, :]

        lamA, lamB = _spectra(w)
        SA = haar_dev(XA) * torch.from_numpy(np.sqrt(lamA)).to(dev)[None, :]
        del XA
        SB = haar_dev(XB) * torch.from_numpy(np.sqrt(lamB)).to(dev)[None, :]
        del XB
        SAt = SA.T.contiguous()
        sp = _sigma_p(w, lamA, lamB)

        def make(k, Z, U, V):
            Zd = torch.from_numpy(Z).to(dev).double()
            X = SB @ Zd @ SAt
            del Zd
            if U is not None:
                X += sp * (torch.from_numpy(U).to(dev).double()
                           @ torch.from_numpy(V).to(dev).double().T)
            G[k] = X.float().to(tdtype)

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
            make(k, Z, U, V)
    return G


def sample_digests(G) -> list:
    """sha256 of every sample's stored bits (numpy array or torch tensor)."""
    out = []
    for i in range(G.shape[0]):
        g = G[i]
        if hasattr(g, "detach"):
            import torch
            g = g.detach()
            if g.dtype == torch.bfloat16:
                g = g.view(torch.int16)
            g = g.cpu().numpy()
        out.append(hashlib.sha256(np.ascontiguousarray(g).tobytes()).hexdigest())
    return out


def spd_start(dim: int, seed: int, rank: int = 256, floor: float = 0.05) -> np.ndarray:
    """A seeded dense SPD matrix for start factors / fixed factors of half
    steps: ``floor * I + W W^T / rank`` with W (dim x rank) iid N(0,1),
    rounded to fp32 (returned as float32).  Its eigenvalues are ``floor``
    (dim - rank times) and about ``floor + dim / rank`` (rank times), so its
    condition number is about dim / (rank floor) (2.2e3 at dim = 28672)."""
    rng = np.random.default_rng([seed, 5, dim])
    r = min(rank, dim)
    W = rng.standard_normal((dim, r), dtype=np.float32).astype(np.float64)
    M = W @ W.T
    M *= 1.0 / r
    M[np.diag_indices(dim)] += floor
    return M.astype(np.float32)
