"""Seeded inputs of the WaterKron quantiser: weights W (m x n) and Kronecker
factors A (n x n), B (m x m).

The paper's rate-distortion analysis (Sections 2.4 and 3) takes W_ij iid
Gaussian and positive definite factors; its experiments quantise LLM layers
with factors estimated from calibration data (Appendix B), which are not
available here.  These draws stand in for them:

* W_ij ~ N(0, sigma_W^2), drawn from ``default_rng([seed, 3])``;
* A = Q_A diag(lambda_A) Q_A^T with the power-law spectrum of
  ``generator.power_law_spectrum`` (mean 1) plus ``floor`` (so that
  cond(A) <= 1 + max(lambda) / floor), Q_A Haar from
  ``default_rng([seed, 4])``;
  B alike from ``default_rng([seed, 5])``;
* everything stored as fp32 (the oracle reads the same fp32 values).

Only random numbers and their products live here: no step of the method.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np

from .generator import BASE_SEED, haar_orthogonal, power_law_spectrum


@dataclass(frozen=True)
class QuantWorkload:
    name: str
    m: int          # output channels (rows of W), B is m x m
    n: int          # input channels (columns of W), A is n x n
    p_A: float
    p_B: float
    floor: float    # spectral floor, relative to the mean eigenvalue
    sigma_W: float
    gamma: float    # step parameter of the waterfilling scales
    index: int      # seed offset

    @property
    def seed(self) -> int:
        return BASE_SEED + 200 + self.index

    @property
    def flop(self) -> float:
        """Products that spread the rounding errors: (L~B E) over the rows,
        E L~A^T over the columns, both triangular."""
        return float(self.m) ** 2 * self.n + float(self.m) * self.n ** 2

    def scaled(self, **kw) -> "QuantWorkload":
        return replace(self, **kw)


QUANT_WORKLOADS = {
    # one ragged tile of each kind: 96 = 64 + 32 rows, 80 = 64 + 16 columns
    "quant_small": QuantWorkload("quant-small-96x80", 96, 80, 1.0, 0.8, 0.2, 1.0, 0.05, 0),
    # 4 x 4 tiles (ragged): every kind of forward push between tiles
    "quant_multi": QuantWorkload("quant-multi-200x200", 200, 200, 1.2, 0.8, 0.05, 1.0, 0.05, 1),
    # an attention projection of the paper's calibration setting (4096 x 4096)
    "quant_attn": QuantWorkload("quant-attn-4096x4096", 4096, 4096, 1.2, 0.8, 0.01, 1.0, 0.05, 2),
}


def quant_workload(key: str) -> QuantWorkload:
    return QUANT_WORKLOADS[key]


@dataclass
class QuantDraw:
    workload: QuantWorkload
    W: np.ndarray   # (m, n) float32
    A: np.ndarray   # (n, n) float32, symmetric
    B: np.ndarray   # (m, m) float32, symmetric


def _factor(dim: int, p: float, floor: float, rng) -> np.ndarray:
    lam = power_law_spectrum(dim, p)
    lam = lam + floor * lam.mean()
    Q = haar_orthogonal(dim, rng)
    F = (Q * lam[None, :]) @ Q.T
    F = 0.5 * (F + F.T)
    return F.astype(np.float32)


def generate_quant(w: QuantWorkload, seed: int | None = None) -> QuantDraw:
    seed = w.seed if seed is None else int(seed)
    W = (w.sigma_W * np.random.default_rng([seed, 3]).standard_normal((w.m, w.n))).astype(np.float32)
    A = _factor(w.n, w.p_A, w.floor, np.random.default_rng([seed, 4]))
    B = _factor(w.m, w.p_B, w.floor, np.random.default_rng([seed, 5]))
    return QuantDraw(w, W, A, B)
