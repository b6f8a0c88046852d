"""Write the expected flip-flop factors of the full-size layer workloads.

Calls only ``oracle`` (the fp64 flip-flop of Section 5, Appendix B order:
B first from A = I, one iteration = one B and one A update, tr(A) = n after
each) and ``synth`` (the seeded inputs).  For every workload it stores, in
``tests/golden/fullsize/<key>.npz``:

* the sha256 of every sample's bf16 bits and of the fixed-point basis, so a
  GPU run can prove it regenerated the same inputs;
* after iteration 1 and after the workload's iteration count: the diagonals
  and a seeded uniform sample of rows of A and B (fp32), the squared
  Frobenius norms, traces and log-determinants of both factors (fp64).

The attention layer and the 4096 x 11008 layer run at their full N (128 and
64).  The two other MLP layers run the full m x n with the first N_p samples
(48 of 128 for the 11008 x 4096 layer, 8 of 32 for the 28672-wide one; each
above the smallest N_p with N_p m >= 2 n and N_p n >= 2 m, which is 6 and 7,
so both factors are well determined): the fp64 oracle at their full N would
take 5 and 7 hours on 8 cores.

Usage: python tests/golden/make_fullsize_expected.py [attn] [mlp_up[:N]] [mlp_down[:N]] [mlp_large[:N]]
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

import numpy as np
import scipy.linalg as sla

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth   # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "fullsize")
PARITY_N = {"attn": 128, "mlp_up": 48, "mlp_down": 64, "mlp_large": 8}
ROWS = 32


def oracle_digest() -> str:
    h = hashlib.sha256()
    for f in sorted(os.listdir(os.path.join(ROOT, "oracle"))):
        if f.endswith(".py"):
            with open(os.path.join(ROOT, "oracle", f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()


def summary(A, B, rowsA, rowsB):
    lA = sla.cho_factor(A, lower=True)[0]
    lB = sla.cho_factor(B, lower=True)[0]
    return {
        "A_rows": A[rowsA].astype(np.float32), "B_rows": B[rowsB].astype(np.float32),
        "A_diag": np.diag(A).copy(), "B_diag": np.diag(B).copy(),
        "stats": np.array([np.sum(A * A), np.sum(B * B), np.trace(A), np.trace(B),
                           2.0 * np.sum(np.log(np.diag(lA))), 2.0 * np.sum(np.log(np.diag(lB)))]),
    }


def run(key: str, N: int | None = None) -> str:
    w = synth.workload(key).scaled(N=N or PARITY_N[key])
    t0 = time.time()
    d = synth.generate(w)
    digests = synth.sample_digests(d.G)
    print(f"[{key}] drew {w.N} samples of {w.m} x {w.n} in {time.time() - t0:.1f} s", flush=True)
    rng = np.random.default_rng([w.seed, 7])
    rowsA = np.sort(rng.choice(w.n, size=min(ROWS, w.n), replace=False))
    rowsB = np.sort(rng.choice(w.m, size=min(ROWS, w.m), replace=False))
    t1 = time.time()
    r1 = oracle.flipflop(d.G, 1)
    t_first = time.time() - t1
    print(f"[{key}] iteration 1 in {t_first:.0f} s", flush=True)
    s1 = summary(r1.A, r1.B, rowsA, rowsB)
    rk = oracle.flipflop(d.G, w.iters - 1, A0=r1.A) if w.iters > 1 else r1
    t_all = time.time() - t1
    print(f"[{key}] {w.iters} iterations in {t_all:.0f} s", flush=True)
    sk = summary(rk.A, rk.B, rowsA, rowsB)
    meta = {
        "workload": w.name, "key": key, "m": w.m, "n": w.n, "N": w.N, "N_full": synth.workload(key).N,
        "iters": w.iters, "order": "B_FIRST", "damping": 0.0, "seed": w.seed,
        "sample_sha256": digests,
        "samples_sha256": hashlib.sha256("".join(digests).encode()).hexdigest(),
        "basis_sha256": synth.basis_digest(w),
        "oracle_sha256": oracle_digest(),
        "oracle_seconds": round(t_all, 1), "cpu_count": os.cpu_count(),
    }
    os.makedirs(OUT, exist_ok=True)
    path = os.path.join(OUT, f"{key}.npz")
    arrays = {"rowsA": rowsA, "rowsB": rowsB, "meta": np.array(json.dumps(meta))}
    for tag, s in (("it1", s1), ("final", sk)):
        for name, v in s.items():
            arrays[f"{tag}_{name}"] = v
    tmp = path + ".tmp.npz"
    np.savez(tmp, **arrays)
    os.replace(tmp, path)
    print(f"[{key}] wrote {path}", flush=True)
    return path


if __name__ == "__main__":
    # key or key:N (N samples instead of the default above)
    for arg in sys.argv[1:] or list(PARITY_N):
        k, _, n = arg.partition(":")
        run(k, int(n) if n else None)
