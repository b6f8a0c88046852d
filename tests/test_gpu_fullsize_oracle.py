"""Full-size parity of the layer workloads against the fp64 oracle.

(1) Iterations.  ``tests/golden/make_fullsize_expected.py`` ran the oracle
    (Section 5 flip-flop, Appendix B order, tr(A) = n) on the CPU and stored,
    keyed by the sha256 of every sample's bf16 bits, a seeded uniform sample
    of rows and the diagonals of A and B after iteration 1 and after the
    workload's iteration count, with their exact squared Frobenius norms.
    Here the samples are regenerated on the device (the fixed-point
    generator is exact, so the bits must match: checked first), the GPU runs
    the same iterations in the benchmark's configuration, and the relative
    Frobenius error of the normalised A (x) B is estimated from the rows:
    ||A(x)B - A*(x)B*||^2 = ||dA||^2 ||B||^2 + ||A*||^2 ||dB||^2 + 2 <dA,A*> <B,dB>,
    with ||B||^2 exact (the GPU's own factor), ||A*||^2 exact (stored) and
    the terms in dA, dB summed over the sampled rows and scaled by dim / rows
    (unbiased for a uniform row sample).  The attention layer runs at its
    full N; the MLP layers with the first N_p samples (see the script).
(2) Half steps at the full N.  With seeded dense SPD fixed factors (A0 of
    n x n, B0 of m x m), one B and one A half step through ff_half_step:
    the full-width factorisations (4096, 11008, 8192, 28672), the whitening
    and the symmetric product at the real sample count, against the oracle's
    rows computed one sample at a time from the host copy, unscaled.
"""
import json
import os

import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = os.path.join(HERE, "golden", "fullsize")
KEYS = ["attn", "mlp_up", "mlp_down", "mlp_large"]
TOL = 5e-3


def _free():
    import gc
    import torch
    gc.collect()
    torch.cuda.empty_cache()


def _expected(key):
    path = os.path.join(GOLDEN, f"{key}.npz")
    if not os.path.exists(path):
        pytest.skip(f"{path} not written yet (tests/golden/make_fullsize_expected.py {key})")
    z = np.load(path, allow_pickle=False)
    return {k: z[k] for k in z.files}, json.loads(str(z["meta"]))


def estimated_error(A, B, exp, tag, rowsA, rowsB):
    """Row-sampled estimate of the relative Frobenius error of A (x) B
    against the stored oracle factors, plus the sampled rows' and the
    diagonals' own relative errors."""
    n, m = A.shape[0], B.shape[0]
    As, Bs = exp[f"{tag}_A_rows"].astype(np.float64), exp[f"{tag}_B_rows"].astype(np.float64)
    nA2, nB2 = exp[f"{tag}_stats"][0], exp[f"{tag}_stats"][1]
    dA = A[rowsA] - As
    dB = B[rowsB] - Bs
    sA, sB = n / len(rowsA), m / len(rowsB)
    dA2 = sA * np.sum(dA * dA)
    dAA = sA * np.sum(dA * As)
    dB2 = sB * np.sum(dB * dB)
    BdB = sB * np.sum((Bs + dB) * dB)
    B2 = float(np.sum(B * B))
    sq = dA2 * B2 + nA2 * dB2 + 2.0 * dAA * BdB
    est = float(np.sqrt(max(sq, 0.0) / (nA2 * nB2)))
    rowsA_err = float(np.linalg.norm(dA) / np.linalg.norm(As))
    rowsB_err = float(np.linalg.norm(dB) / np.linalg.norm(Bs))
    dgA = np.diag(A) - exp[f"{tag}_A_diag"]
    dgB = np.diag(B) - exp[f"{tag}_B_diag"]
    diag_err = max(float(np.linalg.norm(dgA) / np.linalg.norm(exp[f"{tag}_A_diag"])),
                   float(np.linalg.norm(dgB) / np.linalg.norm(exp[f"{tag}_B_diag"])))
    return est, rowsA_err, rowsB_err, diag_err


@pytest.mark.parametrize("key", KEYS)
def test_iterations_match_the_oracle(gpu, key):
    import torch
    import paper_2609_14706_amd as ffe
    exp, meta = _expected(key)
    w = synth.workload(key).scaled(N=meta["N"])
    assert (w.m, w.n, w.iters, w.seed) == (meta["m"], meta["n"], meta["iters"], meta["seed"])
    assert synth.basis_digest(w) == meta["basis_sha256"], "fixed-point basis differs"
    print(f"[{key}] {w.m} x {w.n}, N = {w.N}: generating on the device", flush=True)
    G = synth.generate_device(w, device=gpu)
    dig = synth.sample_digests(G)
    bad = [i for i, (a, b) in enumerate(zip(dig, meta["sample_sha256"])) if a != b]
    assert not bad, f"samples {bad[:8]} differ from the ones the oracle ran on"
    print(f"[{key}] all {w.N} samples bitwise identical to the oracle's inputs", flush=True)
    rowsA, rowsB = exp["rowsA"], exp["rowsB"]
    f = ffe.FlipFlop(G)
    f.iterate(1)
    A1, B1 = (X.double().cpu().numpy() for X in f.factors())
    f.iterate(w.iters - 1)
    A, B = (X.double().cpu().numpy() for X in f.factors())
    sA, sB, pA, pB = f.whiten_split_state()
    f.close()
    print(f"[{key}] automatic whitening split: s(A) {sA:.2f}, s(B) {sB:.2f}, passes {pA}", flush=True)
    del G
    _free()
    out = {}
    for tag, (AA, BB) in (("it1", (A1, B1)), ("final", (A, B))):
        est, ea, eb, ed = estimated_error(AA, BB, exp, tag, rowsA, rowsB)
        out[tag] = est
        print(f"[{key}] {tag}: estimated rel. Frobenius error of A(x)B {est:.3e} "
              f"(sampled rows of A {ea:.3e}, of B {eb:.3e}; diagonals {ed:.3e})", flush=True)
        assert est < TOL and ea < TOL and eb < TOL and ed < TOL
    assert abs(np.trace(A) - w.n) < 1e-6 * w.n


def _progress(tag, N):
    def cb(i):
        if i % max(1, N // 8) == 0 or i == N - 1:
            print(f"    {tag}: sample {i + 1} of {N}", flush=True)
    return cb


@pytest.mark.parametrize("key", KEYS)
def test_half_steps_at_full_n(gpu, key):
    import torch
    import paper_2609_14706_amd as ffe
    w = synth.workload(key)
    print(f"[{key}] {w.m} x {w.n}, N = {w.N}: generating on the device", flush=True)
    G = synth.generate_device(w, device=gpu)
    A0 = synth.spd_start(w.n, w.seed)
    B0 = synth.spd_start(w.m, w.seed + 1)
    f = ffe.FlipFlop(G)
    Bh = f.half_step("B", torch.from_numpy(A0))
    Ah = f.half_step("A", torch.from_numpy(B0))
    f.close()
    rng = np.random.default_rng([w.seed, 9])
    rowsB = np.sort(rng.choice(w.m, size=24, replace=False))
    rowsA = np.sort(rng.choice(w.n, size=24, replace=False))
    gotB = Bh[torch.from_numpy(rowsB).to(gpu)].double().cpu().numpy()
    gotA = Ah[torch.from_numpy(rowsA).to(gpu)].double().cpu().numpy()
    del Bh, Ah
    Gh = G.view(torch.int16).cpu().numpy().view(np.uint16)
    del G
    _free()
    print(f"[{key}] oracle: rows of the B half step (Cholesky of the {w.n} x {w.n} A0)", flush=True)
    refB = oracle.half_step_B_rows(Gh, A0.astype(np.float64), rowsB, progress=_progress("B", w.N))
    print(f"[{key}] oracle: rows of the A half step (Cholesky of the {w.m} x {w.m} B0)", flush=True)
    refA = oracle.half_step_A_rows(Gh, B0.astype(np.float64), rowsA, progress=_progress("A", w.N))
    del Gh
    eB = np.linalg.norm(gotB - refB, axis=1) / np.linalg.norm(refB, axis=1)
    eA = np.linalg.norm(gotA - refA, axis=1) / np.linalg.norm(refA, axis=1)
    fB = float(np.linalg.norm(gotB - refB) / np.linalg.norm(refB))
    fA = float(np.linalg.norm(gotA - refA) / np.linalg.norm(refA))
    print(f"[{key}] half steps at N = {w.N}, unscaled: B rows {fB:.3e} (worst row {eB.max():.3e}), "
          f"A rows {fA:.3e} (worst row {eA.max():.3e})", flush=True)
    assert fB < TOL and fA < TOL
    assert eB.max() < 2 * TOL and eA.max() < 2 * TOL
