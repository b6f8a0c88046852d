"""The seeded input generator (CPU, no GPU needed).

The fixed-point ("kron") construction must give the same bits whatever
evaluates it: every product is a sum of integers below 2**52 and every
rescaling a power of two followed by round-half-even.  Here the plain numpy
evaluation and the torch evaluation (another BLAS, other kernels and
summation orders; the device generator runs the same torch code on the GPU)
must agree bit for bit, and the draws must follow the stated law."""
import numpy as np
import pytest

import oracle
import synth
from synth import generator as gen


def numpy_draw(w, samples):
    bA, bB = gen._kron_bases(w, w.seed)
    sp = gen._kron_sigma_p(w, bA, bB)
    ops = gen._NumpyOps()
    cA, cB = gen._basis_consts(ops, bA), gen._basis_consts(ops, bB)
    out = []
    for i in samples:
        Z, U, V = gen._draw_sample_randoms(w, w.seed, i)
        X = gen._exact_sample(ops, w, bA, bB, cA, cB, bA.root, bB.root, sp, Z, U, V)
        X32 = X.astype(np.float32)
        out.append(gen.f32_to_bf16_bits(X32) if w.dtype == "bf16" else X32)
    return np.stack(out)


@pytest.mark.parametrize("key,kw", [
    ("attn", dict(m=600, n=520, N=3)),          # two Kronecker stages per side
    ("mlp_down", dict(m=256, n=344, N=2)),      # Student-t entries
    ("attn", dict(m=37, n=100, N=2)),           # a prime side: one dense factor
    ("attn", dict(m=1, n=20, N=2)),             # a 1 x 1 side
    ("tiny", dict(m=48, n=80, N=2, basis="kron")),  # fp32 storage, no low-rank term
])
def test_fixed_point_generator_is_backend_independent(key, kw):
    w = synth.workload(key).scaled(**kw)
    d = synth.generate(w)                       # torch evaluation
    ref = numpy_draw(w, range(w.N))             # numpy evaluation
    assert synth.sample_digests(d.G) == synth.sample_digests(ref)
    sub = synth.generate(w, samples=[w.N - 1])  # any sample can be drawn alone
    assert synth.sample_digests(sub.G) == synth.sample_digests(d.G)[-1:]


def test_fixed_point_basis_digest_is_stable():
    w = synth.workload("attn").scaled(m=600, n=520)
    assert synth.basis_digest(w) == synth.basis_digest(w)
    assert synth.basis_digest(w) != synth.basis_digest(w, seed=w.seed + 1)


def test_fixed_point_truth_has_the_power_law_spectrum():
    w = synth.workload("attn").scaled(m=96, n=120, N=2)
    d = synth.generate(w)
    for T, dim, p in ((d.A_true, w.n, w.p_A), (d.B_true, w.m, w.p_B)):
        lam = np.linalg.eigvalsh(T)[::-1]
        np.testing.assert_allclose(lam, synth.power_law_spectrum(dim, p), rtol=2e-3, atol=2e-3)


def test_fixed_point_draws_follow_the_matrix_normal_law():
    """Without the low-rank term the flip-flop estimate from the draws
    approaches the true factors at the N^-1/2 rate (the error roughly halves
    when N grows four times), as for the dense Haar construction."""
    errs = []
    for N in (100, 400, 1600):
        w = synth.workload("attn").scaled(m=12, n=10, N=N, rank=0, rho=0.0, dtype="f32")
        d = synth.generate(w)
        r = oracle.flipflop(d.G, 15)
        c = np.trace(d.A_true) / w.n
        errs.append(oracle.kron_rel_error(r.A, r.B, d.A_true / c, d.B_true * c))
    assert errs[0] > errs[1] > errs[2]
    assert 0.3 < errs[2] / errs[1] < 0.8 and 0.3 < errs[1] / errs[0] < 0.8


def test_spd_start_is_seeded_and_positive_definite():
    M = synth.spd_start(300, 5, rank=32)
    assert M.dtype == np.float32 and np.array_equal(M, synth.spd_start(300, 5, rank=32))
    lam = np.linalg.eigvalsh(M.astype(np.float64))
    assert lam.min() > 0.04 and lam.max() / lam.min() < 2e3
