"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Inputs are the seeded synthetic workloads; the oracle never sees anything
the GPU produced.  Tolerances (relative Frobenius error of the normalised
A (x) B, evaluated in fp64): 1e-5 on the fp32 path, 5e-3 on the bf16 path,
with identical iteration counts.
"""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-5
TOL_BF16 = 5e-3


def to_device(G_np, device):
    import torch
    if G_np.dtype == np.uint16:
        return torch.from_numpy(G_np.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(G_np, dtype=np.float32)).to(device)


def run_gpu(G_np, iters, device, **kw):
    import paper_2609_14706_amd as ffe
    f = ffe.FlipFlop(to_device(G_np, device), **kw)
    ll = f.iterate(iters)
    A, B = f.factors()
    out = (A.double().cpu().numpy(), B.double().cpu().numpy(), ll, f.iters_done)
    f.close()
    return out


def small_workload(key, **kw):
    return synth.workload(key).scaled(**kw)


# ------------------------------------------------------------- fp32 path

def test_tiny_first_iteration(gpu):
    d = synth.generate(synth.workload("tiny"))
    A, B, ll, done = run_gpu(d.G, 1, gpu)
    ref = oracle.flipflop(d.G, 1)
    assert done == 1
    assert abs(np.trace(A) - 128) < 1e-3
    assert oracle.kron_rel_error(A, B, ref.A, ref.B) < TOL_F32


def test_tiny_workload_full_parity(gpu):
    """The 64 x 128, N = 256 workload: 20 iterations from A = I, fp32."""
    w = synth.workload("tiny")
    d = synth.generate(w)
    A, B, ll, done = run_gpu(d.G, w.iters, gpu)
    ref = oracle.flipflop(d.G, w.iters)
    err = oracle.kron_rel_error(A, B, ref.A, ref.B)
    esf = oracle.kron_rel_error_scale_free(A, B, ref.A, ref.B)
    print(f"tiny fp32 20 iterations: rel err {err:.3e} (scale-free {esf:.3e})")
    assert done == w.iters
    assert err < TOL_F32 and esf < TOL_F32
    # per-iteration log-likelihood against the oracle's, for the last iterate
    assert abs(ll[-1] - oracle.loglik(d.G, ref.A, ref.B)) < 1e-6 * abs(ll[-1])
    assert all(b >= a - 1e-6 * abs(a) for a, b in zip(ll, ll[1:]))


@pytest.mark.parametrize("m,n,N", [(100, 37, 3), (37, 100, 4), (130, 70, 5), (1, 20, 30), (20, 1, 30)])
def test_fp32_ragged_shapes(gpu, m, n, N):
    rng = np.random.default_rng(m * 1000 + n)
    G = (rng.standard_normal((N, m, n)) * np.linspace(0.5, 2.0, n)[None, None, :]).astype(np.float32)
    A, B, ll, done = run_gpu(G, 4, gpu)
    ref = oracle.flipflop(G, 4)
    assert done == 4
    assert oracle.kron_rel_error(A, B, ref.A, ref.B) < TOL_F32


@pytest.mark.parametrize("order,damping", [("A_FIRST", 0.0), ("B_FIRST", 0.1), ("A_FIRST", 0.1)])
def test_fp32_order_and_damping(gpu, order, damping):
    d = synth.generate(small_workload("tiny", m=48, n=80, N=40))
    A, B, ll, done = run_gpu(d.G, 6, gpu, order=order, damping=damping)
    ref = oracle.flipflop(d.G, 6, order=order, damping=damping)
    assert oracle.kron_rel_error(A, B, ref.A, ref.B) < TOL_F32


def test_fp32_start_factor(gpu):
    rng = np.random.default_rng(5)
    d = synth.generate(small_workload("tiny", m=40, n=72, N=30))
    Q = synth.haar_orthogonal(72, rng)
    A0 = (Q * np.geomspace(3.0, 0.3, 72)) @ Q.T
    import torch
    A, B, ll, done = run_gpu(d.G, 3, gpu, A0=torch.from_numpy(A0.astype(np.float32)))
    ref = oracle.flipflop(d.G, 3, A0=A0.astype(np.float32).astype(np.float64))
    assert oracle.kron_rel_error(A, B, ref.A, ref.B) < TOL_F32


# -------------------------------------------------------------- bf16 path

@pytest.mark.parametrize("split", [0, 1, 2])
def test_bf16_ragged_multi_tile(gpu, split):
    """Attention-layer generator (power-law spectra, 10% rank-32 noise) at a
    size the oracle finishes in seconds: 3 x 3 tiles with ragged tails."""
    w = small_workload("attn", m=600, n=520, N=6)
    d = synth.generate(w)
    A, B, ll, done = run_gpu(d.G, w.iters, gpu, whiten_split=split)
    ref = oracle.flipflop(d.G, w.iters)
    err = oracle.kron_rel_error(A, B, ref.A, ref.B)
    print(f"bf16 600x520 N=6 split={split}: rel err {err:.3e}")
    assert done == w.iters
    assert err < TOL_BF16


@pytest.mark.parametrize("key,m,n,N", [("mlp_down", 256, 688, 64), ("mlp_up", 768, 512, 16)])
def test_bf16_config_shaped(gpu, key, m, n, N):
    """Reduced layers with the aspect ratio and samples-per-dimension of the
    MLP workloads (N m / n and N n / m as in the full configurations)."""
    w = small_workload(key, m=m, n=n, N=N)
    d = synth.generate(w)
    A, B, ll, done = run_gpu(d.G, w.iters, gpu)
    ref = oracle.flipflop(d.G, w.iters)
    err = oracle.kron_rel_error(A, B, ref.A, ref.B)
    esf = oracle.kron_rel_error_scale_free(A, B, ref.A, ref.B)
    A1, B1, _, _ = run_gpu(d.G, 1, gpu)
    r1 = oracle.flipflop(d.G, 1)
    err1 = oracle.kron_rel_error(A1, B1, r1.A, r1.B)
    print(f"bf16 {key} {m}x{n} N={N}: rel err {err:.3e} after {w.iters} (scale-free {esf:.3e}), "
          f"{err1:.3e} after 1")
    assert done == w.iters
    assert err < TOL_BF16 and err1 < TOL_BF16 and esf < TOL_BF16


def test_bf16_ill_conditioned_split(gpu):
    """Few samples per input channel (N m / n = 1.6) make the estimated A very
    ill-conditioned (condition ~7e4, rounding sensitivity s(A) = 10 after the
    first iteration, 26 after the tenth); one bf16 pass of L^-1 then costs
    about 8e-3, and the hi/lo split of L^-1 (two passes) brings the error
    back under the bar.  The default (automatic) rule switches both
    whitenings to two passes once s(A) > 16 and meets the bar."""
    w = small_workload("mlp_down", m=512, n=1280, N=4)
    d = synth.generate(w)
    ref = oracle.flipflop(d.G, w.iters)
    errs = {}
    for split in (1, 2, 0):
        A, B, ll, done = run_gpu(d.G, w.iters, gpu, whiten_split=split)
        errs[split] = oracle.kron_rel_error(A, B, ref.A, ref.B)
    print(f"bf16 512x1280 N=4: split1 {errs[1]:.3e}, split2 {errs[2]:.3e}, automatic {errs[0]:.3e}")
    assert errs[2] < TOL_BF16 and errs[0] < TOL_BF16
    assert errs[2] < 0.5 * errs[1]


def test_automatic_split_statistic(gpu):
    """The device statistic s = (1/dim) sum_j F_jj (F^-1)_jj of the last
    factorised A and B equals its fp64 evaluation from the returned factors
    (s is invariant under the trace normalisation's scaling), and both
    whitenings use two passes exactly when max(s(A), s(B)) > 16 or fewer than
    16 samples per dimension determine a factor (min(N m / n, N n / m); the
    rank-one form: T / max(m, n))."""
    import torch
    import paper_2609_14706_amd as ffe

    def expected_passes(sA, sB, r):
        return 2 if (max(sA, sB) > 16 or r < 16) else 1

    for key, kw in (("mlp_down", dict(m=512, n=1280, N=4)), ("attn", dict(m=512, n=768, N=8)),
                    ("attn", dict(m=512, n=512, N=32))):
        w = small_workload(key, **kw)
        d = synth.generate(w)
        f = ffe.FlipFlop(to_device(d.G, gpu))
        f.iterate(w.iters)
        A, B = (X.double().cpu().numpy() for X in f.factors())
        sA, sB, pA, pB = f.whiten_split_state()
        f.close()
        ref = [float(np.mean(np.diag(X) * np.diag(np.linalg.inv(X)))) for X in (A, B)]
        r = w.N * min(w.m, w.n) / max(w.m, w.n)
        print(f"{w.name}: device s(A) {sA:.6f} s(B) {sB:.6f}; fp64 {ref[0]:.6f} {ref[1]:.6f}; "
              f"{r:.1f} samples per dimension; passes {pA} / {pB}")
        assert abs(sA - ref[0]) < 1e-3 * ref[0] and abs(sB - ref[1]) < 1e-3 * ref[1]
        assert pA == pB == expected_passes(sA, sB, r)
    # the rank-one (per-token) form computes the same statistic from its factorisations
    wt = synth.token_workload("tokens_attn").scaled(T=3000, m=320, n=384, iters=4)
    dt = synth.generate_tokens(wt)
    f = ffe.FlipFlop(tokens=(to_device(dt.x, gpu), to_device(dt.g, gpu)))
    f.iterate(wt.iters)
    A, B = (X.double().cpu().numpy() for X in f.factors())
    sA, sB, pA, pB = f.whiten_split_state()
    f.close()
    ref = [float(np.mean(np.diag(X) * np.diag(np.linalg.inv(X)))) for X in (A, B)]
    print(f"{wt.name}: device s(A) {sA:.6f} s(B) {sB:.6f}; fp64 {ref[0]:.6f} {ref[1]:.6f}")
    assert abs(sA - ref[0]) < 1e-3 * ref[0] and abs(sB - ref[1]) < 1e-3 * ref[1]
    assert pA == pB == expected_passes(sA, sB, wt.T / max(wt.m, wt.n))
    # forced settings report their pass counts and no statistic
    w = small_workload("attn", m=256, n=256, N=4)
    G = to_device(synth.generate(w).G, gpu)
    for split in (1, 2):
        f = ffe.FlipFlop(G, whiten_split=split)
        f.iterate(2)
        sA, sB, pA, pB = f.whiten_split_state()
        f.close()
        assert np.isnan(sA) and np.isnan(sB) and (pA, pB) == (split, split)


# ------------------------------------------------------------- kron apply

def test_kron_apply_matches_oracle(gpu):
    import torch
    import paper_2609_14706_amd as ffe
    rng = np.random.default_rng(11)
    m, n = 70, 150
    QA, QB = synth.haar_orthogonal(n, rng), synth.haar_orthogonal(m, rng)
    A0 = ((QA * np.geomspace(2.0, 0.2, n)) @ QA.T).astype(np.float32)
    B0 = ((QB * np.geomspace(4.0, 0.5, m)) @ QB.T).astype(np.float32)
    G = rng.standard_normal((3, m, n)).astype(np.float32)
    f = ffe.FlipFlop(to_device(G, gpu), A0=torch.from_numpy(A0), B0=torch.from_numpy(B0))
    X = rng.standard_normal((5, m, n)).astype(np.float32)
    Y = f.kron_apply(torch.from_numpy(X)).double().cpu().numpy()
    Yi = f.kron_apply(torch.from_numpy(X), inverse=True).double().cpu().numpy()
    f.close()
    ref = oracle.kron_apply(A0.astype(np.float64), B0.astype(np.float64), X)
    refi = oracle.kron_apply(A0.astype(np.float64), B0.astype(np.float64), X, inverse=True)
    assert np.linalg.norm(Y - ref) / np.linalg.norm(ref) < 1e-5
    assert np.linalg.norm(Yi - refi) / np.linalg.norm(refi) < 1e-4


@pytest.mark.parametrize("m,n,tol", [(300, 1000, 1e-5), (64, 6600, 1e-5)])
def test_kron_apply_inverse_blocked_factorisation(gpu, m, n, tol):
    """The inverse application at widths that take the blocked factorisation
    (1000: eight 128-column panels with a ragged last block; 6600: outer
    panels of 1024 columns and a ragged last outer panel), against fp64
    solves with the same start factors."""
    import torch
    import paper_2609_14706_amd as ffe
    rng = np.random.default_rng(12)
    QA, QB = synth.haar_orthogonal(n, rng), synth.haar_orthogonal(m, rng)
    A0 = ((QA * np.geomspace(2.0, 0.2, n)) @ QA.T).astype(np.float32)
    B0 = ((QB * np.geomspace(4.0, 0.5, m)) @ QB.T).astype(np.float32)
    G = rng.standard_normal((1, m, n)).astype(np.float32)
    f = ffe.FlipFlop(to_device(G, gpu), A0=torch.from_numpy(A0), B0=torch.from_numpy(B0))
    X = rng.standard_normal((2, m, n)).astype(np.float32)
    Yi = f.kron_apply(torch.from_numpy(X), inverse=True).double().cpu().numpy()
    f.close()
    refi = oracle.kron_apply(A0.astype(np.float64), B0.astype(np.float64), X, inverse=True)
    err = np.linalg.norm(Yi - refi) / np.linalg.norm(refi)
    print(f"m={m} n={n}: inverse application rel err {err:.2e}")
    assert err < tol


# --------------------------------------------------------- failure handling

def test_rank_deficient_samples_report_not_spd(gpu):
    import paper_2609_14706_amd as ffe
    rng = np.random.default_rng(10)
    G = rng.standard_normal((2, 3, 9)).astype(np.float32)   # N m = 6 < n = 9
    with pytest.raises(oracle.NotSPDError) as oi:
        oracle.flipflop(G, 3)
    f = ffe.FlipFlop(to_device(G, gpu))
    with pytest.raises(ffe.FlipFlopError) as ei:
        f.iterate(3)
    assert ei.value.code == ffe.FF_ERR_NOT_SPD
    assert ei.value.iters_done == oi.value.iteration - 1
    A, B = f.factors()                                      # last completed iteration kept
    ref = oracle.flipflop(G, oi.value.iteration - 1)
    assert oracle.kron_rel_error(A.double().cpu().numpy(), B.double().cpu().numpy(),
                                 ref.A, ref.B) < TOL_F32
    f.close()
    # an iteration whose new factor is singular still completes on its own,
    # as in the oracle; the next one, which must invert it, fails
    f = ffe.FlipFlop(to_device(G, gpu))
    ll = f.iterate(1)
    assert f.iters_done == 1 and len(ll) == 1 and np.isnan(ll[0])
    with pytest.raises(ffe.FlipFlopError) as ei:
        f.iterate(1)
    assert ei.value.code == ffe.FF_ERR_NOT_SPD and ei.value.iters_done == 0
    f.close()
    # damping makes the same samples well posed
    A, B, ll, done = run_gpu(G, 3, gpu, damping=0.1)
    ref = oracle.flipflop(G, 3, damping=0.1)
    assert done == 3 and oracle.kron_rel_error(A, B, ref.A, ref.B) < TOL_F32


def test_nan_samples_report_not_spd(gpu):
    import paper_2609_14706_amd as ffe
    G = np.random.default_rng(3).standard_normal((4, 16, 8)).astype(np.float32)
    G[2, 5, 3] = np.nan
    f = ffe.FlipFlop(to_device(G, gpu))
    with pytest.raises(ffe.FlipFlopError) as ei:
        f.iterate(2)
    assert ei.value.code == ffe.FF_ERR_NOT_SPD and ei.value.iters_done == 0
    A, B = f.factors()
    assert np.array_equal(A.cpu().numpy(), np.eye(8, dtype=np.float32))
    f.close()


# ----------------------------------------------- resume and determinism

def test_resume_and_bitwise_determinism(gpu):
    import paper_2609_14706_amd as ffe
    d = synth.generate(small_workload("attn", m=512, n=768, N=4))
    G = to_device(d.G, gpu)
    f1 = ffe.FlipFlop(G)
    f1.iterate(3)
    f1.iterate(2)
    A1, B1 = f1.factors()
    f2 = ffe.FlipFlop(G)
    f2.iterate(5)
    A2, B2 = f2.factors()
    assert bool((A1 == A2).all()) and bool((B1 == B2).all())
    f1.close()
    f2.close()


@pytest.mark.parametrize("key,m,n,N", [("attn", 512, 768, 4), ("tiny", 64, 128, 32)])
@pytest.mark.parametrize("order", ["B_FIRST", "A_FIRST"])
def test_identity_start_is_exact(gpu, key, m, n, N, order):
    """Without A0 / B0 the first half step skips the whitening by the inverse
    factor of I and the factorisation of I; with the identity passed
    explicitly both run.  A product with I is exact in every precision, so the
    iterates must agree bitwise (bf16 and fp32 paths, both orders)."""
    import torch
    import paper_2609_14706_amd as ffe
    d = synth.generate(small_workload(key, m=m, n=n, N=N))
    G = to_device(d.G, gpu)
    kw = {"A0": torch.eye(n)} if order == "B_FIRST" else {"B0": torch.eye(m)}
    f1 = ffe.FlipFlop(G, order=order)
    ll1 = f1.iterate(3)
    A1, B1 = f1.factors()
    f2 = ffe.FlipFlop(G, order=order, **kw)
    ll2 = f2.iterate(3)
    A2, B2 = f2.factors()
    f1.close()
    f2.close()
    assert bool((A1 == A2).all()) and bool((B1 == B2).all())
    assert ll1 == ll2


# ------------------------------------------------------- mismatch objective

def _spd(dim, rng, cond):
    Q = synth.haar_orthogonal(dim, rng)
    return ((Q * np.geomspace(1.0, 1.0 / cond, dim)) @ Q.T).astype(np.float32)


@pytest.mark.parametrize("dtype,tol", [("f32", 1e-5), ("bf16", 5e-3)])
def test_objective_at_given_factors(gpu, dtype, tol):
    """psi = log Phi(H, A (x) B) + log|H|/(mn) (Section 4) at factors that are
    not a fixed point, through the handle's own path; A, B are the same fp32
    values on both sides."""
    import torch
    import paper_2609_14706_amd as ffe
    rng = np.random.default_rng(21)
    m, n, N = (48, 80, 40) if dtype == "f32" else (600, 520, 6)
    w = small_workload("attn", m=m, n=n, N=N)
    d = synth.generate(w) if dtype == "bf16" else None
    G = d.G if dtype == "bf16" else synth.generate(small_workload("tiny", m=m, n=n, N=N)).G
    A, B = _spd(n, rng, 30.0), _spd(m, rng, 50.0)
    f = ffe.FlipFlop(to_device(G, gpu))
    psi = f.objective(torch.from_numpy(A), torch.from_numpy(B))
    f.close()
    ref = oracle.objective(G, A.astype(np.float64), B.astype(np.float64))
    print(f"objective {dtype} {m}x{n} N={N}: device {psi:.9f} oracle {ref:.9f}")
    assert abs(psi - ref) < tol


def test_objective_of_current_factors_and_handle_state(gpu):
    """Default factors are the handle's current ones; psi falls over the
    iterations as the oracle's does; evaluating foreign factors leaves the
    iteration itself unchanged (bitwise against an undisturbed handle); a
    factor that is not positive definite is reported."""
    import torch
    import paper_2609_14706_amd as ffe
    rng = np.random.default_rng(22)
    d = synth.generate(small_workload("tiny", m=40, n=72, N=30))
    G = to_device(d.G, gpu)
    f = ffe.FlipFlop(G)
    g = ffe.FlipFlop(G)
    psis = []
    for k in range(3):
        f.iterate(1)
        g.iterate(1)
        psis.append(f.objective())
        f.objective(torch.from_numpy(_spd(72, rng, 5.0)), None)   # foreign A, then keep going
    refs = [oracle.objective(d.G, r.A, r.B) for r in
            (oracle.flipflop(d.G, k) for k in (1, 2, 3))]
    print("psi device", psis, "oracle", refs)
    assert all(abs(a - b) < 1e-5 for a, b in zip(psis, refs))
    assert psis[0] >= psis[1] >= psis[2]
    f.iterate(2)
    g.iterate(2)
    A1, B1 = f.factors()
    A2, B2 = g.factors()
    assert bool((A1 == A2).all()) and bool((B1 == B2).all())
    bad = -torch.eye(72)
    with pytest.raises(ffe.FlipFlopError) as ei:
        f.objective(bad, None)
    assert ei.value.code == ffe.FF_ERR_NOT_SPD
    f.iterate(1)
    g.iterate(1)
    A1, _ = f.factors()
    A2, _ = g.factors()
    assert bool((A1 == A2).all())
    f.close()
    g.close()
