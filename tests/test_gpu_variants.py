"""GPU parity of the Table 1 estimators other than FlipFlop (ff_config.estimator),
through the C ABI, against the fp64 oracle of ``oracle/variants.py`` (pinned
to the Van Loan-Pitsianis rearrangement, exact Kronecker designs and the
FlipFlop oracle).  Tolerances as for FlipFlop: relative Frobenius error of
the normalised A (x) B 1e-5 on the fp32 path, 5e-3 on the bf16 path, with
identical iteration counts."""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-5
TOL_BF16 = 5e-3


def dev(V, gpu):
    import torch
    if V.dtype == np.uint16:
        return torch.from_numpy(V.view(np.int16)).to(gpu).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(V, dtype=np.float32)).to(gpu)


def run(gpu, iters, G=None, tokens=None, **kw):
    import paper_2609_14706_amd as ffe
    if tokens is not None:
        f = ffe.FlipFlop(tokens=(dev(tokens[0], gpu), dev(tokens[1], gpu)), **kw)
    else:
        f = ffe.FlipFlop(dev(G, gpu), **kw)
    ll = f.iterate(iters)
    A, B = f.factors()
    out = (A.double().cpu().numpy(), B.double().cpu().numpy(), ll, f.iters_done)
    f.close()
    return out


# --------------------------------------------------------------- Frobenius

def test_frobenius_tiny_fp32(gpu):
    w = synth.workload("tiny")
    d = synth.generate(w)
    A, B, ll, done = run(gpu, 8, G=d.G, estimator="frobenius")
    ref = oracle.frobenius(d.G, 8)
    err = oracle.kron_rel_error(A, B, ref.A, ref.B)
    print(f"frobenius tiny fp32 8 iterations: rel err {err:.3e}")
    assert done == 8 and err < TOL_F32
    assert all(np.isnan(v) for v in ll)                      # no likelihood for this estimator
    # it is not the FlipFlop estimate
    ff = oracle.flipflop(d.G, 8)
    assert oracle.kron_rel_error(ref.A, ref.B, ff.A, ff.B) > 100 * TOL_F32


@pytest.mark.parametrize("m,n,N", [(100, 37, 3), (37, 100, 4), (130, 70, 5), (1, 20, 30), (300, 260, 2)])
def test_frobenius_fp32_ragged(gpu, m, n, N):
    """Shapes with ragged tails (the dense products with the factor run over
    zero-padded operands)."""
    rng = np.random.default_rng(m * 1000 + n + 7)
    G = (rng.standard_normal((N, m, n)) * np.linspace(0.5, 2.0, n)[None, None, :]).astype(np.float32)
    A, B, ll, done = run(gpu, 3, G=G, estimator="frobenius")
    ref = oracle.frobenius(G, 3)
    err = oracle.kron_rel_error(A, B, ref.A, ref.B)
    print(f"frobenius fp32 {m}x{n} N={N}: rel err {err:.3e}")
    assert done == 3 and err < TOL_F32


def test_frobenius_fp32_wide_factor(gpu):
    """A 6600-wide input factor (dense products over 6600-long rows).  With
    N m = 96 < n the update is singular; the paper's damping makes it
    positive definite."""
    rng = np.random.default_rng(6600)
    m, n, N = 48, 6600, 2
    G = (rng.standard_normal((N, m, n)) * np.linspace(0.5, 2.0, n)[None, None, :]).astype(np.float32)
    A, B, ll, done = run(gpu, 2, G=G, estimator="frobenius", damping=0.1)
    ref = oracle.frobenius(G, 2, damping=0.1)
    err = oracle.kron_rel_error(A, B, ref.A, ref.B)
    print(f"frobenius fp32 {m}x{n} N={N}: rel err {err:.3e}")
    assert done == 2 and err < TOL_F32


def test_frobenius_damping_and_order(gpu):
    import paper_2609_14706_amd as ffe
    d = synth.generate(synth.workload("tiny").scaled(m=48, n=80, N=40))
    A, B, ll, done = run(gpu, 5, G=d.G, estimator="frobenius", damping=0.1)
    ref = oracle.frobenius(d.G, 5, damping=0.1)
    assert oracle.kron_rel_error(A, B, ref.A, ref.B) < TOL_F32
    # with A first the trace normalisation lets B's scale grow doubly
    # exponentially (the fp64 oracle's B reaches ~1e44 after 5 iterations)
    ra = oracle.frobenius(d.G, 5, order="A_FIRST")
    assert np.abs(ra.B).max() > 1e30
    with pytest.raises(ffe.FlipFlopError) as ei:
        ffe.FlipFlop(dev(d.G, gpu), estimator="frobenius", order="A_FIRST")
    assert ei.value.code == ffe.FF_ERR_INVALID_ARG


@pytest.mark.parametrize("split", [1, 2])
def test_frobenius_bf16_multi_tile(gpu, split):
    """With the paper's damping (0.1 x mean diagonal, Appendix B)."""
    w = synth.workload("attn").scaled(m=600, n=520, N=6)
    d = synth.generate(w)
    A, B, ll, done = run(gpu, 4, G=d.G, estimator="frobenius", whiten_split=split, damping=0.1)
    ref = oracle.frobenius(d.G, 4, damping=0.1)
    err = oracle.kron_rel_error(A, B, ref.A, ref.B)
    print(f"frobenius bf16 600x520 N=6 split={split} damping 0.1: rel err {err:.3e}")
    assert done == 4 and err < TOL_BF16


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_frobenius_undamped_ill_conditioned(gpu, dtype):
    """Undamped on 6 samples, the Frobenius A reaches a condition number of
    7e7 after two iterations (fp64 oracle), beyond what an fp32 factorisation
    of it could take.  The iteration uses the factors themselves (dense
    products, no factorisation, Section 5), so all four iterations run, as in
    the oracle, and match it."""
    w = synth.workload("attn").scaled(m=600, n=520, N=6)
    d = synth.generate(w)
    hist = oracle.frobenius(d.G, 4, keep_history=True).history
    assert np.linalg.cond(hist[1][0]) > 1e7
    G = d.G if dtype == "bf16" else oracle.as_f64_samples(d.G).astype(np.float32)  # exact upcast
    A, B, ll, done = run(gpu, 4, G=G, estimator="frobenius")
    err = oracle.kron_rel_error(A, B, *hist[3])
    err1 = oracle.kron_rel_error(*run(gpu, 1, G=G, estimator="frobenius")[:2], *hist[0])
    print(f"frobenius undamped {dtype}: rel err after 1 iteration {err1:.3e}, after 4 {err:.3e}")
    assert done == 4 and err < (TOL_F32 if dtype == "f32" else TOL_BF16)


def test_frobenius_tokens(gpu):
    w = synth.token_workload("tokens_tiny")
    d = synth.generate_tokens(w)
    A, B, ll, done = run(gpu, 6, tokens=(d.x, d.g), estimator="frobenius")
    ref = oracle.frobenius_tokens(d.x, d.g, 6)
    err = oracle.kron_rel_error(A, B, ref.A, ref.B)
    print(f"frobenius tokens fp32: rel err {err:.3e}")
    assert done == 6 and err < TOL_F32
    wb = synth.token_workload("tokens_attn").scaled(T=6000, m=320, n=384)
    db = synth.generate_tokens(wb)
    A, B, ll, done = run(gpu, 3, tokens=(db.x, db.g), estimator="frobenius")
    ref = oracle.frobenius_tokens(db.x, db.g, 3)
    err = oracle.kron_rel_error(A, B, ref.A, ref.B)
    print(f"frobenius tokens bf16 320x384 T=6000: rel err {err:.3e}")
    assert err < TOL_BF16


def test_frobenius_resume_and_kron_apply(gpu):
    """3 + 2 iterations equal 5 (bitwise), also with an inverse Kronecker
    application in between (it factorises the factors for their inverses in
    the buffers the iteration uses; the Frobenius operand must be rebuilt)."""
    import torch
    import paper_2609_14706_amd as ffe
    d = synth.generate(synth.workload("tiny").scaled(m=40, n=72, N=30))
    f = ffe.FlipFlop(dev(d.G, gpu), estimator="frobenius")
    f.iterate(3)
    f.kron_apply(torch.ones((1, 40, 72)), inverse=True)
    f.iterate(2)
    A1, B1 = f.factors()
    f.close()
    A2, B2, _, _ = run(gpu, 5, G=d.G, estimator="frobenius")
    assert np.array_equal(A1.double().cpu().numpy(), A2) and np.array_equal(B1.double().cpu().numpy(), B2)


# ------------------------------------------------------ Marginal and Input

@pytest.mark.parametrize("estimator", ["marginal", "input"])
@pytest.mark.parametrize("damping", [0.0, 0.1])
def test_token_means_fp32(gpu, estimator, damping):
    w = synth.token_workload("tokens_tiny").scaled(T=2777, m=33, n=65)
    d = synth.generate_tokens(w)
    A, B, ll, done = run(gpu, 2, tokens=(d.x, d.g), estimator=estimator, damping=damping)
    if estimator == "marginal":
        rA, rB = oracle.marginal_tokens(d.x, d.g, damping=damping)
    else:
        rA, rB = oracle.input_tokens(d.x, w.m, damping=damping)
    err = oracle.kron_rel_error(A, B, rA, rB)
    print(f"{estimator} fp32 damping {damping}: rel err {err:.3e}")
    assert done == 2 and err < TOL_F32 and all(np.isnan(v) for v in ll)


@pytest.mark.parametrize("estimator", ["marginal", "input"])
def test_token_means_bf16(gpu, estimator):
    w = synth.token_workload("tokens_attn").scaled(T=9000, m=520, n=600)
    d = synth.generate_tokens(w)
    A, B, ll, done = run(gpu, 1, tokens=(d.x, d.g), estimator=estimator)
    if estimator == "marginal":
        rA, rB = oracle.marginal_tokens(d.x, d.g)
    else:
        rA, rB = oracle.input_tokens(d.x, w.m)
    err = oracle.kron_rel_error(A, B, rA, rB)
    print(f"{estimator} bf16 520x600 T=9000: rel err {err:.3e}")
    assert err < TOL_BF16


def test_token_means_need_tokens(gpu):
    import paper_2609_14706_amd as ffe
    G = np.ones((2, 4, 5), np.float32)
    for est in ("marginal", "input"):
        with pytest.raises(ffe.FlipFlopError) as ei:
            ffe.FlipFlop(dev(G, gpu), estimator=est)
        assert ei.value.code == ffe.FF_ERR_INVALID_ARG


# ---------------------------------------------------------------- full size

@pytest.mark.timeout(600)
def test_frobenius_full_size_attention_layer(gpu):
    """4096 x 4096, N = 128, bf16, the paper's damping: the returned A is the
    damped, trace-normalised half step (1/(N m)) sum_i G_i^T B G_i of the
    returned B (the last update of the iteration), evaluated here in fp64;
    and the factors are symmetric positive definite with tr(A) = n."""
    import torch
    import paper_2609_14706_amd as ffe
    w = synth.workload("attn")
    G = synth.generate_device(w, device=gpu)
    f = ffe.FlipFlop(G, estimator="frobenius", damping=0.1)
    ll = f.iterate(3)
    A, B = f.factors()
    f.close()
    assert len(ll) == 3 and all(np.isnan(v) for v in ll)
    assert abs(float(torch.trace(A.double())) - w.n) < 1e-3
    assert bool((A == A.T).all()) and bool((B == B.T).all())
    torch.linalg.cholesky(A.double())
    torch.linalg.cholesky(B.double())
    Bd = B.double()
    M = torch.zeros((w.n, w.n), dtype=torch.float64, device=gpu)
    for i in range(w.N):
        Gi = G[i].double()
        M += Gi.T @ (Bd @ Gi)
    M = M / (w.N * w.m)
    M = M + (0.1 * float(torch.trace(M)) / w.n) * torch.eye(w.n, dtype=torch.float64, device=gpu)
    M = M * (w.n / float(torch.trace(M)))
    err = float(torch.linalg.norm(A.double() - M) / torch.linalg.norm(M))
    print(f"frobenius full size: last half step vs fp64 {err:.3e}", flush=True)
    assert err < TOL_BF16
