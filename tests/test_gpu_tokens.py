"""GPU parity of the per-token (rank-one) form, G_t = g_t x_t^T, through the
C ABI (ff_config.form = FF_SAMPLES_RANK1), against the fp64 token oracle
(itself pinned to the dense oracle on the materialised samples).
Tolerances as for the dense form: 1e-5 (fp32 path), 5e-3 (bf16 path),
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


def run(x, g, iters, gpu, **kw):
    import paper_2609_14706_amd as ffe
    f = ffe.FlipFlop(tokens=(dev(x, gpu), dev(g, gpu)), **kw)
    ll = f.iterate(iters)
    A, B = f.factors()
    psi = f.objective()
    out = (A.double().cpu().numpy(), B.double().cpu().numpy(), ll, f.iters_done, psi)
    f.close()
    return out


def test_tokens_tiny_full_parity(gpu):
    w = synth.token_workload("tokens_tiny")
    d = synth.generate_tokens(w)
    A, B, ll, done, psi = run(d.x, d.g, w.iters, gpu)
    ref = oracle.flipflop_tokens(d.x, d.g, w.iters)
    err = oracle.kron_rel_error(A, B, ref.A, ref.B)
    print(f"tokens tiny fp32: rel err {err:.3e}")
    assert done == w.iters and err < TOL_F32
    llref = oracle.loglik_tokens(d.x, d.g, ref.A, ref.B)
    assert abs(ll[-1] - llref) < 1e-6 * abs(llref)
    assert abs(psi - oracle.objective_tokens(d.x, d.g, ref.A, ref.B)) < TOL_F32


@pytest.mark.parametrize("T,m,n", [(777, 33, 65), (300, 70, 130), (5000, 1, 40), (5000, 40, 1)])
def test_tokens_fp32_ragged(gpu, T, m, n):
    w = synth.token_workload("tokens_tiny").scaled(T=T, m=m, n=n)
    d = synth.generate_tokens(w)
    A, B, ll, done, _ = run(d.x, d.g, 5, gpu)
    ref = oracle.flipflop_tokens(d.x, d.g, 5)
    assert done == 5 and oracle.kron_rel_error(A, B, ref.A, ref.B) < TOL_F32


@pytest.mark.parametrize("order,damping", [("A_FIRST", 0.0), ("B_FIRST", 0.1)])
def test_tokens_order_and_damping(gpu, order, damping):
    w = synth.token_workload("tokens_tiny").scaled(T=2000, m=40, n=72)
    d = synth.generate_tokens(w)
    A, B, _, _, _ = run(d.x, d.g, 6, gpu, order=order, damping=damping)
    ref = oracle.flipflop_tokens(d.x, d.g, 6, order=order, damping=damping)
    assert oracle.kron_rel_error(A, B, ref.A, ref.B) < TOL_F32


@pytest.mark.parametrize("split", [0, 1, 2])
def test_tokens_bf16_multi_tile(gpu, split):
    """3 x 3 tiles of 256 with ragged tails on both sides, bf16 tokens."""
    w = synth.token_workload("tokens_attn").scaled(T=6000, m=600, n=520, iters=6)
    d = synth.generate_tokens(w)
    A, B, ll, done, psi = run(d.x, d.g, w.iters, gpu, whiten_split=split)
    ref = oracle.flipflop_tokens(d.x, d.g, w.iters)
    err = oracle.kron_rel_error(A, B, ref.A, ref.B)
    print(f"tokens bf16 600x520 T=6000 split={split}: rel err {err:.3e}")
    assert done == w.iters and err < TOL_BF16
    assert abs(psi - oracle.objective_tokens(d.x, d.g, ref.A, ref.B)) < TOL_BF16


def test_tokens_attn_fullsize(gpu):
    """The paper's calibration size (256 x 2048 = 524288 tokens) at the
    attention width 4096 x 4096, bf16: sampled rows of the first B update
    (with A = I) from the token oracle, then properties after 10 iterations:
    trace normalisation, symmetry, positive definiteness, the likelihood
    rising then flat, the trace identity (1/(T m n)) sum_t w_t v_t = 1, and
    the device log-likelihood against an fp64 evaluation from the factors."""
    import torch
    import paper_2609_14706_amd as ffe
    w = synth.token_workload("tokens_attn")
    print(f"[{w.name}] generating on the device", flush=True)
    x, g = synth.generate_tokens_device(w, device=gpu)
    f = ffe.FlipFlop(tokens=(x, g))
    f.iterate(1)
    _, B1 = f.factors()
    f.close()
    rows = np.array([0, 1, 1000, 2049, 4095])
    print(f"[{w.name}] oracle rows of the first B update", flush=True)
    xh = x.view(torch.int16).cpu().numpy().view(np.uint16)
    gh = g.view(torch.int16).cpu().numpy().view(np.uint16)
    ref = oracle.half_step_B_tokens_rows(xh, gh, None, rows)
    del xh, gh
    got = B1.double().cpu().numpy()[rows]
    # Unlike the dense form (where A = I makes the first update exact up to
    # fp32 accumulation), the tokens scaled by sqrt(w_t) are rounded to bf16
    # before the product, so the bf16 bar applies here (measured ~8e-5).
    for k, r in enumerate(rows):
        a = got[k] / got[k, r]
        b = ref[k] / ref[k, r]
        err = np.linalg.norm(a - b) / np.linalg.norm(b)
        print(f"[{w.name}] row {r}: rel err {err:.3e}", flush=True)
        assert err < TOL_BF16, (r, err)
    print(f"[{w.name}] {w.iters} iterations", flush=True)
    f = ffe.FlipFlop(tokens=(x, g))
    ll = f.iterate(w.iters)
    A, B = f.factors()
    f.close()
    print(f"[{w.name}] loglik per iteration: {ll}", flush=True)
    Tmn = w.T * w.m * w.n
    assert abs(float(torch.trace(A.double())) - w.n) < 1e-6 * w.n
    assert bool((A == A.T).all()) and bool((B == B.T).all())
    LA = torch.linalg.cholesky(A.double())
    LB = torch.linalg.cholesky(B.double())
    assert ll[1] > ll[0] and ll[-1] > ll[0]
    tail = ll[w.iters // 2:]
    assert max(tail) - min(tail) < 1e-4 * Tmn
    tot = 0.0
    LA32, LB32 = LA.float(), LB.float()
    for t0 in range(0, w.T, 65536):
        xs = torch.linalg.solve_triangular(LA32, x[t0:t0 + 65536].float().T, upper=False)
        gs = torch.linalg.solve_triangular(LB32, g[t0:t0 + 65536].float().T, upper=False)
        tot += float(((xs.double() ** 2).sum(0) * (gs.double() ** 2).sum(0)).sum())
    t = tot / Tmn
    print(f"[{w.name}] trace identity: {t:.6f}", flush=True)
    assert abs(t - 1.0) < 5e-3
    ldA = 2.0 * float(torch.log(torch.diagonal(LA)).sum())
    ldB = 2.0 * float(torch.log(torch.diagonal(LB)).sum())
    llref = -0.5 * w.T * (w.m * ldA + w.n * ldB) - 0.5 * Tmn * (1.0 + np.log(2 * np.pi))
    bound = 32 * float(np.finfo(np.float32).eps) * Tmn      # fp32 pivots, as for the dense form
    print(f"[{w.name}] loglik device {ll[-1]:.9e} fp64 {llref:.9e} (bound {bound:.3e})", flush=True)
    assert abs(ll[-1] - llref) < bound
