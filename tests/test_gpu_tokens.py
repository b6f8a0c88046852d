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


@pytest.mark.parametrize("split", [1, 2])
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
