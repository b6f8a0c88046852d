"""The allocation-free entry point (ff_fit_noalloc) against the workspace
path (ff_init + ff_iterate + ff_factors) through the C ABI: two calls in a
row on one device, the second with a smaller input, each bitwise equal to
the workspace path and within the fp32 bar of the oracle."""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu


def _config(G, dtype):
    import torch
    import paper_2609_14706_amd as ffe
    cfg = ffe.ff_config()
    cfg.N, cfg.m, cfg.n = G.shape
    cfg.dtype = ffe.FF_BF16 if dtype == "bf16" else ffe.FF_F32
    cfg.G = G.data_ptr()
    cfg.stream = torch.cuda.current_stream(G.device).cuda_stream
    cfg.whiten_split = 0  # the library's default (automatic), as in the workspace path below
    return cfg


def _noalloc(G, iters, dtype):
    import torch
    import paper_2609_14706_amd as ffe
    N, m, n = G.shape
    A = torch.full((n, n), float("nan"), dtype=torch.float32, device=G.device)
    B = torch.full((m, m), float("nan"), dtype=torch.float32, device=G.device)
    torch.cuda.synchronize()
    done, ll = ffe.ff_fit_noalloc(_config(G, dtype), iters, A.data_ptr(), B.data_ptr())
    return done, ll, A, B


def _workspace_path(G, iters):
    import paper_2609_14706_amd as ffe
    f = ffe.FlipFlop(G, whiten_split=0)
    ll = f.iterate(iters)
    A, B = f.factors()
    f.close()
    return ll, A, B


@pytest.mark.parametrize("first,second", [
    (("tiny", dict(m=64, n=128, N=256), "f32", 6), ("tiny", dict(m=33, n=70, N=12), "f32", 4)),
    (("attn", dict(m=600, n=520, N=6), "bf16", 3), ("attn", dict(m=130, n=260, N=5), "bf16", 2)),
])
def test_noalloc_matches_workspace_path_two_calls(gpu, first, second):
    import torch
    for key, kw, dtype, iters in (first, second):
        w = synth.workload(key).scaled(**kw, dtype=dtype)
        print(f"no-alloc: {w.m} x {w.n}, N = {w.N}, {dtype}, {iters} iterations", flush=True)
        d = synth.generate(w)
        if dtype == "bf16":
            G = torch.from_numpy(d.G.view(np.int16)).to(gpu).view(torch.bfloat16)
        else:
            G = torch.from_numpy(d.G).to(gpu)
        done, ll, A, B = _noalloc(G, iters, dtype)
        ll_ref, A_ref, B_ref = _workspace_path(G, iters)
        assert done == iters
        assert torch.equal(A, A_ref) and torch.equal(B, B_ref)
        np.testing.assert_array_equal(np.array(ll), np.array(ll_ref))
        ref = oracle.flipflop(d.G, iters)
        err = oracle.kron_rel_error(A.double().cpu().numpy(), B.double().cpu().numpy(), ref.A, ref.B)
        print(f"  bitwise equal to the workspace path; {err:.2e} from the oracle", flush=True)
        assert err < (1e-5 if dtype == "f32" else 5e-3)


def test_noalloc_rejects_problems_beyond_its_scratch(gpu):
    import torch
    import paper_2609_14706_amd as ffe
    G = torch.zeros((128, 1024, 1024), dtype=torch.bfloat16, device=gpu)
    A = torch.zeros((1024, 1024), dtype=torch.float32, device=gpu)
    cfg = _config(G, "bf16")
    assert ffe.ff_workspace_size(cfg) > ffe.FF_NOALLOC_SCRATCH_BYTES
    with pytest.raises(ffe.FlipFlopError) as ei:
        ffe.ff_fit_noalloc(cfg, 1, A.data_ptr(), A.data_ptr())
    assert ei.value.code == ffe.FF_ERR_WORKSPACE
    assert "bytes of scratch" in str(ei.value)
