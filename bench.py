"""Benchmark of the FlipFlop Hessian engine on one MI355X.

A step is one flip-flop iteration (Section 5): both whitening passes, both
symmetric products and reductions, both Cholesky + inverse factorisations,
the trace normalisation and the log-likelihood.  The timed region is one
whole job: ff_init on the device-resident samples (internal transposed copy)
followed by ff_iterate over `--steps` iterations, bracketed by stream
synchronisation; the value is iterations per second of that job.

Prints one JSON line.  The per-kernel durations come from HIP events
recorded by the library on its stream inside the timed region; the CPU
baseline times the fp64 oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "flip-flop iter/s + TFLOP/s (% bf16 MFMA peak), m=n=4096, N=128"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_attn-4096x4096-N128.md")
KERNEL_SRC = os.path.join(ROOT, "paper_2609_14706_amd", "csrc", "ff_gemm_bf16.hip")


def recorded_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed counter summary, or
    None when none was taken for that kernel/workload or the kernel source
    has changed since."""
    import hashlib
    if workload != "attn-4096x4096-N128" or not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    for line in open(TRAFFIC_FILE):
        if "=" in line and line.startswith("traffic_"):
            k, v = line.strip().split("=", 1)
            kv[k] = v
    src = hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()
    key = f"traffic_{kernel}_bytes_per_launch"
    if key not in kv or kv.get("traffic_source_sha256") != src:
        return None
    return int(kv[key])


PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}


def host_description() -> str:
    """The host the oracle ran on: CPU model, logical CPUs, BLAS library."""
    from threadpoolctl import threadpool_info
    model = "unknown CPU"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    blas = sorted({f"{i.get('internal_api')} {i.get('version') or ''}".strip()
                   for i in threadpool_info() if i.get("user_api") == "blas"}) or ["unknown BLAS"]
    return f"{model}, {os.cpu_count()} logical CPUs, {', '.join(blas)}"


def cpu_baseline(G, w, budget_s: float, estimator: str = "flipflop"):
    """Oracle time of one iteration, from a bounded number of samples.

    Both half steps are timed on the first k samples (k grows until the
    budget is used), each against a fixed SPD factor (the per-sample cost of
    a Cholesky solve does not depend on its values); an iteration over all N
    samples costs N/k times that, the two Cholesky factorisations being
    negligible next to the per-sample solves and products.
    """
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    import oracle

    In = np.eye(w.n)
    Im = np.eye(w.m)
    t_total = 0.0
    k = 0
    host = []
    while k < w.N and (t_total < budget_s or k < 1):
        Gi = G[k:k + 1]
        if Gi.dtype == torch.bfloat16:
            host.append(Gi.view(torch.int16).cpu().numpy().view(np.uint16))
        else:
            host.append(Gi.cpu().numpy())
        Gs = np.concatenate(host)
        t0 = time.perf_counter()
        Gk = oracle.as_f64_samples(Gs[-1:])
        if estimator == "frobenius":
            oracle.frob_half_step_B(Gk, In)
            oracle.frob_half_step_A(Gk, Im)
        else:
            oracle.half_step_B(Gk, In)
            oracle.half_step_A(Gk, Im)
        t_total += time.perf_counter() - t0
        k += 1
    per_iter = t_total / k * w.N
    threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"]
                  or [1])
    return {"value": 1.0 / per_iter, "unit": "iter/s", "cores": int(threads), "kind": "oracle",
            "sample": f"both fp64 {estimator} half steps (direct form) on {k} of {w.N} samples "
                      f"of {w.name}, {t_total:.1f} s, scaled to a full iteration ({per_iter:.1f} s)"}


def cpu_baseline_tokens(x, g, w, budget_s: float, estimator: str = "flipflop"):
    """Oracle time of one iteration of the per-token form, from a bounded
    number of tokens: both half steps on the first k tokens (k grows in
    blocks of 4096 until the budget is used), against fixed SPD factors,
    scaled by T / k."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    import oracle

    In, Im = np.eye(w.n), np.eye(w.m)
    k, t_total = 0, 0.0
    while k < w.T and (t_total < budget_s or k == 0):
        kb = min(4096, w.T - k)
        xs = x[k:k + kb].view(torch.int16).cpu().numpy().view(np.uint16) if x.dtype == torch.bfloat16 \
            else x[k:k + kb].cpu().numpy()
        gs = g[k:k + kb].view(torch.int16).cpu().numpy().view(np.uint16) if g.dtype == torch.bfloat16 \
            else g[k:k + kb].cpu().numpy()
        t0 = time.perf_counter()
        if estimator == "marginal":
            oracle.marginal_tokens(xs, gs)
        elif estimator == "input":
            oracle.input_tokens(xs, w.m)
        elif estimator == "frobenius":
            oracle.frobenius_tokens(xs, gs, 1)
        else:
            oracle.half_step_B_tokens(xs, gs, In)
            oracle.half_step_A_tokens(xs, gs, Im)
        t_total += time.perf_counter() - t0
        k += kb
    per_iter = t_total * w.T / k
    cores = max((i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"),
                default=1)
    return {"value": 1.0 / per_iter, "unit": "iter/s", "cores": cores, "kind": "oracle",
            "sample": f"fp64 {estimator} estimate (rank-one form) on {k} of {w.T} tokens of {w.name}, "
                      f"{t_total:.1f} s, scaled to a full iteration ({per_iter:.1f} s)"}


def cpu_baseline_quant(w, budget_s: float):
    """Oracle time of Algorithm 2 on the layer, from bounded sub-problems.

    The oracle updates the whole m x n matrix after every entry, so its time
    grows as (m n)^2; it is timed on the leading k x k blocks of a 256 x 256
    instance of the workload's recipe (k doubling until the budget is used)
    and scaled to m x n by that law.  Its updates are numpy elementwise
    operations, which run on one thread.
    """
    import numpy as np
    import oracle
    import synth
    d = synth.generate_quant(w.scaled(m=min(w.m, 256), n=min(w.n, 256)))
    k, used, last = 16, 0.0, None
    while k <= min(w.m, w.n, 256) and used < budget_s:
        W = d.W[:k, :k].astype(np.float64)
        A = d.A[:k, :k].astype(np.float64)
        B = d.B[:k, :k].astype(np.float64)
        al, be = oracle.waterfilling_scales(A, B, w.gamma)
        t0 = time.perf_counter()
        oracle.two_sided_gptq(W, A, B, al, be)
        dt = time.perf_counter() - t0
        used += dt
        last = (k, dt)
        k *= 2
    k, dt = last
    per_layer = dt * (w.m * w.n / float(k * k)) ** 2
    return {"value": 1.0 / per_layer, "unit": "quantisations/s", "cores": 1, "kind": "oracle",
            "sample": f"fp64 Algorithm 2 on the leading {k}x{k} block of a 256x256 instance "
                      f"({dt:.2f} s), scaled to {w.m}x{w.n} by the oracle's (m n)^2 cost law"}


def main_quant(args):
    """A step is one whole WaterKron quantisation of the layer (ff_quantize):
    both reverse Cholesky factorisations, the waterfilling scales, the
    anti-diagonal sweep of Algorithm 2, the grid values and the distortion."""
    import torch
    import synth
    import paper_2609_14706_amd as ffe

    dev = torch.device("cuda:0")
    w = synth.quant_workload(args.workload)
    d = synth.generate_quant(w, seed=args.seed)
    W = torch.from_numpy(d.W).to(dev)
    A = torch.from_numpy(d.A).to(dev)
    B = torch.from_numpy(d.B).to(dev)
    G = torch.zeros((1, w.m, w.n), dtype=torch.float32, device=dev)
    G[0, 0, 0] = 1.0
    stream = torch.cuda.current_stream(dev)
    h = ffe.FlipFlop(G, stream=stream)
    ws = torch.empty(h.quantize_workspace_bytes(w.m, w.n), dtype=torch.uint8, device=dev)
    for _ in range(args.warmup):
        h.quantize(W, A, B, gamma=w.gamma, workspace=ws)
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} quantisations of {w.name})", file=sys.stderr,
          flush=True)
    h.set_timing(True)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        Z, V, al, be, D = h.quantize(W, A, B, gamma=w.gamma, workspace=ws)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_total = ev0.elapsed_time(ev1)
    n_d, ms_d, fl_d = h.kernel_timing("quant_diag")
    n_c, ms_c, _ = h.kernel_timing("cholinv")
    h.close()
    ms_per_step = ms_total / args.steps
    achieved = fl_d / (ms_d * 1e-3) / 1e12 if ms_d > 0 else 0.0
    print(f"[bench] {args.steps} quantisations in {ms_total:.2f} ms; sweep {n_d} launches "
          f"{ms_d:.2f} ms, factorisations {n_c} x {ms_c / max(n_c, 1):.3f} ms, D = {D:.6e}",
          file=sys.stderr, flush=True)
    peak = PEAK_TFLOPS["f32"]
    out = {
        "metric": f"WaterKron quantisations/s (two-sided GPTQ, waterfilling scales), "
                  f"m={w.m} n={w.n}",
        "value": round(1000.0 / ms_per_step, 4),
        "unit": "quantisations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "m": w.m, "n": w.n, "gamma": w.gamma,
                   "timed_job": f"{args.steps} x ff_quantize"},
        "weights_per_s": round(w.m * w.n * 1000.0 / ms_per_step, 1),
        "distortion": D,
        "kernels_ms": {"quant_diag": round(ms_d, 3), "cholinv": round(ms_c, 3)},
        "roofline": {"bound": "mfma", "kernel": "k_wk_diagonal",
                     "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 5), "traffic": None,
                     "launches": n_d, "avg_launch_ms": round(ms_d / max(n_d, 1), 4),
                     "alg_flop_per_launch": fl_d / max(n_d, 1)},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the fp64 oracle on host cores", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline_quant(w, args.cpu_budget)
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10, help="timed flip-flop iterations")
    ap.add_argument("--warmup", type=int, default=2, help="untimed iterations on the timed handle before the timed ones")
    ap.add_argument("--workload", default="attn",
                    help="tiny | attn | mlp_up | mlp_down | mlp_large | tokens_tiny | tokens_attn"
                         " | quant_small | quant_multi | quant_attn")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--whiten-split", type=int, default=0,
                    help="0 = automatic (per factorisation), 1 = one bf16 pass, 2 = hi + lo passes")
    ap.add_argument("--estimator", default="flipflop",
                    help="flipflop | frobenius | marginal | input (Table 1; the last two need tokens)")
    ap.add_argument("--damping", type=float, default=0.0, help="kappa (Appendix B damping)")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle time")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the FlipFlop engine is a single-GPU build "
              "(sharding over samples is described in the design notes, not built).",
              file=sys.stderr)
        sys.exit(2)

    if args.gpus == 1 and not args.no_cpu_baseline:
        import oracle  # noqa: F401  (its set-up starts a child process: before the GPU is in use)

    if args.workload.startswith("quant"):
        return main_quant(args)

    import torch

    import synth
    import paper_2609_14706_amd as ffe

    dev = torch.device("cuda:0")
    tokens = args.workload.startswith("tokens")
    t0 = time.perf_counter()
    if tokens:
        w = synth.token_workload(args.workload)
        x, g = synth.generate_tokens_device(w, seed=args.seed, device=dev)
        src = {"tokens": (x, g)}
        nbytes_in = (x.numel() + g.numel()) * x.element_size()
        N = w.T
    else:
        w = synth.workload(args.workload)
        G = synth.generate_device(w, seed=args.seed, device=dev)
        src = {"G": G}
        nbytes_in = G.numel() * G.element_size()
        N = w.N
    torch.cuda.synchronize()
    print(f"[bench] generated {w.name} ({nbytes_in / 1e9:.2f} GB) in "
          f"{time.perf_counter() - t0:.1f} s", file=sys.stderr, flush=True)
    nbytes = ffe.FlipFlop.workspace_bytes(w.m, w.n, N, w.dtype, args.whiten_split, rank1=tokens)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)

    # One handle: the warm-up iterations (at least one) run untimed on it, so
    # the timed window holds only steady-state iterations (the first
    # iteration from the identity start skips one whitening and one
    # factorisation, and ff_init's transposed sample copy is set-up).
    f = ffe.FlipFlop(**src, whiten_split=args.whiten_split, workspace=ws, stream=stream,
                     estimator=args.estimator, damping=args.damping)
    warm = max(1, args.warmup)
    f.iterate(warm)
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({warm} iterations on the timed handle)", file=sys.stderr, flush=True)

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    f.set_timing(True)
    torch.cuda.synchronize()
    ev0.record(stream)
    ll = f.iterate(args.steps)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_total = ev0.elapsed_time(ev1)
    kern = {k: f.kernel_timing(k) for k in ("whiten", "syrk", "reduce", "cholinv")}
    f.close()
    ms_per_step = ms_total / args.steps
    iters_per_s = 1000.0 / ms_per_step
    flop_iter = w.flop_per_iter
    if args.estimator in ("marginal", "input"):   # token means: symmetric products only
        flop_iter = float(w.T) * (w.n * w.n + (w.m * w.m if args.estimator == "marginal" else 0))
    tflops = flop_iter / (ms_per_step * 1e-3) / 1e12
    peak = PEAK_TFLOPS[w.dtype]
    print(f"[bench] {args.steps} iterations in {ms_total:.2f} ms; kernels: " +
          ", ".join(f"{k}: {n} x {ms / max(n, 1):.3f} ms" for k, (n, ms, _) in kern.items()),
          file=sys.stderr, flush=True)

    dom = max(("whiten", "syrk"), key=lambda k: kern[k][1])
    n_l, ms_l, fl_l = kern[dom]
    achieved = fl_l / (ms_l * 1e-3) / 1e12 if ms_l > 0 else 0.0
    wname = "k_whiten_norm_bf16" if tokens else "k_whiten_bf16"
    roofline = {"bound": "mfma", "kernel": {"whiten": wname, "syrk": "k_syrk_bf16"}[dom]
                if w.dtype == "bf16" else "k_gemm_f32",
                "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": None,
                "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-scaled)",
                "launches": n_l, "avg_launch_ms": round(ms_l / max(n_l, 1), 4),
                "alg_flop_per_launch": fl_l / max(n_l, 1)}

    if w.dtype == "bf16":
        roofline["traffic"] = recorded_traffic(roofline["kernel"], w.name)
    flipflop = args.estimator == "flipflop"
    if flipflop:
        if tokens:
            metric = f"flip-flop iter/s + TFLOP/s, per-token form, m={w.m} n={w.n} T={w.T}"
        elif w.name == "attn-4096x4096-N128":
            metric = METRIC
        else:
            metric = f"flip-flop iter/s + TFLOP/s (% bf16 MFMA peak), m={w.m}, n={w.n}, N={N}"
    else:
        metric = (f"{args.estimator} estimator iter/s, m={w.m} n={w.n} " +
                  (f"T={w.T}" if tokens else f"N={N}"))
    out = {
        "metric": metric,
        "value": round(iters_per_s, 4),
        "unit": "iter/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "m": w.m, "n": w.n, ("T" if tokens else "N"): N,
                   "timed_job": f"{args.steps} iterations after {warm} untimed on the same handle",
                   "whiten_split": {0: "auto", 1: 1, 2: 2}[args.whiten_split], "estimator": args.estimator,
                   "damping": args.damping},
        "tflops": round(tflops, 2),
        "pct_peak": round(100.0 * tflops / peak, 2),
        "alg_flop_per_iter": flop_iter,
        "loglik_last": ll[-1] if ll and args.estimator == "flipflop" else None,
        "kernels_ms": {k: round(ms, 3) for k, (n, ms, _) in kern.items()},
        "roofline": roofline,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the fp64 oracle on host cores", file=sys.stderr, flush=True)
        cb = (cpu_baseline_tokens(x, g, w, args.cpu_budget, args.estimator)
              if tokens else cpu_baseline(G, w, args.cpu_budget, args.estimator))
        # algorithmic rate of the oracle (its direct form executes about twice F_alg)
        cb["alg_gflops"] = round(cb["value"] * flop_iter / 1e9, 2)
        cb["host"] = host_description()
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
