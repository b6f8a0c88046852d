"""ctypes binding of libff.so (include/ff.h): argument marshalling only.

Every step of the estimate runs in the HIP library; torch supplies device
memory (the samples, the workspace, outputs) and the stream.  If the library
is not built this module raises at first use: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libff.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "ff.h")

FF_OK, FF_ERR_INVALID_ARG, FF_ERR_NOT_SPD, FF_ERR_WORKSPACE, FF_ERR_HIP, FF_ERR_STATE = range(6)
FF_F32, FF_BF16 = 0, 1
FF_ORDER_B_FIRST, FF_ORDER_A_FIRST = 0, 1
FF_APPLY, FF_APPLY_INV = 0, 1
FF_SAMPLES_DENSE, FF_SAMPLES_RANK1 = 0, 1
FF_SCALES_WATERFILL, FF_SCALES_GIVEN = 0, 1
FF_EST_FLIPFLOP, FF_EST_FROBENIUS, FF_EST_MARGINAL, FF_EST_INPUT = 0, 1, 2, 3
FF_HALF_B, FF_HALF_A = 0, 1
FF_NOALLOC_SCRATCH_BYTES = 64 << 20   # include/ff.h
ESTIMATORS = {"flipflop": FF_EST_FLIPFLOP, "frobenius": FF_EST_FROBENIUS,
              "marginal": FF_EST_MARGINAL, "input": FF_EST_INPUT}
KERNEL_IDS = {"whiten": 0, "syrk": 1, "reduce": 2, "cholinv": 3, "quant_diag": 4}


class ff_config(ctypes.Structure):
    _fields_ = [
        ("m", ctypes.c_int64),
        ("n", ctypes.c_int64),
        ("N", ctypes.c_int64),
        ("dtype", ctypes.c_int),
        ("G", ctypes.c_void_p),
        ("stream", ctypes.c_void_p),
        ("order", ctypes.c_int),
        ("damping", ctypes.c_double),
        ("A0", ctypes.c_void_p),
        ("B0", ctypes.c_void_p),
        ("whiten_split", ctypes.c_int),
        ("workspace", ctypes.c_void_p),
        ("workspace_bytes", ctypes.c_size_t),
        ("form", ctypes.c_int),
        ("x", ctypes.c_void_p),
        ("g", ctypes.c_void_p),
        ("estimator", ctypes.c_int),
    ]


_LIB = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libff.so once and declare the signatures of ff.h."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2609_14706_amd.build`"
                           " (the FlipFlop engine has no fallback path)")
    lib = ctypes.CDLL(path)
    H = ctypes.c_void_p
    st = ctypes.c_int
    sig = {
        "ff_workspace_size": (st, [ctypes.POINTER(ff_config), ctypes.POINTER(ctypes.c_size_t)]),
        "ff_init": (st, [ctypes.POINTER(ff_config), ctypes.POINTER(H)]),
        "ff_iterate": (st, [H, ctypes.c_int, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_double)]),
        "ff_iterate_tol": (st, [H, ctypes.c_int, ctypes.c_double, ctypes.POINTER(ctypes.c_int),
                                ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
        "ff_half_step": (st, [H, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]),
        "ff_fit_noalloc": (st, [ctypes.POINTER(ff_config), ctypes.c_int, ctypes.POINTER(ctypes.c_int),
                                ctypes.POINTER(ctypes.c_double), ctypes.c_void_p, ctypes.c_void_p]),
        "ff_factors": (st, [H, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]),
        "ff_kron_apply": (st, [H, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int]),
        "ff_objective": (st, [H, ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)]),
        "ff_quantize_workspace_size": (st, [ctypes.c_int64, ctypes.c_int64,
                                            ctypes.POINTER(ctypes.c_size_t)]),
        "ff_quantize": (st, [H, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_double,
                             ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                             ctypes.c_void_p, ctypes.POINTER(ctypes.c_double), ctypes.c_void_p,
                             ctypes.c_size_t]),
        "ff_destroy": (st, [H]),
        "ff_whiten_split_state": (st, [H, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int)]),
        "ff_set_timing": (st, [H, ctypes.c_int]),
        "ff_kernel_timing": (st, [H, ctypes.c_int, ctypes.POINTER(ctypes.c_int64),
                                  ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
        "ff_status_string": (ctypes.c_char_p, [st]),
        "ff_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _LIB = lib
    return lib


def header_functions(path: str = HEADER) -> list[str]:
    """Names of the functions ff.h declares."""
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ff_\w+)\s*\(", text)))


class FlipFlopError(RuntimeError):
    def __init__(self, code: int, msg: str, iters_done: int = 0):
        super().__init__(f"{ff_status_string(code)}: {msg}")
        self.code = code
        self.iters_done = iters_done


def ff_status_string(code: int) -> str:
    return load_library().ff_status_string(code).decode()


def ff_last_error() -> str:
    return load_library().ff_last_error().decode()


def _check(code: int, iters_done: int = 0):
    if code != FF_OK:
        raise FlipFlopError(code, ff_last_error(), iters_done)


# ------------------------------------------------------------ thin wrappers
def ff_workspace_size(cfg: ff_config) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().ff_workspace_size(ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def ff_init(cfg: ff_config) -> ctypes.c_void_p:
    h = ctypes.c_void_p()
    _check(load_library().ff_init(ctypes.byref(cfg), ctypes.byref(h)))
    return h


def ff_iterate(h, iters: int, want_loglik: bool = True):
    done = ctypes.c_int(0)
    ll = (ctypes.c_double * max(iters, 1))() if want_loglik else None
    code = load_library().ff_iterate(h, iters, ctypes.byref(done), ll)
    lls = list(ll[:done.value]) if ll is not None else []
    if code != FF_OK:
        err = FlipFlopError(code, ff_last_error(), done.value)
        err.loglik = lls
        raise err
    return done.value, lls


def ff_iterate_tol(h, max_iters: int, tol: float):
    """(iterations done, log-likelihoods, relative changes of A (x) B)."""
    done = ctypes.c_int(0)
    ll = (ctypes.c_double * max(max_iters, 1))()
    dl = (ctypes.c_double * max(max_iters, 1))()
    code = load_library().ff_iterate_tol(h, max_iters, float(tol), ctypes.byref(done), ll, dl)
    lls, dls = list(ll[:done.value]), list(dl[:done.value])
    if code != FF_OK:
        err = FlipFlopError(code, ff_last_error(), done.value)
        err.loglik, err.delta = lls, dls
        raise err
    return done.value, lls, dls


def ff_half_step(h, which: int, F_ptr, out_ptr):
    _check(load_library().ff_half_step(h, which, F_ptr, out_ptr))


def ff_fit_noalloc(cfg: ff_config, iters: int, A_ptr, B_ptr):
    """(iterations done, log-likelihoods); cfg.workspace is ignored."""
    done = ctypes.c_int(0)
    ll = (ctypes.c_double * max(iters, 1))()
    code = load_library().ff_fit_noalloc(ctypes.byref(cfg), iters, ctypes.byref(done), ll, A_ptr,
                                         B_ptr)
    lls = list(ll[:done.value])
    if code != FF_OK:
        err = FlipFlopError(code, ff_last_error(), done.value)
        err.loglik = lls
        raise err
    return done.value, lls


def ff_factors(h, A_ptr: int, B_ptr: int, on_host: int):
    _check(load_library().ff_factors(h, A_ptr, B_ptr, on_host))


def ff_kron_apply(h, X_ptr: int, Y_ptr: int, batch: int, mode: int):
    _check(load_library().ff_kron_apply(h, X_ptr, Y_ptr, batch, mode))


def ff_objective(h, A_ptr, B_ptr) -> float:
    out = ctypes.c_double(0.0)
    _check(load_library().ff_objective(h, A_ptr, B_ptr, ctypes.byref(out)))
    return out.value


def ff_quantize_workspace_size(m: int, n: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().ff_quantize_workspace_size(m, n, ctypes.byref(out)))
    return out.value


def ff_quantize(h, W_ptr, A_ptr, B_ptr, gamma: float, mode: int, alpha_ptr, beta_ptr, Z_ptr,
                V_ptr, ws_ptr, ws_bytes: int) -> float:
    out = ctypes.c_double(0.0)
    _check(load_library().ff_quantize(h, W_ptr, A_ptr, B_ptr, float(gamma), mode, alpha_ptr,
                                      beta_ptr, Z_ptr, V_ptr, ctypes.byref(out), ws_ptr, ws_bytes))
    return out.value


def ff_destroy(h):
    _check(load_library().ff_destroy(h))


def ff_whiten_split_state(h):
    sA, sB = ctypes.c_double(), ctypes.c_double()
    pA, pB = ctypes.c_int(), ctypes.c_int()
    _check(load_library().ff_whiten_split_state(h, ctypes.byref(sA), ctypes.byref(sB),
                                                 ctypes.byref(pA), ctypes.byref(pB)))
    return sA.value, sB.value, pA.value, pB.value


def ff_set_timing(h, enable: bool):
    _check(load_library().ff_set_timing(h, 1 if enable else 0))


def ff_kernel_timing(h, kernel: int):
    n = ctypes.c_int64(0)
    ms = ctypes.c_double(0)
    fl = ctypes.c_double(0)
    _check(load_library().ff_kernel_timing(h, kernel, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(fl)))
    return n.value, ms.value, fl.value


# --------------------------------------------------------------- torch API
class FlipFlop:
    """FlipFlop Hessian estimate A (x) B of samples G (N, m, n) on the GPU.

    G: contiguous CUDA tensor, float32 or bfloat16.  The handle borrows G
    and keeps it alive; the workspace is a torch uint8 tensor on G's device.
    """

    def __init__(self, G=None, *, tokens=None, order: str = "B_FIRST", damping: float = 0.0,
                 A0=None, B0=None, whiten_split: int = 0, stream=None, workspace=None,
                 estimator: str = "flipflop"):
        """G: (N, m, n) samples; or tokens = (x, g) with x (N, n) inputs and
        g (N, m) output gradients, the samples being G_t = g_t x_t^T (the
        rank-one form; both tensors of one dtype).  estimator: "flipflop",
        "frobenius", "marginal" or "input" (Table 1; the last two need
        tokens).  whiten_split (bf16 samples): 0 = automatic per
        factorisation, 1 = one bf16 pass, 2 = hi + lo passes."""
        import torch
        if (G is None) == (tokens is None):
            raise ValueError("give either G or tokens=(x, g)")
        if tokens is not None:
            x, g = tokens
            for name, T in (("x", x), ("g", g)):
                if not isinstance(T, torch.Tensor) or not T.is_cuda:
                    raise TypeError(f"{name} must be a CUDA tensor")
                if T.dim() != 2 or not T.is_contiguous():
                    raise ValueError(f"{name} must be a contiguous (N, dim) tensor")
            if x.shape[0] != g.shape[0] or x.dtype != g.dtype or x.device != g.device:
                raise ValueError("x and g must have the same N, dtype and device")
            ref, (N, n), m = x, x.shape, g.shape[1]
            form = FF_SAMPLES_RANK1
        else:
            if not isinstance(G, torch.Tensor) or not G.is_cuda:
                raise TypeError("G must be a CUDA tensor")
            if G.dim() != 3 or not G.is_contiguous():
                raise ValueError("G must be a contiguous (N, m, n) tensor")
            ref = G
            N, m, n = G.shape
            form = FF_SAMPLES_DENSE
        if ref.dtype == torch.bfloat16:
            dt = FF_BF16
        elif ref.dtype == torch.float32:
            dt = FF_F32
        else:
            raise TypeError("samples must be float32 or bfloat16")
        self.device = ref.device
        self.stream = stream if stream is not None else torch.cuda.current_stream(ref.device)
        self.m, self.n, self.N = int(m), int(n), int(N)
        cfg = ff_config()
        cfg.m, cfg.n, cfg.N = self.m, self.n, self.N
        cfg.dtype = dt
        cfg.form = form
        cfg.estimator = ESTIMATORS[estimator]
        if form == FF_SAMPLES_RANK1:
            self._keep = [x, g]
            cfg.x, cfg.g = x.data_ptr(), g.data_ptr()
        else:
            self._keep = [G]
            cfg.G = G.data_ptr()
        G = ref
        cfg.stream = self.stream.cuda_stream
        cfg.order = {"B_FIRST": FF_ORDER_B_FIRST, "A_FIRST": FF_ORDER_A_FIRST}[order]
        cfg.damping = float(damping)
        for name, T, dim in (("A0", A0, self.n), ("B0", B0, self.m)):
            if T is not None:
                T = T.to(device=G.device, dtype=torch.float32).contiguous()
                if T.shape != (dim, dim):
                    raise ValueError(f"{name} must be {dim} x {dim}")
                self._keep.append(T)
                setattr(cfg, name, T.data_ptr())
        cfg.whiten_split = int(whiten_split)
        nbytes = ff_workspace_size(cfg)
        if workspace is not None:
            if (workspace.device != G.device or workspace.dtype != torch.uint8
                    or workspace.numel() < nbytes + 256):
                raise ValueError(f"workspace must be a uint8 tensor of >= {nbytes + 256} bytes on {G.device}")
            self.workspace = workspace
        else:
            with torch.cuda.device(G.device):
                self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=G.device)
        base = self.workspace.data_ptr()
        cfg.workspace = (base + 255) // 256 * 256
        cfg.workspace_bytes = nbytes
        self.cfg = cfg
        self.h = ff_init(cfg)
        self.iters_done = 0

    @staticmethod
    def workspace_bytes(m: int, n: int, N: int, dtype: str = "bf16", whiten_split: int = 0,
                        rank1: bool = False) -> int:
        """Bytes a caller-provided workspace tensor needs (alignment slack included)."""
        cfg = ff_config()
        cfg.m, cfg.n, cfg.N = m, n, N
        cfg.form = FF_SAMPLES_RANK1 if rank1 else FF_SAMPLES_DENSE
        cfg.dtype = FF_BF16 if dtype == "bf16" else FF_F32
        cfg.whiten_split = whiten_split
        return ff_workspace_size(cfg) + 256

    def iterate(self, iters: int):
        """Run `iters` iterations; returns the per-iteration log-likelihoods."""
        try:
            done, ll = ff_iterate(self.h, int(iters))
        except FlipFlopError as e:
            self.iters_done += e.iters_done
            raise
        self.iters_done += done
        return ll

    def iterate_tol(self, max_iters: int, tol: float = 0.0):
        """Up to `max_iters` iterations, stopping after the first whose relative
        change of A (x) B is <= tol (tol = 0: never); returns
        (iterations done, log-likelihoods, relative changes); see ff_iterate_tol."""
        try:
            done, ll, dl = ff_iterate_tol(self.h, int(max_iters), tol)
        except FlipFlopError as e:
            self.iters_done += e.iters_done
            raise
        self.iters_done += done
        return done, ll, dl

    def half_step(self, which: str, F=None):
        """One unscaled, undamped half step with the other factor fixed:
        which = "B": (1/(N n)) sum_i G_i F^-1 G_i^T (F n x n, default the
        current A); which = "A": (1/(N m)) sum_i G_i^T F^-1 G_i (F m x m,
        default the current B).  Returns a new fp32 CUDA tensor."""
        import torch
        code, dim_out, dim_in = {"B": (FF_HALF_B, self.m, self.n),
                                 "A": (FF_HALF_A, self.n, self.m)}[which]
        keep = None
        pf = None
        if F is not None:
            keep = F.to(device=self.device, dtype=torch.float32).contiguous()
            if tuple(keep.shape) != (dim_in, dim_in):
                raise ValueError(f"F must be {dim_in} x {dim_in}")
            pf = keep.data_ptr()
        out = torch.empty((dim_out, dim_out), dtype=torch.float32, device=self.device)
        torch.cuda.current_stream(self.device).synchronize()
        ff_half_step(self.h, code, pf, out.data_ptr())
        del keep
        return out

    def factors(self):
        """(A, B) as new fp32 CUDA tensors, tr(A) = n."""
        import torch
        A = torch.empty((self.n, self.n), dtype=torch.float32, device=self.device)
        B = torch.empty((self.m, self.m), dtype=torch.float32, device=self.device)
        ff_factors(self.h, A.data_ptr(), B.data_ptr(), 0)
        self.stream.synchronize()
        return A, B

    def kron_apply(self, X, inverse: bool = False):
        """Y_b = B X_b A (or B^-1 X_b A^-1) for X of shape (batch, m, n)."""
        import torch
        X = X.to(device=self.device, dtype=torch.float32).contiguous()
        squeeze = X.dim() == 2
        if squeeze:
            X = X[None]
        if tuple(X.shape[1:]) != (self.m, self.n):
            raise ValueError("X must be (batch, m, n)")
        Y = torch.empty_like(X)
        ff_kron_apply(self.h, X.data_ptr(), Y.data_ptr(), X.shape[0],
                      FF_APPLY_INV if inverse else FF_APPLY)
        return Y[0] if squeeze else Y

    def objective(self, A=None, B=None) -> float:
        """log Phi(H, A (x) B) + log|H| / (m n) of the given factors (default:
        the current ones); see ff_objective."""
        import torch
        keep = []

        def ptr(M, dim):
            if M is None:
                return None
            M = M.to(device=self.device, dtype=torch.float32).contiguous()
            if tuple(M.shape) != (dim, dim):
                raise ValueError(f"factor must be {dim} x {dim}")
            keep.append(M)
            return M.data_ptr()
        pa, pb = ptr(A, self.n), ptr(B, self.m)
        torch.cuda.current_stream(self.device).synchronize()
        return ff_objective(self.h, pa, pb)

    def quantize(self, W, A=None, B=None, *, gamma=None, alpha=None, beta=None, workspace=None):
        """WaterKron quantisation of W (m, n): two-sided GPTQ (Algorithm 2)
        under A (x) B (default: the current factors).  Give either gamma (the
        Corollary 3.2 waterfilling scales are computed) or alpha (n) and
        beta (m).  Returns (Z int32, V fp32, alpha, beta, distortion D_{A,B});
        see ff_quantize."""
        import torch
        if (gamma is None) == (alpha is None or beta is None):
            raise ValueError("give either gamma or both alpha and beta")
        dev = self.device
        keep = []

        def dev32(M, shape, name):
            M = M.to(device=dev, dtype=torch.float32).contiguous()
            if tuple(M.shape) != shape:
                raise ValueError(f"{name} must have shape {shape}")
            keep.append(M)
            return M
        W = dev32(W, (self.m, self.n), "W")
        pa = None if A is None else dev32(A, (self.n, self.n), "A").data_ptr()
        pb = None if B is None else dev32(B, (self.m, self.m), "B").data_ptr()
        if gamma is None:
            al = dev32(alpha, (self.n,), "alpha").clone()
            be = dev32(beta, (self.m,), "beta").clone()
            mode, g = FF_SCALES_GIVEN, 0.0
        else:
            al = torch.empty(self.n, dtype=torch.float32, device=dev)
            be = torch.empty(self.m, dtype=torch.float32, device=dev)
            mode, g = FF_SCALES_WATERFILL, float(gamma)
        Z = torch.empty((self.m, self.n), dtype=torch.int32, device=dev)
        V = torch.empty((self.m, self.n), dtype=torch.float32, device=dev)
        nbytes = ff_quantize_workspace_size(self.m, self.n)
        if workspace is None:
            workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=dev)
        elif (workspace.device != dev or workspace.dtype != torch.uint8
              or workspace.numel() < nbytes + 256):
            raise ValueError(f"workspace must be a uint8 tensor of >= {nbytes + 256} bytes on {dev}")
        base = (workspace.data_ptr() + 255) // 256 * 256
        torch.cuda.current_stream(dev).synchronize()
        dist = ff_quantize(self.h, W.data_ptr(), pa, pb, g, mode, al.data_ptr(), be.data_ptr(),
                           Z.data_ptr(), V.data_ptr(), base, nbytes)
        return Z, V, al, be, dist

    @staticmethod
    def quantize_workspace_bytes(m: int, n: int) -> int:
        """Bytes a caller-provided quantiser workspace tensor needs (slack included)."""
        return ff_quantize_workspace_size(m, n) + 256

    def whiten_split_state(self):
        """(s_A, s_B, passes_A, passes_B) of the most recent whitening operands
        (automatic split; s is NaN where it was not computed)."""
        return ff_whiten_split_state(self.h)

    def set_timing(self, enable: bool = True):
        ff_set_timing(self.h, enable)

    def kernel_timing(self, kernel: str):
        """(launches, total ms, algorithmic flop) recorded since timing was enabled."""
        return ff_kernel_timing(self.h, KERNEL_IDS[kernel])

    def close(self):
        if getattr(self, "h", None):
            ff_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
