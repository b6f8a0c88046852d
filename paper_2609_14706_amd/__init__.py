"""FlipFlop Hessian estimation on AMD MI355X (gfx950).

Estimates the Kronecker-factored Hessian A (x) B of a linear layer from
gradient samples G_i with the flip-flop iteration (WaterKron and FlipFlop
Hessian, Section 5), and quantises its weights with WaterKron (two-sided
GPTQ with waterfilling scales, Section 3), entirely in the HIP library
``libff.so`` whose C ABI is ``include/ff.h``.  This package is the thin
binding (ctypes + torch memory).
"""
from .binding import (FF_APPLY, FF_APPLY_INV, FF_BF16, FF_ERR_HIP, FF_ERR_INVALID_ARG,
                      FF_ERR_NOT_SPD, FF_ERR_STATE, FF_ERR_WORKSPACE, FF_F32, FF_OK,
                      FF_ORDER_A_FIRST, FF_ORDER_B_FIRST, FF_SAMPLES_DENSE, FF_SAMPLES_RANK1,
                      FF_SCALES_GIVEN, FF_SCALES_WATERFILL, FF_EST_FLIPFLOP, FF_EST_FROBENIUS,
                      FF_EST_MARGINAL, FF_EST_INPUT, ESTIMATORS, FlipFlop, FlipFlopError, ff_config,
                      ff_destroy, ff_factors, ff_fit_noalloc, ff_half_step, ff_init, ff_iterate,
                      ff_iterate_tol, ff_kernel_timing, FF_HALF_A, FF_HALF_B, FF_NOALLOC_SCRATCH_BYTES,
                      ff_kron_apply, ff_last_error, ff_objective, ff_quantize,
                      ff_quantize_workspace_size, ff_set_timing, ff_status_string,
                      ff_whiten_split_state,
                      ff_workspace_size, header_functions, load_library, LIB_PATH)

__all__ = [n for n in dir() if not n.startswith("_")]
