"""fp64 CPU oracle for the FlipFlop Hessian estimate.

TEST INFRASTRUCTURE ONLY.  This package is the slow, plain reference that the
GPU path is checked against.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import it; the product path (the HIP
library and its Python binding) never does, and shares no code with it.

Every function cites the passage of the paper it follows.  Where the paper
leaves a choice open, the reading taken is stated in the docstring.
"""
from .flipflop import (FlipFlopResult, NotSPDError, as_f64_samples, half_step_B, half_step_B_rows,
                       half_step_A, half_step_A_rows, normalise, damp, flipflop, loglik, objective)
from .metrics import kron_rel_error, kron_rel_error_scale_free, trace_identity
from .kron import kron_apply, mismatch_factor
from .waterkron import (rev_cholesky, normalised_inverse, waterfilling_scales, gptq,
                        two_sided_gptq, distortion)
from .variants import (frobenius, frobenius_tokens, frob_half_step_A, frob_half_step_B,
                       marginal_tokens, input_tokens)
from .tokens import (half_step_A_tokens, half_step_B_tokens, half_step_B_tokens_rows, flipflop_tokens, loglik_tokens,
                     objective_tokens, materialise, token_weights)

__all__ = ["FlipFlopResult", "NotSPDError", "as_f64_samples", "half_step_B", "half_step_B_rows",
           "half_step_A", "half_step_A_rows", "normalise", "damp", "flipflop", "loglik", "objective",
           "kron_rel_error", "kron_rel_error_scale_free", "trace_identity",
           "kron_apply", "mismatch_factor", "half_step_A_tokens", "half_step_B_tokens", "half_step_B_tokens_rows",
           "flipflop_tokens", "loglik_tokens", "objective_tokens", "materialise", "token_weights",
           "rev_cholesky", "normalised_inverse", "waterfilling_scales", "gptq", "two_sided_gptq",
           "distortion", "frobenius", "frobenius_tokens", "frob_half_step_A", "frob_half_step_B",
           "marginal_tokens", "input_tokens"]
