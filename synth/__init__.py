"""Seeded synthetic inputs for the FlipFlop Hessian estimate.

This module only *draws* inputs: samples ``G_i`` of a matrix-normal law
``Cov(vec G) = A (x) B`` (column-major ``vec``, Section 2 notation and
Section 5), with known SPD factors, plus an optional per-sample low-rank
term that breaks the Kronecker structure.  It contains none of the
estimation arithmetic (no factorisation, solve, whitening or second
moment of the samples).  Both the fp64 oracle and the GPU path read the
same stored values drawn here.

The paper calibrates on LLM layers (256 x 2048 tokens of a public text
corpus, gradients of real models; Appendix B).  Neither the weights nor the
data are available here, so these draws stand in for them at the layer
shapes of the workloads below.  ``tokens`` draws the per-token form instead
(inputs x_t and output gradients g_t, samples G_t = g_t x_t^T); ``quant``
draws the weights and factors the WaterKron quantiser consumes.
"""
from .generator import (WORKLOADS, Workload, workload, generate, generate_device,
                        power_law_spectrum, haar_orthogonal, f32_to_bf16_bits,
                        bf16_bits_to_f32, sample_digests, basis_digest, spd_start)
from .tokens import (TOKEN_WORKLOADS, TokenWorkload, token_workload, generate_tokens,
                     generate_tokens_device)
from .quant import QUANT_WORKLOADS, QuantWorkload, quant_workload, generate_quant

__all__ = ["WORKLOADS", "Workload", "workload", "generate", "generate_device",
           "power_law_spectrum", "haar_orthogonal", "f32_to_bf16_bits",
           "bf16_bits_to_f32", "sample_digests", "basis_digest", "spd_start", "TOKEN_WORKLOADS", "TokenWorkload", "token_workload",
           "generate_tokens", "generate_tokens_device", "QUANT_WORKLOADS", "QuantWorkload",
           "quant_workload", "generate_quant"]
