"""Seeded synthetic inputs for session-prefill attention.

This module is shared by the tests, the bench and the oracle harness.  It
holds only input generation: random draws, bf16 rounding of those draws,
sequence lengths, page permutations and block tables.  It contains none of
the attention arithmetic, so the oracle and the HIP path can both consume
its output without sharing any of the method's computation.

Workload shapes follow the paper's trace statistics (Section 2.1, "Continuation
inputs": median prompt 25K tokens, p95 105K) and the five synthetic
configurations named in the module-level ``CONFIGS`` table.
"""
from .gen import (  # noqa: F401
    BF16_NAN,
    CONFIGS,
    Workload,
    bf16_bits_from_f32,
    f32_from_bf16_bits,
    lognormal_prefix_lengths,
    make_workload,
    workload_from_lengths,
)
