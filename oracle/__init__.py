"""Float64 CPU oracle of the fused sub-kernels and the stitched block.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  The library's
product path (``paper_2609_30059_amd``) never imports it and shares no code
with it; the two meet only through the seeded inputs of ``fusedsub_data``.

Parity status: every function here is pinned by the CPU tests
``tests/test_oracle_*.py`` to closed forms, invariants, special cases and
printed reference values (``tests/golden/``).
"""
from .subkernels import (ACTS, apply_act, byte_mask_additive, causal_mask, causal_written_width, gelu_erf, gemm_epilogue_reduce,
                         layernorm_residual, pointwise_chain, pointwise_program, PROGRAM_OPS, relu, residual_store_bf16,
                         rmsnorm_residual, round_to_bf16, row_argmax, row_reduce, row_softmax,
                         sigmoid, strided_copy)
from .block import block_forward, block_forward_sequence, STAGES

__all__ = [
    "ACTS", "apply_act", "byte_mask_additive", "causal_mask", "causal_written_width", "gelu_erf", "gemm_epilogue_reduce",
    "layernorm_residual", "pointwise_chain", "pointwise_program", "PROGRAM_OPS", "relu", "residual_store_bf16",
    "rmsnorm_residual", "row_reduce", "row_argmax",
    "round_to_bf16", "row_softmax", "sigmoid", "strided_copy", "block_forward",
    "block_forward_sequence", "STAGES",
]
