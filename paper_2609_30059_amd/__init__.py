"""libfusedsub for MI355X (gfx950): fused pointwise chains, row softmax,
LayerNorm / RMSNorm + residual, row sum/mean/max/argmax and GEMM epilogue +
row reduction as hand-written HIP kernels behind a C ABI, with the GEMMs kept
as hipBLASLt library calls.

The native libraries are loaded on first use; a missing or unloadable
library raises ``NativeLibraryError`` -- there is no CPU fallback.
"""
from ._native import (FS_LAYERNORM_MAX_COLS, FS_SOFTMAX_MAX_COLS, FusedSubError,  # noqa: F401
                      GemmError, NativeLibraryError)
from .ops import (as_rows, causal_softmax_trimmed, copy_, copy_strided, gemm, gemm_epilogue_reduce, gemm_strided_batched,  # noqa: F401
                  layernorm_residual, pointwise_chain, pointwise_program, rmsnorm_residual,
                  row_argmax, row_reduce, row_softmax)
from .block import TransformerBlock  # noqa: F401

__version__ = "0.1.0"
