"""ctypes binding of libfusedsub (include/fusedsub.h) and libfsgemm
(include/fsgemm.h).

The raw functions carry the C names and signatures unchanged (pointers and
the stream as integers).  The tensor helpers in ``ops.py`` only marshal
torch tensors into those arguments; every computation runs in the native
libraries.  There is no fallback: if a library is missing or fails to load,
an ImportError-like ``NativeLibraryError`` is raised.

torch is imported before the libraries are loaded, so the libraries bind to
the HIP runtime torch already mapped (same SONAME); a second runtime in the
process would make torch's stream handles invalid in ours.
"""
from __future__ import annotations

import ctypes
import os
import threading

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_FUSEDSUB = os.path.join(HERE, "libfusedsub.so")
LIB_FSGEMM = os.path.join(HERE, "libfsgemm.so")

# enums of fusedsub.h
FS_OK = 0
STATUS_NAMES = {0: "FS_OK", 1: "FS_ERR_NULL_POINTER", 2: "FS_ERR_BAD_SHAPE",
                3: "FS_ERR_BAD_STRIDE", 4: "FS_ERR_UNSUPPORTED_DTYPE", 5: "FS_ERR_ALIASING",
                6: "FS_ERR_BAD_ARGUMENT", 7: "FS_ERR_HIP"}
FS_F32, FS_BF16, FS_U8 = 0, 1, 2
ACTS = {"none": 0, "gelu_erf": 1, "sigmoid": 2, "relu": 3}
REDUCES = {"sum": 0, "mean": 1, "max": 2, "logsumexp": 3}
ROW_OPS = {"sum": 0, "mean": 1, "max": 2, "logsumexp": 3}
FS_ABI_VERSION = 2
FS_SOFTMAX_MAX_COLS = 16777216
FS_LAYERNORM_MAX_COLS = 16777216

# every symbol the headers declare
FUSEDSUB_SYMBOLS = ("fs_pointwise_chain", "fs_pointwise_program", "fs_row_softmax",
                    "fs_causal_softmax_trimmed",
                    "fs_layernorm_residual",
                    "fs_rmsnorm_residual", "fs_row_reduce", "fs_row_argmax",
                    "fs_gemm_epilogue_reduce", "fs_copy_strided", "fs_copy",
                    "fs_status_string",
                    "fs_last_error_message", "fs_abi_version")
FSGEMM_SYMBOLS = ("fsg_gemm_bf16", "fsg_gemm_bf16_ex", "fsg_last_error_message")


class NativeLibraryError(ImportError):
    pass


class FusedSubError(RuntimeError):
    def __init__(self, fn, status, message):
        self.status = status
        super().__init__(f"{fn} -> {STATUS_NAMES.get(status, status)}: {message}")


_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I = ctypes.c_int
_F = ctypes.c_float

FS_PROGRAM_MAX_OPS = 16
# fs_op_code by the oracle's operation names, with the parameter count
PROGRAM_OPS = {"scale": (0, 1), "shift": (1, 1), "add_bias": (2, 0), "mul_column": (3, 0),
               "add_residual": (4, 0), "mul_residual": (5, 0), "clamp": (6, 2),
               "gelu_erf": (7, 0), "sigmoid": (8, 0), "relu": (9, 0), "tanh": (10, 0),
               "silu": (11, 0), "leaky_relu": (12, 1)}


class FsOp(ctypes.Structure):
    """struct fs_op of fusedsub.h."""
    _fields_ = [("code", ctypes.c_int32), ("a", ctypes.c_float), ("b", ctypes.c_float)]


_SIGS = {
    "fs_pointwise_chain": [_P, _I64, _P, _P, _I64, _P, _I64, _I64, _I64, _F, _I, _I, _P],
    "fs_pointwise_program": [_P, _I64, ctypes.POINTER(FsOp), _I, _P, _P, _P, _I64, _P, _I64, _I64,
                             _I64, _I, _P],
    "fs_row_softmax": [_P, _I64, _P, _I64, _I, _P, _I64, _I64, _I64, _F, _I64, _I, _P],
    "fs_layernorm_residual": [_P, _I64, _P, _I64, _P, _P, _P, _I64, _P, _I64, _I64, _I64, _F, _I,
                              _P],
    "fs_rmsnorm_residual": [_P, _I64, _P, _I64, _P, _P, _I64, _P, _I64, _I64, _I64, _F, _I, _P],
    "fs_row_reduce": [_P, _I64, _I, _I, _P, _I64, _I64, _P],
    "fs_row_argmax": [_P, _I64, _I, _P, _I64, _I64, _P],
    "fs_gemm_epilogue_reduce": [_P, _I64, _I, _P, _I, _P, _I, _I, _P, _I64, _I64, _P],
    "fs_causal_softmax_trimmed": [_P, _I64, _P, _I64, _I64, _I64, _F, _I64, _I64, _I, _P],
    "fs_copy_strided": [_P, _I64, _I64, _P, _I64, _I64, _I64, _I64, _I64, _I, _P],
    "fs_copy": [_P, _P, _I64, _P],
    "fs_status_string": [_I],
    "fs_last_error_message": [],
    "fs_abi_version": [],
    "fsg_gemm_bf16": [_P, _I64, _I64, _P, _I64, _I64, _I, _P, _I64, _I64, _I64, _I64, _I64, _I64,
                      _F, _P, _P, ctypes.c_size_t, _P],
    "fsg_gemm_bf16_ex": [_P, _I64, _I64, _P, _I64, _I64, _I, _P, _I64, _I64, _I64, _I64, _I64,
                         _I64, _F, _P, _P, _I, _I, _P, _I64, _I64, _F, _P, ctypes.c_size_t, _P],
    "fsg_last_error_message": [],
}
_RESTYPES = {"fs_status_string": ctypes.c_char_p, "fs_last_error_message": ctypes.c_char_p,
             "fsg_last_error_message": ctypes.c_char_p}

_lock = threading.Lock()
_libs = {}


def _load(path, symbols):
    import torch  # noqa: F401  -- maps torch's HIP runtime first (see module doc)
    if not os.path.exists(path):
        raise NativeLibraryError(
            f"{os.path.basename(path)} is not built; run `python -m paper_2609_30059_amd.build` "
            "(or __graft_entry__.build())")
    try:
        lib = ctypes.CDLL(path, mode=ctypes.RTLD_LOCAL)
    except OSError as e:
        raise NativeLibraryError(f"cannot load {path}: {e}") from e
    for name in symbols:
        fn = getattr(lib, name)
        fn.argtypes = _SIGS[name]
        fn.restype = _RESTYPES.get(name, ctypes.c_int)
    return lib


def fusedsub():
    """The loaded libfusedsub (loaded on first use)."""
    with _lock:
        if "fusedsub" not in _libs:
            lib = _load(LIB_FUSEDSUB, FUSEDSUB_SYMBOLS)
            if lib.fs_abi_version() != FS_ABI_VERSION:
                raise NativeLibraryError("libfusedsub ABI version mismatch")
            _libs["fusedsub"] = lib
        return _libs["fusedsub"]


def fsgemm():
    with _lock:
        if "fsgemm" not in _libs:
            _libs["fsgemm"] = _load(LIB_FSGEMM, FSGEMM_SYMBOLS)
        return _libs["fsgemm"]


def hip_runtimes_mapped():
    """Paths of every libamdhip64 mapped into this process."""
    paths = set()
    with open("/proc/self/maps") as f:
        for line in f:
            if "libamdhip64" in line:
                paths.add(line.split()[-1])
    return sorted(paths)


# ---------------------------------------------------------------------------
# raw entry points, same names and arguments as the C ABI; return the status
# ---------------------------------------------------------------------------
def fs_pointwise_chain(x, ld_x, bias, residual, ld_r, y, ld_y, rows, cols, scale, act, dtype,
                       stream):
    return fusedsub().fs_pointwise_chain(x, ld_x, bias, residual, ld_r, y, ld_y, rows, cols,
                                         scale, act, dtype, stream)


def fs_pointwise_program(x, ld_x, ops, n_ops, bias, col, residual, ld_r, y, ld_y, rows, cols,
                         dtype, stream):
    return fusedsub().fs_pointwise_program(x, ld_x, ops, n_ops, bias, col, residual, ld_r, y, ld_y,
                                           rows, cols, dtype, stream)


def fs_row_softmax(x, ld_x, mask, ld_mask, mask_dtype, y, ld_y, rows, cols, scale, causal_q_len,
                   dtype, stream):
    return fusedsub().fs_row_softmax(x, ld_x, mask, ld_mask, mask_dtype, y, ld_y, rows, cols,
                                     scale, causal_q_len, dtype, stream)


def fs_layernorm_residual(x, ld_x, residual, ld_r, gamma, beta, y, ld_y, residual_out, ld_ro,
                          rows, cols, eps, dtype, stream):
    return fusedsub().fs_layernorm_residual(x, ld_x, residual, ld_r, gamma, beta, y, ld_y,
                                            residual_out, ld_ro, rows, cols, eps, dtype, stream)


def fs_rmsnorm_residual(x, ld_x, residual, ld_r, gamma, y, ld_y, residual_out, ld_ro, rows, cols,
                        eps, dtype, stream):
    return fusedsub().fs_rmsnorm_residual(x, ld_x, residual, ld_r, gamma, y, ld_y, residual_out,
                                          ld_ro, rows, cols, eps, dtype, stream)


def fs_row_reduce(x, ld_x, dtype, op, out, rows, cols, stream):
    return fusedsub().fs_row_reduce(x, ld_x, dtype, op, out, rows, cols, stream)


def fs_row_argmax(x, ld_x, dtype, out, rows, cols, stream):
    return fusedsub().fs_row_argmax(x, ld_x, dtype, out, rows, cols, stream)


def fs_gemm_epilogue_reduce(c, ld_c, c_dtype, bias, bias_dtype, col_scale, act, reduce, row_out,
                            rows, cols, stream):
    return fusedsub().fs_gemm_epilogue_reduce(c, ld_c, c_dtype, bias, bias_dtype, col_scale, act,
                                              reduce, row_out, rows, cols, stream)


def fs_causal_softmax_trimmed(x, ld_x, y, ld_y, rows, cols, scale, causal_q_len, block, dtype,
                              stream):
    return fusedsub().fs_causal_softmax_trimmed(x, ld_x, y, ld_y, rows, cols, scale, causal_q_len,
                                                block, dtype, stream)


def fs_copy_strided(src, ld_src, stride_src, dst, ld_dst, stride_dst, rows, cols, batch, dtype,
                    stream):
    return fusedsub().fs_copy_strided(src, ld_src, stride_src, dst, ld_dst, stride_dst, rows, cols,
                                      batch, dtype, stream)


def fs_copy(src, dst, nbytes, stream):
    return fusedsub().fs_copy(src, dst, nbytes, stream)


def fs_status_string(status):
    return fusedsub().fs_status_string(status).decode()


def fs_last_error_message():
    return fusedsub().fs_last_error_message().decode()


def fs_abi_version():
    return fusedsub().fs_abi_version()


def fsg_gemm_bf16(a, lda, stride_a, b, ldb, stride_b, trans_b, c, ldc, stride_c, m, n, k, batch,
                  alpha, bias, workspace, workspace_bytes, stream):
    return fsgemm().fsg_gemm_bf16(a, lda, stride_a, b, ldb, stride_b, trans_b, c, ldc, stride_c,
                                  m, n, k, batch, alpha, bias, workspace, workspace_bytes, stream)


def fsg_gemm_bf16_ex(a, lda, stride_a, b, ldb, stride_b, trans_b, c, ldc, stride_c, m, n, k, batch,
                     alpha, alpha_col, bias, bias_f32, act, c_in, ld_cin, stride_cin, beta,
                     workspace, workspace_bytes, stream):
    return fsgemm().fsg_gemm_bf16_ex(a, lda, stride_a, b, ldb, stride_b, trans_b, c, ldc, stride_c,
                                     m, n, k, batch, alpha, alpha_col, bias, bias_f32, act, c_in,
                                     ld_cin, stride_cin, beta, workspace, workspace_bytes, stream)


def fsg_last_error_message():
    return fsgemm().fsg_last_error_message().decode()


def check(fn_name, status):
    """Raise FusedSubError for a non-OK status of a libfusedsub call."""
    if status != FS_OK:
        raise FusedSubError(fn_name, status, fs_last_error_message())


GEMM_STATUS_NAMES = {0: "FSG_OK", 1: "FSG_ERR_NULL_POINTER", 2: "FSG_ERR_BAD_SHAPE",
                     3: "FSG_ERR_BAD_STRIDE", 4: "FSG_ERR_BAD_ARGUMENT", 5: "FSG_ERR_LIBRARY",
                     6: "FSG_ERR_NO_ALGO", 7: "FSG_ERR_HIP"}


class GemmError(RuntimeError):
    def __init__(self, status, message):
        self.status = status
        super().__init__(f"fsg_gemm_bf16 -> {GEMM_STATUS_NAMES.get(status, status)}: {message}")


def check_gemm(status):
    """Raise GemmError for a non-OK status of fsg_gemm_bf16."""
    if status != 0:
        raise GemmError(status, fsg_last_error_message())
