"""Tensor-level calls of the fused sub-kernels and the GEMM wrapper.

Argument marshalling only: each function turns torch tensors into the device
pointers, row strides and HIP stream the C ABI takes, allocates outputs with
torch (device memory is torch's job here), calls the native entry point and
raises on a non-OK status.  No arithmetic happens in Python.
"""
from __future__ import annotations

from typing import Optional, Tuple

import torch

from . import _native as N

__all__ = ["pointwise_chain", "row_softmax", "layernorm_residual", "rmsnorm_residual",
           "row_reduce", "row_argmax", "gemm_epilogue_reduce", "copy_", "gemm",
           "gemm_strided_batched", "as_rows", "fs_dtype"]


def fs_dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return N.FS_F32
    if t.dtype == torch.bfloat16:
        return N.FS_BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 and bfloat16 only)")


def as_rows(t: torch.Tensor) -> Tuple[int, int, int]:
    """(rows, cols, ld) of a tensor viewed as [prod(leading dims), last dim].

    The last dim must have unit stride, the leading dims must collapse onto
    one row stride (a batch of rows), and distinct rows must not overlap:
    broadcast (stride-0) and overlapping views are refused, since a kernel
    would read or write past the memory they cover."""
    nd = t.dim()
    if nd >= 2 and t.is_contiguous():
        cols = t.shape[-1]
        if cols > 0:                       # dense rows: ld = cols
            return t.numel() // cols, cols, cols
    if nd == 0:
        raise ValueError("scalar tensors are not supported")
    cols = t.shape[-1]
    if cols > 1 and t.stride(-1) != 1:
        raise ValueError("the last dimension must be contiguous")
    if nd == 1:
        return 1, cols, max(cols, 1)
    # leading dims of extent > 1, innermost first: the innermost gives the
    # row stride, each outer one must step over whole inner blocks
    lead = [(t.shape[i], t.stride(i)) for i in range(nd - 2, -1, -1) if t.shape[i] > 1]
    rows = 1
    for s in t.shape[:-1]:
        rows *= s
    if rows <= 1 or not lead:
        return rows, cols, max(cols, 1)
    ld = lead[0][1]
    for (n_in, s_in), (_, s_out) in zip(lead, lead[1:]):
        if s_out != s_in * n_in:
            raise ValueError("leading dimensions do not collapse onto one row stride")
    if cols == 0:
        return rows, 0, max(ld, 1)
    if ld < cols:
        raise ValueError(f"rows overlap or are broadcast (row stride {ld} < {cols} columns); "
                         "make the tensor contiguous")
    return rows, cols, ld


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


# torch's raw accessors of the current device and stream (the public calls
# build Python objects: 2.5 us per call against 0.05); the public API is the
# fallback where a torch build lacks them
_RAW_STREAM = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_RAW_DEVICE = getattr(torch._C, "_cuda_getDevice", None)


def _current_device() -> int:
    return _RAW_DEVICE() if _RAW_DEVICE is not None else torch.cuda.current_device()


def _stream() -> int:
    """The current stream of the current device, as a raw hipStream_t (the
    handle torch.cuda.current_stream().cuda_stream returns)."""
    if _RAW_STREAM is not None:
        return _RAW_STREAM(_current_device())
    return torch.cuda.current_stream().cuda_stream


def _cuda(**tensors) -> None:
    """Every tensor handed to a kernel must live on the current GPU."""
    dev = None
    for name, t in tensors.items():
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError(f"{name} must be a CUDA (HIP) device tensor")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError(f"{name} is on {t.device}, expected {dev}")
    if dev is not None and dev.index is not None and dev.index != _current_device():
        raise ValueError(f"tensors are on {dev}; make it the current device")


def _like(out: torch.Tensor, x: torch.Tensor, name: str) -> int:
    """out must have x's rows, columns and dtype; returns its row stride."""
    if out.dtype != x.dtype:
        raise ValueError(f"{name} must have dtype {x.dtype}")
    r, c, ld = as_rows(out)
    rx, cx, _ = as_rows(x)
    if (r, c) != (rx, cx):
        raise ValueError(f"{name} must be [{rx}, {cx}] as rows, got [{r}, {c}]")
    return ld


def _vec(t: Optional[torch.Tensor], cols: int, name: str):
    if t is None:
        return None
    if t.dim() != 1 or t.shape[0] != cols or (cols > 1 and t.stride(0) != 1):
        raise ValueError(f"{name} must be a contiguous [{cols}] vector")
    return t


def pointwise_chain(x: torch.Tensor, bias: Optional[torch.Tensor] = None,
                    residual: Optional[torch.Tensor] = None, scale: float = 1.0,
                    act: str = "none", out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """y = act(x * scale + bias) + residual  (fs_pointwise_chain)."""
    rows, cols, ld_x = as_rows(x)
    if out is None:
        out = torch.empty_like(x, memory_format=torch.contiguous_format)
    _cuda(x=x, bias=bias, residual=residual, out=out)
    ld_y = _like(out, x, "out")
    ld_r = 0
    if residual is not None:
        if residual.shape != x.shape or residual.dtype != x.dtype:
            raise ValueError("residual must match x")
        ld_r = as_rows(residual)[2]
    if bias is not None and bias.dtype != x.dtype:
        raise ValueError("bias dtype must match x")
    _vec(bias, cols, "bias")
    st = N.fs_pointwise_chain(x.data_ptr(), ld_x, _ptr(bias), _ptr(residual), ld_r,
                              out.data_ptr(), ld_y, rows, cols, float(scale), N.ACTS[act],
                              fs_dtype(x), _stream())
    N.check("fs_pointwise_chain", st)
    return out


def program_ops(ops) -> "ctypes.Array":
    """An fs_op array from operations given as (name, *params) with the
    names of fusedsub.h's fs_op_code in lower case (``("scale", 0.5)``,
    ``("clamp", -1, 1)``, ``("gelu_erf",)``, ...)."""
    ops = list(ops)
    arr = (N.FsOp * max(len(ops), 1))()
    for k, op in enumerate(ops):
        name, prm = op[0], list(op[1:])
        if name not in N.PROGRAM_OPS:
            raise ValueError(f"unknown operation {name!r}")
        code, n = N.PROGRAM_OPS[name]
        if len(prm) != n:
            raise ValueError(f"{name} takes {n} parameter(s), got {len(prm)}")
        prm += [0.0] * (2 - n)
        arr[k] = N.FsOp(code, float(prm[0]), float(prm[1]))
    return arr


def pointwise_program(x: torch.Tensor, ops, bias: Optional[torch.Tensor] = None,
                      col: Optional[torch.Tensor] = None,
                      residual: Optional[torch.Tensor] = None,
                      out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """y = op_n(... op_1(x) ...) elementwise (fs_pointwise_program); see
    ``program_ops`` for the form of ``ops``."""
    ops = list(ops)
    arr = program_ops(ops)
    rows, cols, ld_x = as_rows(x)
    if out is None:
        out = torch.empty_like(x, memory_format=torch.contiguous_format)
    _cuda(x=x, bias=bias, col=col, residual=residual, out=out)
    ld_y = _like(out, x, "out")
    ld_r = 0
    if residual is not None:
        if residual.shape != x.shape or residual.dtype != x.dtype:
            raise ValueError("residual must match x")
        ld_r = as_rows(residual)[2]
    for name, v in (("bias", bias), ("col", col)):
        if v is not None and v.dtype != x.dtype:
            raise ValueError(f"{name} dtype must match x")
        _vec(v, cols, name)
    st = N.fs_pointwise_program(x.data_ptr(), ld_x, arr, len(ops), _ptr(bias), _ptr(col),
                                _ptr(residual), ld_r, out.data_ptr(), ld_y, rows, cols,
                                fs_dtype(x), _stream())
    N.check("fs_pointwise_program", st)
    return out


def mask_dtype(m: torch.Tensor) -> int:
    """fs_dtype of a softmax mask: float32 and bfloat16 masks are additive;
    bool and uint8 masks are byte masks (FS_U8), where a nonzero element
    excludes its position (True = masked out, as in ``masked_fill``)."""
    if m.dtype in (torch.bool, torch.uint8):
        return N.FS_U8
    return fs_dtype(m)


def row_softmax(x: torch.Tensor, mask: Optional[torch.Tensor] = None, scale: float = 1.0,
                causal_q_len: int = 0, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """softmax(x * scale + mask) along the last dim (fs_row_softmax).  A bool
    or uint8 mask excludes the positions where it is nonzero (see
    ``mask_dtype``)."""
    rows, cols, ld_x = as_rows(x)
    if out is None:
        out = torch.empty_like(x, memory_format=torch.contiguous_format)
    _cuda(x=x, mask=mask, out=out)
    ld_y = _like(out, x, "out")
    ld_m, mdt = 0, fs_dtype(x)
    if mask is not None:
        if mask.shape != x.shape:
            raise ValueError("mask must have the shape of x")
        ld_m, mdt = as_rows(mask)[2], mask_dtype(mask)
    st = N.fs_row_softmax(x.data_ptr(), ld_x, _ptr(mask), ld_m, mdt, out.data_ptr(), ld_y, rows,
                          cols, float(scale), int(causal_q_len), fs_dtype(x), _stream())
    N.check("fs_row_softmax", st)
    return out


def causal_softmax_trimmed(x: torch.Tensor, scale: float, causal_q_len: int, block: int,
                           out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Causal softmax(x * scale) writing only the columns j < w(r) of each
    row, w(r) = min(cols, (floor(s / block) + 1) * block + cols - q) with
    s = r mod q  (fs_causal_softmax_trimmed); the rest of out is untouched."""
    rows, cols, ld_x = as_rows(x)
    if out is None:
        out = torch.empty_like(x, memory_format=torch.contiguous_format)
    _cuda(x=x, out=out)
    ld_y = _like(out, x, "out")
    st = N.fs_causal_softmax_trimmed(x.data_ptr(), ld_x, out.data_ptr(), ld_y, rows, cols,
                                     float(scale), int(causal_q_len), int(block), fs_dtype(x),
                                     _stream())
    N.check("fs_causal_softmax_trimmed", st)
    return out


def layernorm_residual(x: torch.Tensor, residual: Optional[torch.Tensor] = None,
                       gamma: Optional[torch.Tensor] = None, beta: Optional[torch.Tensor] = None,
                       eps: float = 1e-5, out: Optional[torch.Tensor] = None,
                       residual_out: Optional[torch.Tensor] = None,
                       store_residual: bool = True):
    """(LN(x + residual), x + residual)  (fs_layernorm_residual).

    Returns (y, residual_out); residual_out is None when there is no residual
    or ``store_residual`` is False."""
    rows, cols, ld_x = as_rows(x)
    if out is None:
        out = torch.empty_like(x, memory_format=torch.contiguous_format)
    ld_r = ld_ro = 0
    if residual is not None:
        if residual.shape != x.shape or residual.dtype != x.dtype:
            raise ValueError("residual must match x")
        ld_r = as_rows(residual)[2]
        if residual_out is None and store_residual:
            residual_out = torch.empty_like(x, memory_format=torch.contiguous_format)
    if residual_out is not None:
        ld_ro = _like(residual_out, x, "residual_out")
    _cuda(x=x, residual=residual, gamma=gamma, beta=beta, out=out, residual_out=residual_out)
    _like(out, x, "out")
    for v, n in ((gamma, "gamma"), (beta, "beta")):
        if v is not None and v.dtype != x.dtype:
            raise ValueError(f"{n} dtype must match x")
        _vec(v, cols, n)
    st = N.fs_layernorm_residual(x.data_ptr(), ld_x, _ptr(residual), ld_r, _ptr(gamma),
                                 _ptr(beta), out.data_ptr(), as_rows(out)[2],
                                 _ptr(residual_out), ld_ro, rows, cols, float(eps), fs_dtype(x),
                                 _stream())
    N.check("fs_layernorm_residual", st)
    return out, residual_out


def rmsnorm_residual(x: torch.Tensor, residual: Optional[torch.Tensor] = None,
                     gamma: Optional[torch.Tensor] = None, eps: float = 1e-6,
                     out: Optional[torch.Tensor] = None,
                     residual_out: Optional[torch.Tensor] = None, store_residual: bool = True):
    """(RMSNorm(x + residual), x + residual)  (fs_rmsnorm_residual)."""
    rows, cols, ld_x = as_rows(x)
    if out is None:
        out = torch.empty_like(x, memory_format=torch.contiguous_format)
    ld_r = ld_ro = 0
    if residual is not None:
        if residual.shape != x.shape or residual.dtype != x.dtype:
            raise ValueError("residual must match x")
        ld_r = as_rows(residual)[2]
        if residual_out is None and store_residual:
            residual_out = torch.empty_like(x, memory_format=torch.contiguous_format)
    if residual_out is not None:
        ld_ro = _like(residual_out, x, "residual_out")
    _cuda(x=x, residual=residual, gamma=gamma, out=out, residual_out=residual_out)
    _like(out, x, "out")
    if gamma is not None and gamma.dtype != x.dtype:
        raise ValueError("gamma dtype must match x")
    _vec(gamma, cols, "gamma")
    st = N.fs_rmsnorm_residual(x.data_ptr(), ld_x, _ptr(residual), ld_r, _ptr(gamma),
                               out.data_ptr(), as_rows(out)[2], _ptr(residual_out), ld_ro, rows,
                               cols, float(eps), fs_dtype(x), _stream())
    N.check("fs_rmsnorm_residual", st)
    return out, residual_out


def row_reduce(x: torch.Tensor, op: str = "sum", out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Row sum / mean / max / logsumexp as float32 [rows]  (fs_row_reduce)."""
    rows, cols, ld_x = as_rows(x)
    if out is None:
        out = torch.empty(rows, dtype=torch.float32, device=x.device)
    if out.dtype != torch.float32 or out.numel() != rows or not out.is_contiguous():
        raise ValueError("out must be a contiguous float32 [rows] tensor")
    _cuda(x=x, out=out)
    st = N.fs_row_reduce(x.data_ptr() if x.numel() else None, ld_x, fs_dtype(x), N.ROW_OPS[op],
                         out.data_ptr(), rows, cols, _stream())
    N.check("fs_row_reduce", st)
    return out


def row_argmax(x: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Row argmax as int64 [rows]: lowest index on ties, first NaN wins  (fs_row_argmax)."""
    rows, cols, ld_x = as_rows(x)
    if out is None:
        out = torch.empty(rows, dtype=torch.int64, device=x.device)
    if out.dtype != torch.int64 or out.numel() != rows or not out.is_contiguous():
        raise ValueError("out must be a contiguous int64 [rows] tensor")
    _cuda(x=x, out=out)
    st = N.fs_row_argmax(x.data_ptr(), ld_x, fs_dtype(x), out.data_ptr(), rows, cols, _stream())
    N.check("fs_row_argmax", st)
    return out


def gemm_epilogue_reduce(c: torch.Tensor, bias: Optional[torch.Tensor] = None,
                         col_scale: Optional[torch.Tensor] = None, act: str = "sigmoid",
                         reduce: str = "sum", out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """out[i] = reduce_j act((c[i, j] + bias[j]) * col_scale[j])  (fs_gemm_epilogue_reduce)."""
    rows, cols, ld_c = as_rows(c)
    if out is None:
        out = torch.empty(rows, dtype=torch.float32, device=c.device)
    if out.dtype != torch.float32 or out.numel() != rows or not out.is_contiguous():
        raise ValueError("out must be a contiguous float32 [rows] tensor")
    _cuda(c=c, bias=bias, col_scale=col_scale, out=out)
    _vec(bias, cols, "bias")
    _vec(col_scale, cols, "col_scale")
    if col_scale is not None and col_scale.dtype != torch.float32:
        raise ValueError("col_scale must be float32")
    st = N.fs_gemm_epilogue_reduce(c.data_ptr(), ld_c, fs_dtype(c), _ptr(bias),
                                   fs_dtype(bias) if bias is not None else N.FS_F32,
                                   _ptr(col_scale), N.ACTS[act], N.REDUCES[reduce],
                                   out.data_ptr(), rows, cols, _stream())
    N.check("fs_gemm_epilogue_reduce", st)
    return out


def copy_strided(dst: torch.Tensor, src: torch.Tensor, rows: int, cols: int, batch: int,
                 ld_src: int, stride_src: int, ld_dst: int, stride_dst: int) -> torch.Tensor:
    """dst[b, r, c] = src[b, r, c] over the flat storage of two contiguous
    tensors of one dtype (fs_copy_strided), with element strides
    src offset b * stride_src + r * ld_src + c and likewise for dst."""
    if src.dtype != dst.dtype:
        raise ValueError("src and dst must have one dtype")
    if not (src.is_contiguous() and dst.is_contiguous()):
        raise ValueError("copy_strided addresses contiguous tensors")
    _cuda(src=src, dst=dst)
    if rows > 0 and cols > 0 and batch > 0:
        for t, ld, st, name in ((src, ld_src, stride_src, "src"), (dst, ld_dst, stride_dst, "dst")):
            last = (batch - 1) * st + (rows - 1) * ld + cols
            if last > t.numel():
                raise ValueError(f"{name} is too small for the requested strides")
    N.check("fs_copy_strided",
            N.fs_copy_strided(src.data_ptr(), ld_src, stride_src, dst.data_ptr(), ld_dst,
                              stride_dst, rows, cols, batch, fs_dtype(src), _stream()))
    return dst


def copy_(dst: torch.Tensor, src: torch.Tensor) -> torch.Tensor:
    """Byte copy of src into dst with the calibration kernel (fs_copy)."""
    if not (src.is_contiguous() and dst.is_contiguous()):
        raise ValueError("copy_ needs contiguous tensors")
    _cuda(src=src, dst=dst)
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("size mismatch")
    N.check("fs_copy", N.fs_copy(src.data_ptr(), dst.data_ptr(), nbytes, _stream()))
    return dst


# ---------------------------------------------------------------------------
# hipBLASLt GEMMs (the fixed library calls)
# ---------------------------------------------------------------------------
_WORKSPACE_BYTES = 64 << 20
_workspaces = {}


def _workspace(device) -> torch.Tensor:
    idx = torch.device(device).index
    if idx is None:
        idx = torch.cuda.current_device()
    ws = _workspaces.get(idx)
    if ws is None:
        ws = torch.empty(_WORKSPACE_BYTES, dtype=torch.uint8, device=f"cuda:{idx}")
        _workspaces[idx] = ws
    return ws


def gemm_strided_batched(a_ptr: int, lda: int, stride_a: int, b_ptr: int, ldb: int,
                         stride_b: int, trans_b: bool, c_ptr: int, ldc: int, stride_c: int,
                         m: int, n: int, k: int, batch: int, alpha: float = 1.0,
                         bias: Optional[torch.Tensor] = None, device="cuda") -> None:
    """Raw-pointer form of fsg_gemm_bf16 for strided views (attention heads)."""
    ws = _workspace(device)
    st = N.fsg_gemm_bf16(a_ptr, lda, stride_a, b_ptr, ldb, stride_b, int(trans_b), c_ptr, ldc,
                         stride_c, m, n, k, batch, float(alpha), _ptr(bias), ws.data_ptr(),
                         ws.numel(), _stream())
    N.check_gemm(st)


GEMM_ACTS = {"none": 0, "gelu": 1, "relu": 2}


def gemm(a: torch.Tensor, b: torch.Tensor, bias: Optional[torch.Tensor] = None,
         out: Optional[torch.Tensor] = None, trans_b: bool = False,
         alpha: float = 1.0, act: str = "none", col_scale: Optional[torch.Tensor] = None,
         c_in: Optional[torch.Tensor] = None, beta: float = 0.0) -> torch.Tensor:
    """out = act(alpha * a @ b (* col_scale) + beta * c_in + bias) for bf16
    row-major a [m, k] and b [k, n] (or b stored [n, k] with trans_b).  The
    activation, column scale and c_in use hipBLASLt's own epilogue
    (fsg_gemm_bf16_ex); bias is bf16, or fp32 on that path."""
    for t in (a, b):
        if t.dtype != torch.bfloat16:
            raise TypeError("gemm takes bfloat16 operands")
    if act not in GEMM_ACTS:
        raise ValueError(f"act must be one of {sorted(GEMM_ACTS)}")
    m, k, lda = as_rows(a)
    if trans_b:
        n, kb, ldb = as_rows(b)
    else:
        kb, n, ldb = as_rows(b)
    if kb != k:
        raise ValueError(f"inner dimensions differ: {k} vs {kb}")
    if out is None:
        out = torch.empty((*a.shape[:-1], n), dtype=torch.bfloat16, device=a.device)
    _cuda(a=a, b=b, bias=bias, out=out, col_scale=col_scale, c_in=c_in)
    mo, no, ldc = as_rows(out)
    if out.dtype != torch.bfloat16 or (mo, no) != (m, n):
        raise ValueError(f"out must be bf16 [{m}, {n}] as rows")
    _vec(bias, n, "bias")
    if bias is not None and bias.dtype not in (torch.bfloat16, torch.float32):
        raise TypeError("bias must be bf16 or fp32")
    extended = act != "none" or col_scale is not None or c_in is not None or beta != 0.0 or (
        bias is not None and bias.dtype == torch.float32)
    if not extended:
        gemm_strided_batched(a.data_ptr(), lda, 0, b.data_ptr(), ldb, 0, trans_b,
                             out.data_ptr(), ldc, 0, m, n, k, 1, alpha, bias, a.device)
        return out
    if col_scale is not None:
        if col_scale.dtype != torch.float32:
            raise TypeError("col_scale must be fp32")
        _vec(col_scale, n, "col_scale")
    ld_cin = 0
    if c_in is not None:
        if c_in.dtype != torch.bfloat16:
            raise TypeError("c_in must be bf16")
        mc, nc, ld_cin = as_rows(c_in)
        if (mc, nc) != (m, n):
            raise ValueError("c_in must be [m, n]")
    ws = _workspace(a.device)
    st = N.fsg_gemm_bf16_ex(a.data_ptr(), lda, 0, b.data_ptr(), ldb, 0, int(trans_b),
                            out.data_ptr(), ldc, 0, m, n, k, 1, float(alpha), _ptr(col_scale),
                            _ptr(bias), int(bias is not None and bias.dtype == torch.float32),
                            GEMM_ACTS[act], _ptr(c_in), ld_cin, 0, float(beta), ws.data_ptr(),
                            ws.numel(), _stream())
    N.check_gemm(st)
    return out
