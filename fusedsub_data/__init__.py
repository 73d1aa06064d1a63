"""Seeded synthetic inputs for the fused sub-kernel workloads.

This module is shared by the float64 oracle (through the tests) and by the
device path.  It holds no arithmetic of the sub-kernels themselves: it draws
random numbers, quantises them to the storage dtype the kernels read, and
decodes stored bits back to exact float64 values.

Draw protocol (every workload): ``numpy.random.default_rng(seed)`` (PCG64),
draws in float64 in the order the workload lists them, then rounded to the
I/O dtype.  fp32 storage uses numpy's float64->float32 cast (IEEE round to
nearest even); bf16 storage rounds that float32 value to bf16 (round to
nearest even on the upper 16 bits).

The named workloads (``CONFIGS``: a pointwise chain, a softmax, a LayerNorm, a
GEMM epilogue and a transformer block, each named by its kind and shape) are
the paper-style shapes the kernels are measured on.  The paper evaluates on KernelBench problems,
which are not reproduced here; these seeded draws stand in for them with the
shapes and distributions of the workloads this library targets.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

__all__ = [
    "f32_to_bf16_bits", "bf16_bits_to_f64", "bf16_bits_to_f32", "Tensor",
    "pointwise_inputs", "softmax_inputs", "layernorm_inputs", "epilogue_inputs",
    "gemm_epilogue_inputs", "block_inputs", "row_inputs", "integer_inputs", "CONFIGS",
    "make_inputs",
    "BLOCK_DIMS",
]

NEG_INF = float("-inf")


# ----------------------------------------------------------------------------
# storage dtype encode / decode (input quantisation only)
# ----------------------------------------------------------------------------
def f32_to_bf16_bits(a) -> np.ndarray:
    """float array -> bf16 bit patterns (uint16), round to nearest even.

    The value is first cast to float32 (numpy RNE), then the low 16 bits are
    rounded away with ties to even.  Infinities pass through; NaN becomes the
    canonical quiet NaN 0x7FC0.
    """
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        r = np.where(nan, np.uint16(0x7FC0), r)
    return r


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact float64 values of bf16 bit patterns."""
    return bf16_bits_to_f32(bits).astype(np.float64)


@dataclasses.dataclass
class Tensor:
    """A host tensor in its storage dtype.

    ``data`` holds float32 values for ``dtype == "f32"``, uint16 bf16 bit
    patterns for ``dtype == "bf16"`` and bytes for ``dtype == "u8"`` (a byte
    mask; ``f64`` gives the byte values themselves).
    """
    data: np.ndarray
    dtype: str

    @property
    def shape(self):
        return self.data.shape

    def f64(self) -> np.ndarray:
        if self.dtype == "f32":
            return self.data.astype(np.float64)
        if self.dtype == "bf16":
            return bf16_bits_to_f64(self.data)
        if self.dtype == "u8":
            return self.data.astype(np.float64)
        raise ValueError(self.dtype)

    def rows(self, idx) -> "Tensor":
        return Tensor(np.ascontiguousarray(self.data[idx]), self.dtype)


def _store(values_f64: np.ndarray, dtype: str) -> Tensor:
    if dtype == "f32":
        return Tensor(np.ascontiguousarray(values_f64.astype(np.float32)), "f32")
    if dtype == "bf16":
        return Tensor(f32_to_bf16_bits(values_f64), "bf16")
    raise ValueError(f"unsupported storage dtype {dtype!r}")


def _normal(rng, shape, mean, std):
    return rng.standard_normal(size=shape, dtype=np.float64) * std + mean


def _uniform(rng, shape, lo, hi):
    return rng.random(size=shape, dtype=np.float64) * (hi - lo) + lo


# ----------------------------------------------------------------------------
# per-class generators
# ----------------------------------------------------------------------------
def pointwise_inputs(seed: int, rows: int, cols: int, dtype: str = "f32",
                     scale: float = 0.7, with_bias: bool = True,
                     with_residual: bool = True) -> Dict[str, object]:
    """x ~ N(0,1) [rows,cols]; r ~ N(0,1) [rows,cols]; b ~ U(-1/2,1/2) [cols].

    Draw order x, r, b.  ``scale`` is returned rounded to float32, the value
    the device receives through a ``float`` argument.
    """
    rng = np.random.default_rng(seed)
    x = _normal(rng, (rows, cols), 0.0, 1.0)
    r = _normal(rng, (rows, cols), 0.0, 1.0)
    b = _uniform(rng, (cols,), -0.5, 0.5)
    return {
        "x": _store(x, dtype),
        "residual": _store(r, dtype) if with_residual else None,
        "bias": _store(b, dtype) if with_bias else None,
        "scale": float(np.float32(scale)),
    }


def softmax_inputs(seed: int, rows: int, cols: int, dtype: str = "bf16",
                   sigma: float = 3.0, mask_dtype: Optional[str] = "bf16",
                   p_masked: float = 0.1, scale: float = 0.125) -> Dict[str, object]:
    """logits ~ N(0, sigma) [rows,cols]; additive mask in {0, -inf}.

    Each mask element is -inf independently with probability ``p_masked``
    (draw order: logits, then one U(0,1) per mask element).  A row that comes
    out fully masked gets column 0 unmasked, so no row is empty.

    ``mask_dtype="u8"`` stores the same pattern as a byte mask: 0 where the
    additive mask is 0, and at each masked position a byte drawn uniformly
    from 1..255 (one more draw per element, after the others, so the logits
    and the pattern equal those of the other mask dtypes for the seed).
    """
    rng = np.random.default_rng(seed)
    x = _normal(rng, (rows, cols), 0.0, sigma)
    out = {"x": _store(x, dtype), "scale": float(np.float32(scale)), "mask": None}
    if mask_dtype is not None:
        u = rng.random(size=(rows, cols), dtype=np.float64)
        masked = u < p_masked
        full = masked.all(axis=1)
        if full.any():
            masked[full, 0] = False
        if mask_dtype == "u8":
            b = rng.integers(1, 256, size=(rows, cols), dtype=np.uint8)
            out["mask"] = Tensor(np.ascontiguousarray(np.where(masked, b, 0).astype(np.uint8)),
                                 "u8")
        else:
            m = np.where(masked, NEG_INF, 0.0)
            out["mask"] = _store(m, mask_dtype)
    return out


def layernorm_inputs(seed: int, rows: int, cols: int, dtype: str = "bf16",
                     with_residual: bool = True, eps: float = 1e-5) -> Dict[str, object]:
    """x, res ~ N(0,1) [rows,cols]; gamma ~ N(1,0.1), beta ~ N(0,0.1) [cols].

    Draw order x, res, gamma, beta.  ``eps`` is returned rounded to float32.
    """
    rng = np.random.default_rng(seed)
    x = _normal(rng, (rows, cols), 0.0, 1.0)
    res = _normal(rng, (rows, cols), 0.0, 1.0)
    g = _normal(rng, (cols,), 1.0, 0.1)
    b = _normal(rng, (cols,), 0.0, 0.1)
    return {
        "x": _store(x, dtype),
        "residual": _store(res, dtype) if with_residual else None,
        "gamma": _store(g, dtype),
        "beta": _store(b, dtype),
        "eps": float(np.float32(eps)),
    }


def epilogue_inputs(seed: int, rows: int, cols: int, c_dtype: str = "bf16",
                    c_std: float = 0.0256, bias_dtype: str = "bf16") -> Dict[str, object]:
    """Epilogue-only inputs: C ~ N(0, c_std) [rows,cols] standing in for a GEMM
    output; bias ~ U(-1/2,1/2) [cols]; col_scale ~ U(0.5,1.5) [cols] fp32.

    ``c_std`` defaults to the standard deviation of a K=4096 product of
    N(0,0.02) entries (0.02 * 0.02 * sqrt(4096)).  Draw order C, bias, scale.
    """
    rng = np.random.default_rng(seed)
    c = _normal(rng, (rows, cols), 0.0, c_std)
    b = _uniform(rng, (cols,), -0.5, 0.5)
    s = _uniform(rng, (cols,), 0.5, 1.5)
    return {
        "c": _store(c, c_dtype),
        "bias": _store(b, bias_dtype) if bias_dtype else None,
        "col_scale": _store(s, "f32"),
    }


def gemm_epilogue_inputs(seed: int, m: int, n: int, k: int) -> Dict[str, object]:
    """Full GEMM + epilogue inputs: A [m,k], B [k,n] ~ N(0,0.02) bf16;
    bias ~ U(-1/2,1/2) [n] bf16; col_scale ~ U(0.5,1.5) [n] fp32.
    Draw order A, B, bias, scale."""
    rng = np.random.default_rng(seed)
    a = _normal(rng, (m, k), 0.0, 0.02)
    b = _normal(rng, (k, n), 0.0, 0.02)
    bias = _uniform(rng, (n,), -0.5, 0.5)
    s = _uniform(rng, (n,), 0.5, 1.5)
    return {"a": _store(a, "bf16"), "b": _store(b, "bf16"),
            "bias": _store(bias, "bf16"), "col_scale": _store(s, "f32")}


def row_inputs(seed: int, rows: int, cols: int, dtype: str = "bf16", mean: float = 0.0,
               std: float = 1.0) -> Tensor:
    """x ~ N(mean, std) [rows, cols] in the storage dtype."""
    rng = np.random.default_rng(seed)
    return _store(_normal(rng, (rows, cols), mean, std), dtype)


def integer_inputs(seed: int, rows: int, cols: int, dtype: str = "bf16", lo: int = -3,
                   hi: int = 4) -> Tensor:
    """Small integers drawn uniformly from [lo, hi) -- exact in bf16 and fp32,
    so rows hold many exact ties."""
    rng = np.random.default_rng(seed)
    return _store(rng.integers(lo, hi, size=(rows, cols)).astype(np.float64), dtype)


BLOCK_DIMS = dict(batch=32, seq=512, hidden=1024, heads=16, mlp=4096)


def block_inputs(seed: int, batch: int = 32, seq: int = 512, hidden: int = 1024,
                 heads: int = 16, mlp: int = 4096, eps: float = 1e-5) -> Dict[str, object]:
    """Pre-LN transformer block inputs, bf16.

    x ~ N(0,1) [batch, seq, hidden]; every Linear weight and bias ~ N(0,0.02);
    LayerNorm gamma ~ N(1,0.1), beta ~ N(0,0.1).  Weights are stored [in, out]
    (y = x @ W + b).  Draw order: x, Wqkv, bqkv, Wo, bo, W1, b1, W2, b2,
    ln1_gamma, ln1_beta, ln2_gamma, ln2_beta.
    """
    rng = np.random.default_rng(seed)
    d = {}
    d["x"] = _store(_normal(rng, (batch, seq, hidden), 0.0, 1.0), "bf16")
    d["w_qkv"] = _store(_normal(rng, (hidden, 3 * hidden), 0.0, 0.02), "bf16")
    d["b_qkv"] = _store(_normal(rng, (3 * hidden,), 0.0, 0.02), "bf16")
    d["w_o"] = _store(_normal(rng, (hidden, hidden), 0.0, 0.02), "bf16")
    d["b_o"] = _store(_normal(rng, (hidden,), 0.0, 0.02), "bf16")
    d["w_1"] = _store(_normal(rng, (hidden, mlp), 0.0, 0.02), "bf16")
    d["b_1"] = _store(_normal(rng, (mlp,), 0.0, 0.02), "bf16")
    d["w_2"] = _store(_normal(rng, (mlp, hidden), 0.0, 0.02), "bf16")
    d["b_2"] = _store(_normal(rng, (hidden,), 0.0, 0.02), "bf16")
    d["ln1_gamma"] = _store(_normal(rng, (hidden,), 1.0, 0.1), "bf16")
    d["ln1_beta"] = _store(_normal(rng, (hidden,), 0.0, 0.1), "bf16")
    d["ln2_gamma"] = _store(_normal(rng, (hidden,), 1.0, 0.1), "bf16")
    d["ln2_beta"] = _store(_normal(rng, (hidden,), 0.0, 0.1), "bf16")
    d["eps"] = float(np.float32(eps))
    d["heads"] = heads
    return d


# ----------------------------------------------------------------------------
# the named workloads
# ----------------------------------------------------------------------------
CONFIGS = {
    "pointwise_256x1024": dict(kind="pointwise", rows=256, cols=1024, dtype="f32", scale=0.7,
                               act="gelu_erf"),
    # same chain and draws at a bandwidth-scale shape (3 GiB moved)
    "pointwise_262144x1024": dict(kind="pointwise", rows=262144, cols=1024, dtype="f32",
                                  scale=0.7, act="gelu_erf"),
    "softmax_8192x4096": dict(kind="softmax", rows=8192, cols=4096, dtype="bf16", sigma=3.0,
                              mask_dtype="bf16", p_masked=0.1, scale=0.125),
    "layernorm_16384x4096": dict(kind="layernorm", rows=16384, cols=4096, dtype="bf16",
                                 eps=1e-5),
    "gemm_epilogue_8192x8192x4096": dict(kind="gemm_epilogue", m=8192, n=8192, k=4096,
                                         act="sigmoid", reduce="sum"),
    "block_32x512x1024": dict(kind="block", **BLOCK_DIMS),
}


def make_inputs(cfg: str, seed: int, rows: Optional[int] = None) -> Dict[str, object]:
    """Inputs of a named workload; ``rows`` overrides the row count (the
    draws of the first rows do not depend on it for x-like tensors only when
    the override equals the original; callers use it for small variants)."""
    c = CONFIGS[cfg]
    kind = c["kind"]
    if kind == "pointwise":
        return pointwise_inputs(seed, rows or c["rows"], c["cols"], c["dtype"], c["scale"])
    if kind == "softmax":
        return softmax_inputs(seed, rows or c["rows"], c["cols"], c["dtype"], c["sigma"],
                              c["mask_dtype"], c["p_masked"], c["scale"])
    if kind == "layernorm":
        return layernorm_inputs(seed, rows or c["rows"], c["cols"], c["dtype"], True, c["eps"])
    if kind == "gemm_epilogue":
        return gemm_epilogue_inputs(seed, rows or c["m"], c["n"], c["k"])
    if kind == "block":
        return block_inputs(seed, batch=rows or c["batch"], seq=c["seq"], hidden=c["hidden"],
                            heads=c["heads"], mlp=c["mlp"])
    raise KeyError(cfg)
