"""Float64 oracle of the four fused sub-kernel classes.

TEST INFRASTRUCTURE ONLY.  Nothing in the library's product path imports,
calls or links this module; only the tests, the smoke check and the CPU
baseline leg of the benchmark do.  It shares no code with the HIP kernels.

Every function is the plain mathematical definition of the fused operation,
evaluated in float64 on the exact values the device receives (fp32 and bf16
inputs are upcast exactly; scalar arguments are the float32 values the C ABI
takes).  No blocking, fusion or reordering: a reader can check each line
against the definition.

Sources in the paper (KernelOPT):
  * Def. 1 (Section 3): a compiled model is a set of generated sub-kernels
    plus fixed vendor-library calls; only the sub-kernels are rewritten.
  * Appendix A, Fusion Agent prompt: the fusion techniques -- pointwise +
    pointwise (load once, apply both, store once), activation + bias fusion,
    reduction + pointwise, normalisation fusion (mean and variance in one
    pass, normalise/scale/bias in the same kernel, fp32 accumulation) and
    residual + norm in one memory pass.
  * Appendix A, Codegen (synthesis) agent prompt: keep the matmul as a
    library call and fuse only its epilogue; single-pass LayerNorm; online
    softmax.
  * Appendix A, Executor prompt: accumulate reductions in fp32 and cast to the
    output dtype only on the final store.

Readings where the paper is silent (each is also listed in the design notes):
  * GELU is the erf form, 0.5*z*(1 + erf(z/sqrt 2)).
  * The pointwise chain applies scale, then bias, then the activation, then
    the residual add; the bias broadcasts along rows (one value per column).
  * Softmax uses an additive mask; a row whose every entry is masked yields
    an all-zero output row (no NaN).  A byte mask (one byte per element, as
    boolean attention masks are stored) stands for the additive mask with
    -inf where the byte is nonzero and 0 where it is zero.
  * The causal rule masks element (r, j) iff j > (r mod q_len) + (cols - q_len).
  * LayerNorm uses the biased variance with eps inside the square root; its
    input is h = x + residual, and the stored residual is the float32 sum
    rounded to bf16.
  * The GEMM epilogue computes sum_j act((C[i,j] + bias[j]) * scale[j]).
"""
from __future__ import annotations

import math

import numpy as np
from scipy import special as _sp

__all__ = [
    "ACTS", "gelu_erf", "sigmoid", "relu", "apply_act",
    "pointwise_chain", "PROGRAM_OPS", "pointwise_program", "causal_mask", "byte_mask_additive", "row_softmax", "layernorm_residual",
    "rmsnorm_residual", "residual_store_bf16", "round_to_bf16", "gemm_epilogue_reduce",
    "row_reduce", "row_argmax",
]

ACTS = ("none", "gelu_erf", "sigmoid", "relu")


# ---------------------------------------------------------------------------
# activations
# ---------------------------------------------------------------------------
def gelu_erf(z):
    """GELU in its exact form z * Phi(z), Phi(z) = (1 + erf(z / sqrt 2)) / 2."""
    z = np.asarray(z, dtype=np.float64)
    return 0.5 * z * (1.0 + _sp.erf(z / math.sqrt(2.0)))


def sigmoid(t):
    """Logistic function 1 / (1 + exp(-t)), overflow-safe in float64."""
    t = np.asarray(t, dtype=np.float64)
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-t))


def relu(z):
    z = np.asarray(z, dtype=np.float64)
    return np.maximum(z, 0.0)


def apply_act(z, act: str):
    if act == "none":
        return np.asarray(z, dtype=np.float64)
    if act == "gelu_erf":
        return gelu_erf(z)
    if act == "sigmoid":
        return sigmoid(z)
    if act == "relu":
        return relu(z)
    raise ValueError(f"unknown activation {act!r}")


# ---------------------------------------------------------------------------
# a1: fused pointwise chain
# ---------------------------------------------------------------------------
def pointwise_chain(x, bias=None, residual=None, scale: float = 1.0, act: str = "none"):
    """y = act(x * scale + bias[col]) + residual.

    Appendix A (Fusion Agent: pointwise + pointwise; activation + bias
    fusion).  ``bias`` is a [cols] vector broadcast over rows, ``residual``
    has the shape of ``x``; either may be None (treated as zero).
    """
    x = np.asarray(x, dtype=np.float64)
    z = x * float(scale)
    if bias is not None:
        z = z + np.asarray(bias, dtype=np.float64)[None, :]
    y = apply_act(z, act)
    if residual is not None:
        y = y + np.asarray(residual, dtype=np.float64)
    return y


# ---------------------------------------------------------------------------
# a1, general form: a fused pointwise program
# ---------------------------------------------------------------------------
# Each operation maps the running value v (starting at x) to a new value;
# the names and their parameters:
PROGRAM_OPS = {
    "scale": 1,          # v * a
    "shift": 1,          # v + a
    "add_bias": 0,       # v + bias[j]
    "mul_column": 0,     # v * col[j]
    "add_residual": 0,   # v + residual[r, j]
    "mul_residual": 0,   # v * residual[r, j]
    "clamp": 2,          # min(max(v, a), b)  (hardtanh for a = -1, b = 1)
    "gelu_erf": 0,       # v * Phi(v)
    "sigmoid": 0,        # 1 / (1 + exp(-v))
    "relu": 0,           # max(v, 0)
    "tanh": 0,           # tanh(v)
    "silu": 0,           # v * sigmoid(v)
    "leaky_relu": 1,     # v if v >= 0 else a * v
}


def pointwise_program(x, ops, bias=None, col=None, residual=None):
    """y = f_n(... f_1(x) ...) elementwise, each f_i an operation of
    ``PROGRAM_OPS`` given as (name, *params).

    The general form of the fused pointwise chain: a compiled graph's group
    of adjacent elementwise operations (a linear layer's output followed by
    a multiply, a hardtanh and a GELU, say) evaluated as one pass (Section 3,
    merging adjacent fusible kernels; Appendix A, Fusion Agent: pointwise +
    pointwise, activation + bias fusion).  ``bias`` and ``col`` are [cols]
    vectors broadcast over rows; ``residual`` has the shape of ``x``.
    """
    v = np.asarray(x, dtype=np.float64)
    for op in ops:
        name, prm = op[0], [float(p) for p in op[1:]]
        if name not in PROGRAM_OPS or len(prm) != PROGRAM_OPS[name]:
            raise ValueError(f"bad program operation {op!r}")
        if name == "scale":
            v = v * prm[0]
        elif name == "shift":
            v = v + prm[0]
        elif name == "add_bias":
            v = v + np.asarray(bias, dtype=np.float64)[None, :]
        elif name == "mul_column":
            v = v * np.asarray(col, dtype=np.float64)[None, :]
        elif name == "add_residual":
            v = v + np.asarray(residual, dtype=np.float64)
        elif name == "mul_residual":
            v = v * np.asarray(residual, dtype=np.float64)
        elif name == "clamp":
            v = np.minimum(np.maximum(v, prm[0]), prm[1])
        elif name == "gelu_erf":
            v = gelu_erf(v)
        elif name == "sigmoid":
            v = sigmoid(v)
        elif name == "relu":
            v = relu(v)
        elif name == "tanh":
            v = np.tanh(v)
        elif name == "silu":
            v = v * sigmoid(v)
        else:   # leaky_relu
            v = np.where(v >= 0.0, v, prm[0] * v)
    return v


# ---------------------------------------------------------------------------
# a2: fused row softmax
# ---------------------------------------------------------------------------
def causal_mask(rows: int, cols: int, q_len: int) -> np.ndarray:
    """Boolean [rows, cols]: True where element (r, j) is masked, i.e.
    j > (r mod q_len) + (cols - q_len).  For square attention (cols == q_len)
    this is j > r mod q_len."""
    r = np.arange(rows, dtype=np.int64)[:, None]
    j = np.arange(cols, dtype=np.int64)[None, :]
    return j > (r % q_len) + (cols - q_len)


def causal_written_width(rows: int, cols: int, q_len: int, block: int) -> np.ndarray:
    """Columns of each row that a causal softmax trimmed to row blocks
    writes: w(r) = min(cols, (floor(s / block) + 1) * block + (cols - q_len)),
    at least 0, with s = r mod q_len.  Row r's live columns j <= s + (cols -
    q_len) all lie below w(r); the columns from w(r) on are all masked and are
    the ones a P.V product issued per row block of `block` rows never reads
    (the dead stores of the causal mask, Appendix A, Planner item 9)."""
    s = np.arange(rows, dtype=np.int64) % q_len
    w = (s // block + 1) * block + (cols - q_len)
    return np.clip(w, 0, cols)


def byte_mask_additive(m):
    """Additive mask of a byte mask: -inf where the byte is nonzero (the
    position is excluded), 0 where it is zero.  The paper's fused softmax
    takes an additive mask (Appendix A, Planner item 9); a byte mask is the
    same {0, -inf} mask stored in one byte per element."""
    m = np.asarray(m)
    return np.where(m != 0, -np.inf, 0.0)


def row_softmax(x, mask=None, scale: float = 1.0, causal_q_len: int = 0):
    """y[r] = softmax_j(x[r, j] * scale + mask[r, j]) along the last dim.

    Appendix A (Planner item 9: fused softmax; Codegen prompt: online
    softmax).  ``mask`` is additive (0 or -inf); ``causal_q_len > 0`` also
    masks the upper triangle by the causal rule.  Entries whose logit is -inf
    come out exactly 0; a fully masked row comes out all zeros.
    """
    x = np.asarray(x, dtype=np.float64)
    a = x * float(scale)
    if mask is not None:
        a = a + np.asarray(mask, dtype=np.float64)
    if causal_q_len:
        a = np.where(causal_mask(a.shape[0], a.shape[1], causal_q_len), -np.inf, a)
    m = a.max(axis=1, keepdims=True)
    empty = ~np.isfinite(m)
    m_safe = np.where(empty, 0.0, m)
    e = np.exp(a - m_safe)               # exp(-inf) = 0 for masked entries
    d = e.sum(axis=1, keepdims=True)
    d_safe = np.where(d > 0.0, d, 1.0)
    return np.where(empty, 0.0, e / d_safe)


# ---------------------------------------------------------------------------
# a3: LayerNorm fused with the residual add
# ---------------------------------------------------------------------------
def layernorm_residual(x, residual=None, gamma=None, beta=None, eps: float = 1e-5):
    """h = x + residual; y = (h - mean) / sqrt(var + eps) * gamma + beta.

    Appendix A (Fusion Agent: normalisation fusion and residual + norm).
    The variance is the biased one (divide by cols).  Returns (y, h); h is
    the exact sum, the value the residual stream carries forward.
    """
    h = np.asarray(x, dtype=np.float64)
    if residual is not None:
        h = h + np.asarray(residual, dtype=np.float64)
    n = h.shape[1]
    mean = h.sum(axis=1, keepdims=True) / n
    var = ((h - mean) ** 2).sum(axis=1, keepdims=True) / n
    y = (h - mean) / np.sqrt(var + float(eps))
    if gamma is not None:
        y = y * np.asarray(gamma, dtype=np.float64)[None, :]
    if beta is not None:
        y = y + np.asarray(beta, dtype=np.float64)[None, :]
    return y, h


def rmsnorm_residual(x, residual=None, gamma=None, eps: float = 1e-6):
    """h = x + residual; y = h / sqrt(mean(h^2) + eps) * gamma.

    The RMS variant of the normalisation fusion (Appendix A, Fusion Agent:
    LayerNorm/RMSNorm sequences): no mean subtraction and no bias.  Returns
    (y, h)."""
    h = np.asarray(x, dtype=np.float64)
    if residual is not None:
        h = h + np.asarray(residual, dtype=np.float64)
    ms = (h * h).sum(axis=1, keepdims=True) / h.shape[1]
    y = h / np.sqrt(ms + float(eps))
    if gamma is not None:
        y = y * np.asarray(gamma, dtype=np.float64)[None, :]
    return y, h


def round_to_bf16(v) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (8 significant bits,
    ties to even, bf16 exponent range), returned as float64.

    Written from the format's definition: a value m * 2**e with m in
    [0.5, 1) keeps 8 significant bits, so its quantum is 2**(e - 8); below
    the smallest normal the quantum stays at 2**-133.
    """
    v = np.asarray(v, dtype=np.float64)
    out = np.array(v, copy=True)
    fin = np.isfinite(v) & (v != 0.0)
    _, e = np.frexp(v[fin])
    q = np.ldexp(1.0, np.maximum(e, -125) - 8)
    r = np.rint(v[fin] / q) * q          # numpy rint rounds halves to even
    big = np.abs(r) > 3.3895313892515355e38   # largest finite bf16
    r = np.where(big, np.copysign(np.inf, r), r)
    out[fin] = r
    return out


def residual_store_bf16(x, residual) -> np.ndarray:
    """The stored residual of the bf16 LayerNorm: the float32 sum of the two
    bf16 inputs, rounded to bf16 (the fp32 add is part of the definition:
    reductions and intermediates live in fp32, the cast to the storage dtype
    happens once, on the store)."""
    s = np.asarray(x, dtype=np.float32) + np.asarray(residual, dtype=np.float32)
    return round_to_bf16(s.astype(np.float64))


# ---------------------------------------------------------------------------
# a4: GEMM epilogue with a row reduction
# ---------------------------------------------------------------------------
def gemm_epilogue_reduce(c, bias=None, col_scale=None, act: str = "sigmoid",
                         reduce: str = "sum"):
    """out[i] = reduce_j act((C[i, j] + bias[j]) * col_scale[j]).

    Appendix A (Codegen prompt: keep the matmul a library call, fuse only the
    epilogue; Fusion Agent: reduction + pointwise).  ``reduce`` is "sum",
    "mean", "max" or "logsumexp" over the columns (the last two as in
    ``row_reduce``: the reductions the paper's level-2 case study chains
    after a linear layer).
    """
    c = np.asarray(c, dtype=np.float64)
    t = c
    if bias is not None:
        t = t + np.asarray(bias, dtype=np.float64)[None, :]
    if col_scale is not None:
        t = t * np.asarray(col_scale, dtype=np.float64)[None, :]
    v = apply_act(t, act)
    if reduce in ("max", "logsumexp"):
        return row_reduce(v, reduce)
    s = v.sum(axis=1)
    if reduce == "sum":
        return s
    if reduce == "mean":
        return s / c.shape[1]
    raise ValueError(f"unknown reduction {reduce!r}")


# ---------------------------------------------------------------------------
# plain row reductions
# ---------------------------------------------------------------------------
def row_reduce(x, op: str = "sum"):
    """out[i] = sum_j x[i, j] ("sum"), that divided by cols ("mean"),
    max_j x[i, j] ("max") or log sum_j exp(x[i, j]) ("logsumexp").  Section 6
    lists sum/mean reductions among the optimised sub-kernel classes; the
    reduction + pointwise fusion pattern is in Appendix A (Fusion Agent); the
    paper's level-2 case study chains a linear layer with sum, max, mean and
    log-sum-exp reductions along the row.

    logsumexp is evaluated as m + log(sum_j exp(x[i, j] - m)) with m the row
    maximum (the same value, without overflow): a row of -inf gives -inf, a
    +inf entry gives +inf and a NaN gives NaN."""
    x = np.asarray(x, dtype=np.float64)
    if op == "sum":
        return x.sum(axis=1)
    if op == "mean":
        return x.sum(axis=1) / x.shape[1]
    if op == "max":
        return x.max(axis=1)
    if op == "logsumexp":
        m = x.max(axis=1)
        out = np.empty(x.shape[0])
        for i in range(x.shape[0]):
            if np.isnan(m[i]) or np.isinf(m[i]):
                out[i] = m[i]          # NaN, +inf, or a row of -inf
            else:
                out[i] = m[i] + math.log(np.exp(x[i] - m[i]).sum())
        return out
    raise ValueError(f"unknown reduction {op!r}")


def row_argmax(x):
    """Index of the largest element of every row; the lowest index wins a
    tie and a NaN counts as larger than any number (the first NaN wins).

    Exact by definition: it is written as an explicit comparison scan, not
    as a library call, so the tie and NaN rules are visible."""
    x = np.asarray(x, dtype=np.float64)
    rows, cols = x.shape
    out = np.zeros(rows, dtype=np.int64)
    nan = np.isnan(x)
    for i in range(rows):
        if nan[i].any():
            out[i] = int(np.flatnonzero(nan[i])[0])
            continue
        row = x[i]
        best = row.max()
        out[i] = int(np.flatnonzero(row == best)[0])   # lowest index of the maximum
    return out


# ---------------------------------------------------------------------------
# layout transform
# ---------------------------------------------------------------------------
def strided_copy(src_flat, dst_flat, rows: int, cols: int, batch: int, ld_src: int,
                 stride_src: int, ld_dst: int, stride_dst: int):
    """The copy a compiled graph inserts when permuted strides must become
    contiguous (Section 4.4, Gate 4): returns a copy of the flat destination
    with dst[b*stride_dst + r*ld_dst + c] = src[b*stride_src + r*ld_src + c]
    for every b < batch, r < rows, c < cols; other destination elements keep
    their values.  Works on any 1-D array (values or raw bit patterns)."""
    src = np.asarray(src_flat).reshape(-1)
    out = np.array(dst_flat, copy=True).reshape(-1)
    for b in range(batch):
        for r in range(rows):
            s0 = b * stride_src + r * ld_src
            d0 = b * stride_dst + r * ld_dst
            out[d0:d0 + cols] = src[s0:s0 + cols]
    return out
