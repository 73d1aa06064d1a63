"""The C ABI from a program with no Python and no PyTorch in it.

tests/abi_consumer.cpp (built next to libfusedsub.so by the package build)
allocates with hipMalloc, copies the seeded inputs in, calls one entry point
on the null stream and writes the outputs back.  Each case here writes the
inputs of the shared generators to a temporary directory, runs the program as
a child process, and checks its outputs against the float64 oracle at the
contract tolerances -- and bit for bit against the same call made through the
Python binding on torch's stream (same kernels, same inputs).
"""
import os
import subprocess

import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
import paper_2609_30059_amd as fs
from paper_2609_30059_amd import _native as N
from paper_2609_30059_amd.build import ABI_CONSUMER
from gpu_util import (TOL, announce, assert_close, bf16_ulp_close, dev, host64,
                      softmax_supplementary)

pytestmark = pytest.mark.gpu

# fp32 tree sum of 8192 terms below 1: |error| <= log2(8192) * ulp(4096) ~ 5e-3
SUM_ATOL = 5e-3


def run_consumer(case, tmp_path, rows, cols, p1, p2, arrays):
    assert os.access(ABI_CONSUMER, os.X_OK), \
        f"{ABI_CONSUMER} is not built (python -m paper_2609_30059_amd.build)"
    for name, a in arrays.items():
        np.ascontiguousarray(a).tofile(str(tmp_path / f"{name}.bin"))
    (tmp_path / "dims.txt").write_text(f"{rows} {cols} {p1!r} {p2!r}\n")
    announce("abi consumer", case, rows, cols)
    r = subprocess.run([ABI_CONSUMER, case, str(tmp_path)], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 0, (r.stdout + r.stderr)[-2000:]
    assert f"abi_consumer {case}: ok" in r.stdout


def load(tmp_path, name, dtype, shape):
    raw = np.fromfile(str(tmp_path / f"{name}.bin"), dtype=dtype)
    assert raw.size == int(np.prod(shape)), f"{name}: {raw.size} elements"
    return raw.reshape(shape)


def bits_of(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.cpu().view(torch.int16).numpy().view(np.uint16)
    return t.cpu().view(torch.int32).numpy().view(np.uint32)


def test_pointwise_chain_fp32(tmp_path):
    rows, cols = 300, 1000
    d = fd.pointwise_inputs(11, rows, cols, "f32")
    run_consumer("pointwise", tmp_path, rows, cols, d["scale"], 0,
                 {"x": d["x"].data, "bias": d["bias"].data, "residual": d["residual"].data})
    y = load(tmp_path, "y", np.float32, (rows, cols))
    ref = oracle.pointwise_chain(d["x"].f64(), d["bias"].f64(), d["residual"].f64(),
                                 d["scale"], "gelu_erf")
    assert_close("pointwise via the C ABI", y.astype(np.float64), ref, *TOL["f32"])
    yt = fs.pointwise_chain(dev(d["x"]), dev(d["bias"]), dev(d["residual"]), d["scale"],
                            "gelu_erf")
    np.testing.assert_array_equal(y.view(np.uint32), bits_of(yt))


def test_masked_softmax_bf16(tmp_path):
    rows, cols = 257, 4096
    d = fd.softmax_inputs(12, rows, cols)
    run_consumer("softmax", tmp_path, rows, cols, d["scale"], 0,
                 {"x": d["x"].data, "mask": d["mask"].data})
    yb = load(tmp_path, "y", np.uint16, (rows, cols))
    got = fd.bf16_bits_to_f64(yb)
    ref = oracle.row_softmax(d["x"].f64(), d["mask"].f64(), d["scale"])
    assert_close("softmax via the C ABI", got, ref, *TOL["bf16"])
    softmax_supplementary("softmax via the C ABI", got, ref, np.isinf(d["mask"].f64()))
    yt = fs.row_softmax(dev(d["x"]), dev(d["mask"]), d["scale"])
    np.testing.assert_array_equal(yb, bits_of(yt))


def test_causal_softmax_bf16(tmp_path):
    # [2 heads x 512 queries, 512 keys], causal with q_len 512, no mask
    rows, cols, q = 1024, 512, 512
    d = fd.softmax_inputs(13, rows, cols, mask_dtype=None)
    zero_mask = np.zeros((rows, cols), np.uint16)    # +0 in bf16: the additive mask is a no-op
    run_consumer("softmax", tmp_path, rows, cols, d["scale"], q,
                 {"x": d["x"].data, "mask": zero_mask})
    yb = load(tmp_path, "y", np.uint16, (rows, cols))
    got = fd.bf16_bits_to_f64(yb)
    ref = oracle.row_softmax(d["x"].f64(), None, d["scale"], causal_q_len=q)
    assert_close("causal softmax via the C ABI", got, ref, *TOL["bf16"])
    bf16_ulp_close("causal softmax via the C ABI", got, ref, ulps=1.0, atol=1e-7)
    masked = oracle.causal_mask(rows, cols, q)
    assert np.all(yb[masked] == 0), "causally masked entries are not +0"
    yt = fs.row_softmax(dev(d["x"]), dev(fd.Tensor(zero_mask, "bf16")), d["scale"],
                        causal_q_len=q)
    np.testing.assert_array_equal(yb, bits_of(yt))


def test_layernorm_residual_bf16(tmp_path):
    rows, cols = 333, 4096
    d = fd.layernorm_inputs(14, rows, cols)
    run_consumer("layernorm", tmp_path, rows, cols, d["eps"], 0,
                 {"x": d["x"].data, "residual": d["residual"].data, "gamma": d["gamma"].data,
                  "beta": d["beta"].data})
    yb = load(tmp_path, "y", np.uint16, (rows, cols))
    rb = load(tmp_path, "residual_out", np.uint16, (rows, cols))
    got = fd.bf16_bits_to_f64(yb)
    ref, _ = oracle.layernorm_residual(d["x"].f64(), d["residual"].f64(), d["gamma"].f64(),
                                       d["beta"].f64(), d["eps"])
    assert_close("layernorm via the C ABI", got, ref, *TOL["bf16"])
    bf16_ulp_close("layernorm via the C ABI", got, ref, ulps=1.0, atol=2e-5)
    np.testing.assert_array_equal(fd.bf16_bits_to_f64(rb),
                                  oracle.residual_store_bf16(d["x"].f64(), d["residual"].f64()))
    yt, rt = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]),
                                   dev(d["beta"]), d["eps"])
    np.testing.assert_array_equal(yb, bits_of(yt))
    np.testing.assert_array_equal(rb, bits_of(rt))


def test_gemm_epilogue_sigmoid_sum(tmp_path):
    rows, cols = 300, 8192
    d = fd.epilogue_inputs(15, rows, cols)
    run_consumer("epilogue", tmp_path, rows, cols, 0, 0,
                 {"c": d["c"].data, "bias": d["bias"].data, "scale": d["col_scale"].data})
    out = load(tmp_path, "out", np.float32, (rows,))
    ref = oracle.gemm_epilogue_reduce(d["c"].f64(), d["bias"].f64(), d["col_scale"].f64(),
                                      "sigmoid", "sum")
    assert_close("epilogue via the C ABI", out.astype(np.float64), ref, *TOL["bf16"])
    assert_close("epilogue via the C ABI (sum)", out.astype(np.float64), ref, SUM_ATOL, 0.0)
    ot = fs.gemm_epilogue_reduce(dev(d["c"]), dev(d["bias"]), dev(d["col_scale"]), "sigmoid",
                                 "sum")
    np.testing.assert_array_equal(out.view(np.uint32), bits_of(ot))


def test_pointwise_program_bf16(tmp_path):
    # the paper's group after a linear layer (bias, multiply, hardtanh, GELU)
    # with a column multiply, a residual and a leaky ReLU around it; the
    # fs_op array is built by the C++ program from "code a b" lines
    rows, cols = 300, 1000
    ops = [("mul_column",), ("add_bias",), ("scale", 0.5), ("clamp", -1.0, 1.0), ("gelu_erf",),
           ("add_residual",), ("leaky_relu", 0.05)]
    d = fd.pointwise_inputs(16, rows, cols, "bf16")
    col = fd.Tensor(np.ascontiguousarray(d["bias"].data[::-1]), "bf16")
    lines = []
    for op in ops:
        prm = list(op[1:]) + [0.0] * (2 - len(op[1:]))
        lines.append(f"{N.PROGRAM_OPS[op[0]][0]} {prm[0]!r} {prm[1]!r}")
    (tmp_path / "ops.txt").write_text("\n".join(lines) + "\n")
    run_consumer("program", tmp_path, rows, cols, 0, 0,
                 {"x": d["x"].data, "bias": d["bias"].data, "col": col.data,
                  "residual": d["residual"].data})
    yb = load(tmp_path, "y", np.uint16, (rows, cols))
    ref = oracle.pointwise_program(d["x"].f64(), ops, d["bias"].f64(), col.f64(),
                                   d["residual"].f64())
    assert_close("program via the C ABI", fd.bf16_bits_to_f64(yb), ref, *TOL["bf16"])
    yt = fs.pointwise_program(dev(d["x"]), ops, bias=dev(d["bias"]), col=dev(col),
                              residual=dev(d["residual"]))
    np.testing.assert_array_equal(yb, bits_of(yt))


def test_byte_mask_softmax_bf16(tmp_path):
    rows, cols = 257, 4096
    d = fd.softmax_inputs(17, rows, cols, "bf16", mask_dtype="u8")
    run_consumer("softmax_u8", tmp_path, rows, cols, d["scale"], 0,
                 {"x": d["x"].data, "mask": d["mask"].data})
    yb = load(tmp_path, "y", np.uint16, (rows, cols))
    got = fd.bf16_bits_to_f64(yb)
    ref = oracle.row_softmax(d["x"].f64(), oracle.byte_mask_additive(d["mask"].data), d["scale"])
    assert_close("byte-mask softmax via the C ABI", got, ref, *TOL["bf16"])
    softmax_supplementary("byte-mask softmax via the C ABI", got, ref, d["mask"].data != 0)
    yt = fs.row_softmax(dev(d["x"]), dev(d["mask"]), d["scale"])
    np.testing.assert_array_equal(yb, bits_of(yt))


def test_row_logsumexp_bf16(tmp_path):
    rows, cols = 300, 8192
    x = fd.row_inputs(18, rows, cols, "bf16", mean=0.25, std=2.0)
    run_consumer("logsumexp", tmp_path, rows, cols, 0, 0, {"x": x.data})
    out = load(tmp_path, "out", np.float32, (rows,))
    # the bound of the row-reduce tests: the relative error of the fp32 sum
    # S >= 1 of exp(x - max) terms, plus the rounding of max + log S
    assert_close("logsumexp via the C ABI", out.astype(np.float64),
                 oracle.row_reduce(x.f64(), "logsumexp"), 2e-5, 2e-6)
    ot = fs.row_reduce(dev(x), "logsumexp")
    np.testing.assert_array_equal(out.view(np.uint32), bits_of(ot))
