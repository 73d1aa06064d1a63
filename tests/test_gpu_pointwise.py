"""GPU parity of fs_pointwise_chain against the float64 oracle."""
import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
import paper_2609_30059_amd as fs
from gpu_util import (SEEDS, TOL, Guarded, announce, assert_close, bf16_ulp_close, dev, host64,
                      rho)

pytestmark = pytest.mark.gpu


def run_case(rows, cols, dtype, act, seed=0, bias=True, residual=True, scale=0.7):
    d = fd.pointwise_inputs(seed, rows, cols, dtype, scale, bias, residual)
    announce("pointwise", rows, cols, dtype, act, seed, bias, residual)
    y = fs.pointwise_chain(dev(d["x"]), dev(d["bias"]), dev(d["residual"]), d["scale"], act)
    torch.cuda.synchronize()
    ref = oracle.pointwise_chain(d["x"].f64(), d["bias"].f64() if bias else None,
                                 d["residual"].f64() if residual else None, d["scale"], act)
    return d, host64(y), ref


@pytest.mark.parametrize("seed", SEEDS)
def test_256x1024_fp32_gelu_five_seeds(seed):
    d, got, ref = run_case(256, 1024, "f32", "gelu_erf", seed)
    assert_close(f"pointwise_256x1024 seed {seed}", got, ref, *TOL["f32"])
    # Gate-3 style diagnostic: an unfused torch fp32 evaluation as r32
    x, b, r = (torch.from_numpy(d[k].data) for k in ("x", "bias", "residual"))
    r32 = torch.nn.functional.gelu(x * d["scale"] + b) + r
    assert rho(got, r32.double().numpy(), ref) <= 10


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("act", ["none", "gelu_erf", "sigmoid", "relu"])
@pytest.mark.parametrize("shape", [(1, 1), (3, 7), (37, 1003), (5, 2048), (17, 4104), (2, 9000)])
def test_shapes_and_acts(dtype, act, shape):
    _, got, ref = run_case(*shape, dtype, act, seed=shape[1])
    assert_close(f"{shape} {dtype} {act}", got, ref, *TOL[dtype])
    if dtype == "bf16":
        bf16_ulp_close(f"{shape} {act}", got, ref)


# rows that are not whole 16-byte vectors: odd widths around the column
# blocks' edges (2048 bf16 / 1024 fp32 columns) and below two vectors (15);
# 2100 rows take several rows per trip
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(9, 15), (9, 17), (6, 1025), (5, 2047), (4, 2055), (4, 2063),
                                   (3, 4097), (2100, 1001)])
def test_odd_rows(dtype, shape):
    _, got, ref = run_case(*shape, dtype, "gelu_erf", seed=shape[1] + 1)
    assert_close(f"{shape} {dtype}", got, ref, *TOL[dtype])
    if dtype == "bf16":
        bf16_ulp_close(f"{shape}", got, ref)


@pytest.mark.parametrize("bias,residual", [(False, True), (True, False), (False, False)])
@pytest.mark.parametrize("rows,cols", [(33, 1024), (2100, 1001)])
def test_optional_operands_odd_rows(bias, residual, rows, cols):
    _, got, ref = run_case(rows, cols, "bf16", "sigmoid", 6, bias, residual)
    assert_close("optional odd rows", got, ref, *TOL["bf16"])


@pytest.mark.parametrize("bias,residual", [(False, True), (True, False), (False, False)])
def test_optional_operands(bias, residual):
    _, got, ref = run_case(33, 1024, "f32", "gelu_erf", 5, bias, residual)
    assert_close("optional", got, ref, *TOL["f32"])


def test_zero_scale_and_bias_is_exact_residual():
    d = fd.pointwise_inputs(3, 64, 1024, "bf16")
    x, r = dev(d["x"]), dev(d["residual"])
    y = fs.pointwise_chain(x, torch.zeros(1024, dtype=torch.bfloat16, device="cuda"), r, 0.0,
                           "gelu_erf")
    assert torch.equal(y, r)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_strided_misaligned_and_guard_bands(dtype):
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rows, cols, ld = 19, 1000, 1027
    d = fd.pointwise_inputs(11, rows, cols, dtype)
    ref = oracle.pointwise_chain(d["x"].f64(), d["bias"].f64(), d["residual"].f64(), d["scale"],
                                 "gelu_erf")
    for offset in (0, 1):          # offset 1 element: scalar path
        announce("pointwise guard", dtype, offset)
        xg = Guarded(rows, cols, ld, tdt, offset=offset)
        xg.view.copy_(dev(d["x"]))
        yg = Guarded(rows, cols, ld + 5, tdt, offset=offset)
        fs.pointwise_chain(xg.view, dev(d["bias"]), dev(d["residual"]), d["scale"], "gelu_erf",
                           out=yg.view)
        torch.cuda.synchronize()
        assert_close(f"strided offset {offset}", host64(yg.view), ref, *TOL[dtype])
        yg.check_untouched("pointwise y")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_strided_same_phase_rows(dtype):
    # x, residual and y share one odd row stride and offset: every row starts
    # at the same offset within a 16-byte unit in all three, and at a
    # different one from row to row
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rows, cols, ld = 23, 3001, 3013
    d = fd.pointwise_inputs(12, rows, cols, dtype)
    ref = oracle.pointwise_chain(d["x"].f64(), d["bias"].f64(), d["residual"].f64(), d["scale"],
                                 "relu")
    for offset in (1, 3):
        announce("pointwise same-phase strided", dtype, offset)
        xg = Guarded(rows, cols, ld, tdt, offset=offset)
        rg = Guarded(rows, cols, ld, tdt, offset=offset)
        yg = Guarded(rows, cols, ld, tdt, offset=offset)
        xg.view.copy_(dev(d["x"]))
        rg.view.copy_(dev(d["residual"]))
        fs.pointwise_chain(xg.view, dev(d["bias"]), rg.view, d["scale"], "relu", out=yg.view)
        torch.cuda.synchronize()
        assert_close(f"same-phase offset {offset}", host64(yg.view), ref, *TOL[dtype])
        yg.check_untouched("pointwise y")


def test_in_place_odd_rows():
    d = fd.pointwise_inputs(8, 41, 2047, "bf16")
    ref = oracle.pointwise_chain(d["x"].f64(), d["bias"].f64(), d["residual"].f64(), d["scale"],
                                 "gelu_erf")
    x, b, r = dev(d["x"]), dev(d["bias"]), dev(d["residual"])
    fs.pointwise_chain(x, b, r, d["scale"], "gelu_erf", out=x)
    assert_close("in place on x, odd rows", host64(x), ref, *TOL["bf16"])


def test_in_place():
    d = fd.pointwise_inputs(7, 50, 2048, "bf16")
    ref = oracle.pointwise_chain(d["x"].f64(), d["bias"].f64(), d["residual"].f64(), d["scale"],
                                 "gelu_erf")
    x, b, r = dev(d["x"]), dev(d["bias"]), dev(d["residual"])
    fs.pointwise_chain(x, b, r, d["scale"], "gelu_erf", out=x)        # y == x
    assert_close("in place on x", host64(x), ref, *TOL["bf16"])
    x2 = dev(d["x"])
    fs.pointwise_chain(x2, b, r, d["scale"], "gelu_erf", out=r)       # y == residual
    assert_close("in place on residual", host64(r), ref, *TOL["bf16"])


def test_empty():
    x = torch.empty(0, 64, device="cuda")
    assert fs.pointwise_chain(x).shape == (0, 64)


@pytest.mark.slow
def test_beyond_2_31_elements():
    # rows * cols > 2^31 exercises 64-bit offsets; the input repeats a seeded
    # block so the sampled rows are known on the host
    rows, cols = (1 << 21) + 3, 1024
    d = fd.pointwise_inputs(2, 64, cols, "bf16")
    announce("pointwise > 2^31 elements", rows, cols)
    xb, rb = dev(d["x"]), dev(d["residual"])
    x = xb.repeat((rows + 63) // 64, 1)[:rows]
    r = rb.repeat((rows + 63) // 64, 1)[:rows]
    y = fs.pointwise_chain(x, dev(d["bias"]), r, d["scale"], "gelu_erf")
    idx = np.array([0, 63, 64, rows // 2, rows - 2, rows - 1])
    got = host64(y[torch.from_numpy(idx).cuda()])
    ref = oracle.pointwise_chain(d["x"].rows(idx % 64).f64(), d["bias"].f64(),
                                 d["residual"].rows(idx % 64).f64(), d["scale"], "gelu_erf")
    assert_close("beyond 2^31", got, ref, *TOL["bf16"])


# dense rows without a bias walk one flat run of 16-byte vectors (large
# tensors only): acts, scale, with and without a residual, a vector count that
# leaves a tail past the last whole chunk, and in place
@pytest.mark.parametrize("dtype,rows,cols", [("bf16", 16387, 1000), ("f32", 4201, 1000),
                                             ("bf16", 2048, 8192)])
@pytest.mark.parametrize("act", ["none", "gelu_erf", "sigmoid", "relu"])
@pytest.mark.parametrize("residual", [True, False])
def test_flat_dense_rows(dtype, rows, cols, act, residual):
    d, got, ref = run_case(rows, cols, dtype, act, seed=rows + cols, bias=False, residual=residual,
                           scale=0.8)
    assert_close(f"flat {rows}x{cols} {dtype} {act}", got, ref, *TOL[dtype])
    if dtype == "bf16":
        bf16_ulp_close(f"flat {rows}x{cols} {act}", got, ref)


def test_flat_dense_rows_in_place():
    d = fd.pointwise_inputs(91, 16385, 1024, "bf16", with_bias=False)
    ref = oracle.pointwise_chain(d["x"].f64(), None, d["residual"].f64(), d["scale"], "none")
    x, r = dev(d["x"]), dev(d["residual"])
    announce("flat in place")
    fs.pointwise_chain(x, None, r, d["scale"], "none", out=r)          # y == residual
    assert_close("flat in place on residual", host64(r), ref, *TOL["bf16"])
    x2, r2 = dev(d["x"]), dev(d["residual"])
    fs.pointwise_chain(x2, None, r2, d["scale"], "none", out=x2)        # y == x
    assert_close("flat in place on x", host64(x2), ref, *TOL["bf16"])
