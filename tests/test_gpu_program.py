"""GPU parity of fs_pointwise_program against the float64 oracle."""
import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
import paper_2609_30059_amd as fs
from gpu_util import SEEDS, TOL, Guarded, announce, assert_close, dev, host64

pytestmark = pytest.mark.gpu

# the paper's fused group after a linear layer: bias, a multiply, a hardtanh
# and a GELU
LINEAR_MUL_HARDTANH_GELU = [("add_bias",), ("scale", 0.5), ("clamp", -1.0, 1.0), ("gelu_erf",)]
# one of every operation (the column vector is the bias again, scaled)
EVERY_OP = [("scale", 0.8), ("shift", 0.1), ("add_bias",), ("mul_column",), ("add_residual",),
            ("tanh",), ("mul_residual",), ("leaky_relu", 0.2), ("clamp", -2.0, 2.0), ("silu",),
            ("sigmoid",), ("shift", -0.5), ("relu",), ("gelu_erf",)]


def inputs(seed, rows, cols, dtype):
    d = fd.pointwise_inputs(seed, rows, cols, dtype)
    col = fd.Tensor(np.ascontiguousarray(d["bias"].data[::-1]), dtype)   # another [cols] vector
    return d, col


def run(d, col, ops, dtype, **kw):
    x = dev(d["x"])
    y = fs.pointwise_program(x, ops, bias=dev(d["bias"]), col=dev(col),
                             residual=dev(d["residual"]), **kw)
    ref = oracle.pointwise_program(d["x"].f64(), ops, d["bias"].f64(), col.f64(),
                                   d["residual"].f64())
    return host64(y), ref


@pytest.mark.parametrize("seed", SEEDS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_linear_mul_hardtanh_gelu_five_seeds(seed, dtype):
    d, col = inputs(seed, 256, 4096, dtype)
    announce("program mul-hardtanh-gelu", seed, dtype)
    got, ref = run(d, col, LINEAR_MUL_HARDTANH_GELU, dtype)
    assert_close(f"seed {seed} {dtype}", got, ref, *TOL[dtype])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("op", [o for o in EVERY_OP if o != ("shift", -0.5)],
                         ids=lambda o: o[0])
# vector rows, element-wise rows (width not a whole number of vectors), one row
@pytest.mark.parametrize("shape", [(37, 1024), (9, 1003), (1, 4104)])
def test_each_operation(dtype, op, shape):
    d, col = inputs(shape[1], *shape, dtype)
    announce("program op", op[0], shape, dtype)
    got, ref = run(d, col, [op], dtype)
    assert_close(f"{op} {shape} {dtype}", got, ref, *TOL[dtype])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(300, 1000), (70000, 256), (5, 9001)])
def test_every_operation_in_one_program(dtype, shape):
    # [70000, 256]: more row groups than the grid, so blocks loop over trips
    d, col = inputs(7, *shape, dtype)
    announce("program every op", shape, dtype)
    got, ref = run(d, col, EVERY_OP, dtype)
    assert_close(f"{shape} {dtype}", got, ref, *TOL[dtype])


def test_sixteen_operations():
    ops = [("scale", 1.01), ("shift", -0.01)] * 8
    d, col = inputs(3, 64, 512, "f32")
    got, ref = run(d, col, ops, "f32")
    assert_close("16 operations", got, ref, *TOL["f32"])
    with pytest.raises(fs.FusedSubError):
        fs.pointwise_program(dev(d["x"]), ops + [("relu",)])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_empty_program_copies_bit_for_bit(dtype):
    d, _ = inputs(4, 33, 777, dtype)
    x = dev(d["x"])
    y = fs.pointwise_program(x, [])
    assert torch.equal(y.view(torch.int16 if dtype == "bf16" else torch.int32),
                       x.view(torch.int16 if dtype == "bf16" else torch.int32))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_in_place_on_x_and_on_the_residual(dtype):
    d, col = inputs(5, 40, 2048, dtype)
    ops = [("scale", 0.5), ("add_residual",), ("silu",)]
    ref = oracle.pointwise_program(d["x"].f64(), ops, residual=d["residual"].f64())
    x, r = dev(d["x"]), dev(d["residual"])
    fs.pointwise_program(x, ops, residual=r, out=x)
    assert_close("in place on x", host64(x), ref, *TOL[dtype])
    x, r = dev(d["x"]), dev(d["residual"])
    fs.pointwise_program(x, ops, residual=r, out=r)
    assert_close("in place on the residual", host64(r), ref, *TOL[dtype])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("offset", [0, 1])
def test_strided_rows_and_guard_bands(dtype, offset):
    # rows 900 wide with row stride 912, starting `offset` elements into an
    # allocation (offset 1: not 16-byte aligned, the element-wise path);
    # nothing outside the rows is written
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rows, cols, ld = 21, 900, 912
    d, col = inputs(11 + offset, rows, cols, dtype)
    announce("program strided", dtype, offset)
    xg = Guarded(rows, cols, ld, tdt, offset=offset)
    xg.view.copy_(dev(d["x"]))
    rg = Guarded(rows, cols, ld, tdt, offset=offset)
    rg.view.copy_(dev(d["residual"]))
    yg = Guarded(rows, cols, ld, tdt, offset=offset)
    ops = [("mul_column",), ("add_residual",), ("tanh",), ("add_bias",)]
    fs.pointwise_program(xg.view, ops, bias=dev(d["bias"]), col=dev(col), residual=rg.view,
                         out=yg.view)
    torch.cuda.synchronize()
    ref = oracle.pointwise_program(d["x"].f64(), ops, d["bias"].f64(), col.f64(),
                                   d["residual"].f64())
    assert_close(f"strided offset {offset}", host64(yg.view), ref, *TOL[dtype])
    yg.check_untouched("program y")
    xg.check_untouched("program x")


def test_special_values():
    # NaN stays NaN through clamp, ReLU and leaky ReLU; infinities saturate
    x = torch.tensor([[float("nan"), float("inf"), float("-inf"), -3.0, 0.25, 3.0, -0.0, 1e-30]],
                     device="cuda").repeat(4, 1)
    # (GELU is left out: at -inf the oracle's z (1 + erf(z / sqrt 2)) / 2 is
    # -inf * 0 = NaN, where the kernel returns the limit 0)
    for ops in ([("clamp", -1.0, 1.0)], [("relu",)], [("leaky_relu", 0.1)], [("tanh",)],
                [("sigmoid",)], [("clamp", float("-inf"), 0.5)]):
        y = host64(fs.pointwise_program(x, ops))
        ref = oracle.pointwise_program(host64(x), ops)
        assert np.array_equal(np.isnan(y), np.isnan(ref)), ops
        fin = ~np.isnan(ref)
        assert_close(str(ops), y[fin], ref[fin], *TOL["f32"])


def test_matches_the_fixed_chain():
    # the fixed chain act(x * s + b) + r as a program: both against the oracle
    d, col = inputs(12, 128, 2048, "f32")
    ops = [("scale", d["scale"]), ("add_bias",), ("gelu_erf",), ("add_residual",)]
    got, ref = run(d, col, ops, "f32")
    chain = host64(fs.pointwise_chain(dev(d["x"]), dev(d["bias"]), dev(d["residual"]), d["scale"],
                                      "gelu_erf"))
    ref_chain = oracle.pointwise_chain(d["x"].f64(), d["bias"].f64(), d["residual"].f64(),
                                       d["scale"], "gelu_erf")
    np.testing.assert_allclose(ref, ref_chain, rtol=1e-15, atol=1e-15)
    assert_close("program", got, ref, *TOL["f32"])
    assert_close("chain", chain, ref, *TOL["f32"])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_relu_keeps_nan_in_the_fixed_chain_and_the_epilogue(dtype):
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    x = torch.tensor([[float("nan"), -1.0, 2.0, -0.0]], device="cuda").repeat(3, 4).to(tdt)
    y = host64(fs.pointwise_chain(x, None, None, 1.0, "relu"))
    assert np.isnan(y[:, 0::4]).all() and (y[:, 1::4] == 0).all() and (y[:, 2::4] == 2).all()
    c = torch.zeros(5, 8192, device="cuda").to(tdt)
    c[2, 100] = float("nan")
    o = host64(fs.gemm_epilogue_reduce(c, None, None, "relu", "sum"))
    assert np.isnan(o[2]) and (o[[0, 1, 3, 4]] == 0).all()


PROGRAMS = {
    "every": EVERY_OP,
    "bias_only": [("scale", 1.5), ("add_bias",), ("gelu_erf",)],
    "column_only": [("mul_column",), ("tanh",), ("add_residual",)],
    "plain": [("shift", 0.25), ("silu",), ("clamp", -0.5, 2.0)],
}


def bits(t):
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).cpu().numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
# rows that are not whole 16-byte vectors: the aligned body (rows of at
# least two vectors), with several trips of four rows per block and a ragged
# last trip ([5001, 1003]), wide rows of several column blocks, and rows of
# 9 columns (two fp32 vectors; fewer than two bf16 vectors: element-wise)
@pytest.mark.parametrize("shape", [(5001, 1003), (130, 4099), (2050, 17), (3000, 9)])
@pytest.mark.parametrize("prog", sorted(PROGRAMS))
def test_odd_width_rows(dtype, shape, prog):
    ops = PROGRAMS[prog]
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    d, col = inputs(shape[0] + shape[1], *shape, dtype)
    announce("program odd rows", shape, dtype, prog)
    x, b, c, r = dev(d["x"]), dev(d["bias"]), dev(col), dev(d["residual"])
    y = fs.pointwise_program(x, ops, bias=b, col=c, residual=r)
    ref = oracle.pointwise_program(d["x"].f64(), ops, d["bias"].f64(), col.f64(),
                                   d["residual"].f64())
    assert_close(f"{shape} {dtype} {prog}", host64(y), ref, *TOL[dtype])
    # y one element into a wider buffer: its rows sit at another phase than
    # x's, which takes the element-wise path -- the same fp32 arithmetic per
    # element, so the same bits
    buf = torch.zeros(shape[0] * shape[1] + 1, dtype=tdt, device="cuda")
    ye = buf[1:].view(shape)
    fs.pointwise_program(x, ops, bias=b, col=c, residual=r, out=ye)
    np.testing.assert_array_equal(bits(y), bits(ye))
    assert buf[0].item() == 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_odd_width_rows_in_place_and_strided(dtype):
    # x, residual and y in strided buffers whose rows start at one phase that
    # changes from row to row (ld 1011): the aligned body in place on x and
    # on the residual, nothing outside the rows written
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rows, cols, ld = 1500, 1001, 1011
    ops = [("mul_column",), ("add_residual",), ("gelu_erf",), ("add_bias",), ("mul_residual",)]
    d, col = inputs(rows + cols, rows, cols, dtype)
    announce("program odd rows in place", dtype)
    ref = oracle.pointwise_program(d["x"].f64(), ops, d["bias"].f64(), col.f64(),
                                   d["residual"].f64())
    for target in ("x", "residual"):
        xg = Guarded(rows, cols, ld, tdt, offset=3)
        xg.view.copy_(dev(d["x"]))
        rg = Guarded(rows, cols, ld, tdt, offset=3)
        rg.view.copy_(dev(d["residual"]))
        out = xg.view if target == "x" else rg.view
        fs.pointwise_program(xg.view, ops, bias=dev(d["bias"]), col=dev(col), residual=rg.view,
                             out=out)
        torch.cuda.synchronize()
        assert_close(f"in place on {target}", host64(out), ref, *TOL[dtype])
        xg.check_untouched("x")
        rg.check_untouched("residual")
