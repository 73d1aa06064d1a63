"""GPU parity of the long-row softmax and LayerNorm/RMSNorm kernels against
the float64 oracle: rows past the 8-wave register rungs (16384 columns), the
16-wave rung (to 32768), the row cache in LDS and registers (to 65536) and its
streamed tail (columns past the cache, read twice), the row cache with
element-wise slots (softmax widths that are not a whole number of 16-byte
vectors) and LayerNorm's element-wise streamed kernel; ragged tails, causal
offsets, in-place outputs, rows whose running statistics must be rescaled
from one chunk to the next, and grids that loop over more rows than they
hold blocks."""
import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
import paper_2609_30059_amd as fs
from gpu_util import (TOL, Guarded, announce, assert_close, bf16_ulp_close, dev, host64)

pytestmark = pytest.mark.gpu

# 16-wave register rungs: 16392, 20000, 32768; row cache without a tail:
# 32776, 49160, 65536; with a tail: 65560, 131112, 262144; widths that are not
# whole 16-byte vectors take element-wise loads: the row cache without a tail
# (50001) and with one (100003)
LONG = [16384 + 8, 20000, 32768, 32768 + 8, 49160, 50001, 65536, 65536 + 24, 100003,
        131072 + 40, 262144]


# ---- softmax -----------------------------------------------------------------
@pytest.mark.parametrize("dtype,mask_dtype", [("f32", "f32"), ("bf16", "bf16"), ("bf16", None),
                                              ("f32", None), ("bf16", "f32")])
@pytest.mark.parametrize("cols", LONG)
def test_softmax_long_rows_widths(dtype, mask_dtype, cols):
    d = fd.softmax_inputs(cols + 7, 3, cols, dtype, mask_dtype=mask_dtype)
    announce("softmax long rows", cols, dtype, mask_dtype)
    y = fs.row_softmax(dev(d["x"]), dev(d["mask"]), d["scale"])
    got = host64(y)
    m = d["mask"].f64() if mask_dtype else None
    ref = oracle.row_softmax(d["x"].f64(), m, d["scale"])
    assert_close(f"cols {cols}", got, ref, *TOL[dtype])
    if dtype == "bf16":
        bf16_ulp_close(f"cols {cols}", got, ref, ulps=1.0, atol=1e-9)
    else:
        np.testing.assert_allclose(got.sum(axis=1), 1.0, rtol=1e-5)
    if m is not None:
        assert np.all(got[np.isinf(m)] == 0.0)


@pytest.mark.parametrize("cols", [50000, 100000])
@pytest.mark.parametrize("order", ["rising", "falling", "spike_last"])
def test_softmax_long_rows_running_max_moves(order, cols):
    # the running max changes in every chunk (rising), only in the first
    # (falling), or only in the last element of the row (spike_last); 50000
    # columns are all in the row cache, 100000 have a streamed tail
    base = np.linspace(-40.0, 40.0, cols)
    if order == "falling":
        base = base[::-1].copy()
    elif order == "spike_last":
        base = np.zeros(cols)
        base[-1] = 30.0
    x = np.stack([base, base * 0.5, -base]).astype(np.float32)
    announce("softmax long rows order", order, cols)
    y = host64(fs.row_softmax(torch.from_numpy(x).cuda(), None, 1.0))
    ref = oracle.row_softmax(x.astype(np.float64), None, 1.0)
    assert_close(order, y, ref, *TOL["f32"])
    np.testing.assert_allclose(y.sum(axis=1), 1.0, rtol=1e-5)


@pytest.mark.parametrize("q_len,cols,rows", [(5, 40000, 11), (64, 70000, 9), (3, 16400, 7),
                                             (25000, 40000, 3), (39990, 40000, 12),
                                             (7, 40001, 9), (4, 70001, 5)])
def test_softmax_long_rows_causal(q_len, cols, rows):
    # the causal limit falls near the row end, mid-row and within the first
    # chunk; 40001 and 70001 columns take element-wise loads
    d = fd.softmax_inputs(q_len * cols, rows, cols, "f32", mask_dtype="f32", p_masked=0.2)
    announce("softmax long rows causal", q_len, cols)
    y = fs.row_softmax(dev(d["x"]), dev(d["mask"]), d["scale"], causal_q_len=q_len)
    ref = oracle.row_softmax(d["x"].f64(), d["mask"].f64(), d["scale"], causal_q_len=q_len)
    got = host64(y)
    assert_close("long-row causal", got, ref, *TOL["f32"])
    masked = oracle.causal_mask(rows, cols, q_len)
    assert np.all(got[masked] == 0.0) and not np.any(np.signbit(got[masked]))


@pytest.mark.parametrize("cols", [30000, 50000, 70000, 30001])
def test_softmax_long_rows_fully_masked_and_single_live(cols):
    x = torch.randn(3, cols, device="cuda")
    m = torch.full((3, cols), float("-inf"), device="cuda")
    m[1, cols - 1] = 0.0                         # only the last element is live
    m[2, 0] = 0.0                                # only the first
    announce("softmax long rows masked", cols)
    y = host64(fs.row_softmax(x, m, 1.0))
    assert np.all(y[0] == 0.0) and not np.any(np.signbit(y[0]))
    want1 = np.zeros(cols)
    want1[-1] = 1.0
    want2 = np.zeros(cols)
    want2[0] = 1.0
    np.testing.assert_array_equal(y[1], want1)
    np.testing.assert_array_equal(y[2], want2)


@pytest.mark.parametrize("cols,ld", [(33333, 33400), (40000, 40016), (70000, 70064)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_softmax_long_rows_strided_in_place(dtype, cols, ld):
    # offset 0 with 16-byte rows takes the row cache with 16-byte slots,
    # offset 1 (rows not on a 16-byte boundary) its element-wise slots
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rows = 4
    d = fd.softmax_inputs(41, rows, cols, dtype, mask_dtype=dtype)
    ref = oracle.row_softmax(d["x"].f64(), d["mask"].f64(), d["scale"])
    for offset in (0, 1):
        announce("softmax long rows guard", dtype, cols, offset)
        xg = Guarded(rows, cols, ld, tdt, offset=offset)
        xg.view.copy_(dev(d["x"]))
        mg = Guarded(rows, cols, ld + 8, tdt, offset=offset)
        mg.view.copy_(dev(d["mask"]))
        fs.row_softmax(xg.view, mg.view, d["scale"], out=xg.view)
        torch.cuda.synchronize()
        assert_close(f"row cache in place offset {offset}", host64(xg.view), ref, *TOL[dtype])
        xg.check_untouched("softmax y")
        mg.check_untouched("softmax mask")


@pytest.mark.parametrize("dtype,mask_dtype", [("bf16", "bf16"), ("bf16", None), ("f32", "f32")])
@pytest.mark.parametrize("cols", [8193, 12001, 24999, 32001, 65537])
def test_softmax_rows_sharing_a_16_byte_phase(dtype, mask_dtype, cols):
    # contiguous rows of a width that is not a whole number of 16-byte
    # vectors start at varying offsets, the same for x, mask and y: the row
    # cache loads each row's aligned body 16 bytes at a time and its head
    # and tail elements one at a time
    rows = 7
    d = fd.softmax_inputs(cols + 11, rows, cols, dtype, mask_dtype=mask_dtype)
    announce("softmax shared phase", cols, dtype, mask_dtype)
    m = d["mask"].f64() if mask_dtype else None
    ref = oracle.row_softmax(d["x"].f64(), m, d["scale"])
    got = host64(fs.row_softmax(dev(d["x"]), dev(d["mask"]), d["scale"]))
    assert_close(f"cols {cols}", got, ref, *TOL[dtype])
    if dtype == "bf16":
        bf16_ulp_close(f"cols {cols}", got, ref, ulps=1.0, atol=1e-9)
    x = dev(d["x"])                                       # in place
    fs.row_softmax(x, dev(d["mask"]), d["scale"], out=x)
    assert_close(f"cols {cols} in place", host64(x), ref, *TOL[dtype])


def test_softmax_rows_of_different_phases():
    # y at a row stride one element longer than x: the phases differ from row
    # to row, so the rows take element-wise loads; same result
    rows, cols = 5, 40001
    d = fd.softmax_inputs(5, rows, cols, "bf16", mask_dtype="bf16")
    ref = oracle.row_softmax(d["x"].f64(), d["mask"].f64(), d["scale"])
    yg = Guarded(rows, cols, cols + 1, torch.bfloat16)
    announce("softmax different phases")
    fs.row_softmax(dev(d["x"]), dev(d["mask"]), d["scale"], out=yg.view)
    torch.cuda.synchronize()
    assert_close("different phases", host64(yg.view), ref, *TOL["bf16"])
    yg.check_untouched("softmax y")


def test_softmax_at_maximum_width():
    cols = fs.FS_SOFTMAX_MAX_COLS
    d = fd.softmax_inputs(17, 1, cols, "bf16", mask_dtype=None)
    announce("softmax max width", cols)
    got = host64(fs.row_softmax(dev(d["x"]), None, d["scale"]))
    ref = oracle.row_softmax(d["x"].f64(), None, d["scale"])
    assert_close("max width", got, ref, *TOL["bf16"])
    bf16_ulp_close("max width", got, ref, ulps=1.0, atol=1e-12)


# ---- LayerNorm / RMSNorm -----------------------------------------------------
def check_ln(name, d, y, ro, dtype, rms=False):
    if rms:
        ref_y, _ = oracle.rmsnorm_residual(d["x"].f64(), d["residual"].f64(), d["gamma"].f64(),
                                           d["eps"])
    else:
        ref_y, _ = oracle.layernorm_residual(d["x"].f64(), d["residual"].f64(), d["gamma"].f64(),
                                             d["beta"].f64(), d["eps"])
    got = host64(y)
    assert_close(name + " y", got, ref_y, *TOL[dtype])
    if dtype == "bf16":
        bf16_ulp_close(name + " y", got, ref_y, ulps=1.0, atol=2e-5)
        want = oracle.residual_store_bf16(d["x"].f64(), d["residual"].f64())
    else:
        want = (d["x"].data + d["residual"].data).astype(np.float64)   # the fp32 sum
    np.testing.assert_array_equal(host64(ro), want, err_msg=name + " residual_out")


@pytest.mark.parametrize("rms", [False, True])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cols", LONG)
def test_norm_streamed_widths(rms, dtype, cols):
    d = fd.layernorm_inputs(cols + 3, 3, cols, dtype)
    announce("norm streamed", "rms" if rms else "ln", cols, dtype)
    if rms:
        y, ro = fs.rmsnorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]), d["eps"])
    else:
        y, ro = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]),
                                      dev(d["beta"]), d["eps"])
    check_ln(f"cols {cols}", d, y, ro, dtype, rms)


@pytest.mark.parametrize("cols", [70001, 70000, 50000])
def test_layernorm_streamed_statistics_properties(cols):
    # gamma = 1, beta = 0, rows with an offset mean: mean 0 and variance
    # var/(var+eps) after normalisation, whatever the chunking
    rng = np.random.default_rng(12)
    x = (rng.standard_normal((4, cols)) + np.array([[0.0], [3.0], [-5.0], [0.5]])).astype(np.float32)
    announce("layernorm streamed properties", cols)
    y, _ = fs.layernorm_residual(torch.from_numpy(x).cuda(), None, None, None, 0.25)
    y = host64(y)
    var = x.astype(np.float64).var(axis=1)
    np.testing.assert_allclose(y.mean(axis=1), 0.0, atol=2e-6)
    np.testing.assert_allclose(y.var(axis=1), var / (var + 0.25), rtol=1e-5)
    ref, _ = oracle.layernorm_residual(x.astype(np.float64), None, None, None, 0.25)
    assert_close("offset rows", y, ref, *TOL["f32"])


@pytest.mark.parametrize("cols", [40000, 90000])
def test_layernorm_streamed_constant_rows_give_beta(cols):
    x = torch.full((2, cols), -7.0, device="cuda")
    beta = torch.linspace(-1, 1, cols, device="cuda")
    gamma = torch.ones(cols, device="cuda")
    y, _ = fs.layernorm_residual(x, None, gamma, beta, 1e-5)
    assert_close("constant rows", host64(y), np.broadcast_to(host64(beta), (2, cols)), 1e-6, 0)


@pytest.mark.parametrize("cols", [50000, 70000])
@pytest.mark.parametrize("rms", [False, True])
def test_norm_streamed_in_place(rms, cols):
    d = fd.layernorm_inputs(7, 3, cols, "bf16")
    x, r = dev(d["x"]), dev(d["residual"])
    announce("norm streamed in place", rms, cols)
    if rms:
        fs.rmsnorm_residual(x, r, dev(d["gamma"]), d["eps"], out=x, residual_out=r)
    else:
        fs.layernorm_residual(x, r, dev(d["gamma"]), dev(d["beta"]), d["eps"], out=x,
                              residual_out=r)
    torch.cuda.synchronize()
    check_ln("in place", d, x, r, "bf16", rms)


@pytest.mark.parametrize("cols,ld", [(24999, 25100), (40000, 40064), (70000, 70032)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_norm_streamed_strided_guards(dtype, cols, ld):
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rows = 3
    d = fd.layernorm_inputs(19, rows, cols, dtype)
    for offset in (0, 1):
        announce("norm streamed guard", dtype, cols, offset)
        xg = Guarded(rows, cols, ld, tdt, offset=offset)
        xg.view.copy_(dev(d["x"]))
        yg = Guarded(rows, cols, ld + 16, tdt, offset=offset)
        og = Guarded(rows, cols, ld + 32, tdt, offset=offset)
        fs.layernorm_residual(xg.view, dev(d["residual"]), dev(d["gamma"]), dev(d["beta"]),
                              d["eps"], out=yg.view, residual_out=og.view)
        torch.cuda.synchronize()
        check_ln(f"strided offset {offset}", d, yg.view, og.view, dtype)
        yg.check_untouched("layernorm y")
        og.check_untouched("layernorm residual_out")


@pytest.mark.parametrize("cols", [30000, 50000, 70000])
def test_norm_optional_operands_streamed(cols):
    d = fd.layernorm_inputs(23, 2, cols, "bf16")
    announce("norm streamed optional", cols)
    y, ro = fs.layernorm_residual(dev(d["x"]), None, None, None, d["eps"])
    assert ro is None
    ref, _ = oracle.layernorm_residual(d["x"].f64(), None, None, None, d["eps"])
    assert_close("plain ln", host64(y), ref, *TOL["bf16"])
    y, ro = fs.rmsnorm_residual(dev(d["x"]), None, None, d["eps"])
    ref, _ = oracle.rmsnorm_residual(d["x"].f64(), None, None, d["eps"])
    assert_close("plain rms", host64(y), ref, *TOL["bf16"])


def test_norm_at_maximum_width():
    cols = fs.FS_LAYERNORM_MAX_COLS
    d = fd.layernorm_inputs(29, 1, cols, "bf16")
    announce("norm max width", cols)
    y, ro = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]),
                                  dev(d["beta"]), d["eps"])
    check_ln("max width", d, y, ro, "bf16")


# ---- grids that loop: more rows than the row caches launch blocks -------------
def _cus():
    return torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count


# one 16-wave block per compute unit: 2 * cus + 3 rows give every block two or
# three rows, so the next row's prefetch, the carried causal position and the
# last block's partial trip all run; 40000 / 70000 take 16-byte slots (without
# and with a streamed tail), 40001 / 70001 element-wise slots, 50257 bf16 with
# a bf16 mask the 16-byte slots over each row's aligned body; q_len 37 does
# not divide the grid, so the causal position advances unevenly between trips
@pytest.mark.parametrize("dtype,mask_dtype,cols,q_len", [
    ("bf16", "bf16", 40000, 0), ("f32", "f32", 40001, 0), ("bf16", None, 70000, 0),
    ("f32", None, 70001, 0), ("bf16", "bf16", 50257, 0), ("f32", None, 40000, 37),
    ("bf16", "bf16", 70001, 37), ("bf16", "bf16", 50257, 37)])
def test_softmax_row_cache_loops_over_rows(dtype, mask_dtype, cols, q_len):
    rows = 2 * _cus() + 3
    d = fd.softmax_inputs(cols + q_len, rows, cols, dtype, mask_dtype=mask_dtype, p_masked=0.2)
    announce("softmax row cache looping", rows, cols, dtype, mask_dtype, q_len)
    y = fs.row_softmax(dev(d["x"]), dev(d["mask"]), d["scale"], causal_q_len=q_len)
    m = d["mask"].f64() if mask_dtype else None
    ref = oracle.row_softmax(d["x"].f64(), m, d["scale"], causal_q_len=q_len)
    got = host64(y)
    assert_close(f"looping cols {cols}", got, ref, *TOL[dtype])
    if dtype == "bf16":
        bf16_ulp_close(f"looping cols {cols}", got, ref, ulps=1.0, atol=1e-9)
    if q_len:
        masked = oracle.causal_mask(rows, cols, q_len)
        assert np.all(got[masked] == 0.0) and not np.any(np.signbit(got[masked]))


# LayerNorm's row cache: 40000 its 16-per-lane register part, 60000 the full
# cache, 70000 a streamed tail, 40001 element-wise slots
@pytest.mark.parametrize("rms", [False, True])
@pytest.mark.parametrize("dtype,cols", [("bf16", 40000), ("f32", 60000), ("bf16", 70000),
                                        ("f32", 40001)])
def test_norm_row_cache_loops_over_rows(rms, dtype, cols):
    rows = 2 * _cus() + 3
    d = fd.layernorm_inputs(cols + 9, rows, cols, dtype)
    announce("norm row cache looping", "rms" if rms else "ln", rows, cols, dtype)
    if rms:
        y, ro = fs.rmsnorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]), d["eps"])
    else:
        y, ro = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]),
                                      dev(d["beta"]), d["eps"])
    check_ln(f"looping cols {cols}", d, y, ro, dtype, rms)
