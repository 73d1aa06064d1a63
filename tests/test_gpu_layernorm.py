"""GPU parity of fs_layernorm_residual against the float64 oracle."""
import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
import paper_2609_30059_amd as fs
from gpu_util import (SEEDS, TOL, Guarded, announce, assert_close, bf16_ulp_close, dev, host64)

pytestmark = pytest.mark.gpu


def check(name, d, y, ro, dtype, has_res=True, affine=True):
    g = d["gamma"].f64() if affine else None
    b = d["beta"].f64() if affine else None
    r = d["residual"].f64() if has_res else None
    ref_y, _ = oracle.layernorm_residual(d["x"].f64(), r, g, b, d["eps"])
    got = host64(y)
    assert_close(name + " y", got, ref_y, *TOL[dtype])
    if dtype == "bf16":
        # fp32 statistics keep y within one bf16 rounding of exact (+ fp32 noise)
        bf16_ulp_close(name + " y", got, ref_y, ulps=1.0, atol=2e-5)
    if ro is not None:
        if dtype == "bf16":
            want = oracle.residual_store_bf16(d["x"].f64(), d["residual"].f64())
            np.testing.assert_array_equal(host64(ro), want, err_msg=name + " residual_out")
        else:
            want = d["x"].data + d["residual"].data        # the fp32 sum
            np.testing.assert_array_equal(host64(ro), want.astype(np.float64))


@pytest.mark.parametrize("seed", SEEDS)
def test_4096_column_rows_five_seeds(seed):
    d = fd.layernorm_inputs(seed, 80, 4096)
    announce("layernorm 4096 columns", seed)
    y, ro = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]),
                                  dev(d["beta"]), d["eps"])
    check(f"seed {seed}", d, y, ro, "bf16")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
# odd widths take the element-wise path: 4099 and 6001 the 2- and 4-wave
# register rungs, 8195 and 12347 the streamed kernel
@pytest.mark.parametrize("cols", [1, 2, 7, 64, 100, 1024, 4096, 4099, 6001, 8192, 8195, 12347,
                                  20000, 65536])
def test_widths(dtype, cols):
    rows = 9 if cols <= 8192 else 3
    d = fd.layernorm_inputs(cols, rows, cols, dtype)
    announce("layernorm width", cols, dtype)
    y, ro = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]),
                                  dev(d["beta"]), d["eps"])
    check(f"cols {cols}", d, y, ro, dtype)


# rows that are not whole 16-byte vectors, with x, residual, y and
# residual_out at one offset within a 16-byte unit per row (contiguous rows: a
# different one each row): the register rungs with gamma and beta staged in
# LDS, across the rungs and their edges
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cols", [17, 100, 1001, 2047, 4097, 8191, 12289, 16383])
def test_odd_rows_sharing_a_phase(dtype, cols):
    rows = 37 if cols <= 4097 else 7
    d = fd.layernorm_inputs(cols + 5, rows, cols, dtype)
    announce("layernorm odd rows", cols, dtype)
    y, ro = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]),
                                  dev(d["beta"]), d["eps"])
    check(f"odd rows {cols}", d, y, ro, dtype)


@pytest.mark.parametrize("has_res,affine,store", [(False, True, False), (True, False, True),
                                                  (False, False, False)])
def test_optional_operands_odd_rows(has_res, affine, store):
    d = fd.layernorm_inputs(6, 29, 3001, "bf16")
    announce("layernorm optional odd rows", has_res, affine, store)
    y, ro = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]) if has_res else None,
                                  dev(d["gamma"]) if affine else None,
                                  dev(d["beta"]) if affine else None, d["eps"],
                                  store_residual=store)
    check("optional odd rows", d, y, ro, "bf16", has_res, affine)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_misaligned_gamma_beta(dtype):
    # whole-vector rows with gamma and beta one element off a 16-byte boundary
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    cols = 4096
    d = fd.layernorm_inputs(14, 11, cols, dtype)
    gb = torch.empty(2 * cols + 2, dtype=tdt, device="cuda")
    g, b = gb[1:cols + 1], gb[cols + 2:]
    g.copy_(dev(d["gamma"]))
    b.copy_(dev(d["beta"]))
    announce("layernorm misaligned gamma beta", dtype)
    y, ro = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]), g, b, d["eps"])
    check("misaligned gamma beta", d, y, ro, dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_strided_same_phase_rows_and_guards(dtype):
    # x, residual, y and residual_out share one odd row stride and offset
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rows, cols, ld = 17, 2501, 2519
    d = fd.layernorm_inputs(15, rows, cols, dtype)
    for offset in (1, 5):
        announce("layernorm same-phase strided", dtype, offset)
        xg = Guarded(rows, cols, ld, tdt, offset=offset)
        rg = Guarded(rows, cols, ld, tdt, offset=offset)
        yg = Guarded(rows, cols, ld, tdt, offset=offset)
        og = Guarded(rows, cols, ld, tdt, offset=offset)
        xg.view.copy_(dev(d["x"]))
        rg.view.copy_(dev(d["residual"]))
        fs.layernorm_residual(xg.view, rg.view, dev(d["gamma"]), dev(d["beta"]), d["eps"],
                              out=yg.view, residual_out=og.view)
        torch.cuda.synchronize()
        check(f"same-phase offset {offset}", d, yg.view, og.view, dtype)
        yg.check_untouched("layernorm y")
        og.check_untouched("layernorm residual_out")


def test_in_place_odd_rows():
    d = fd.layernorm_inputs(16, 23, 4093, "bf16")
    x, r = dev(d["x"]), dev(d["residual"])
    fs.layernorm_residual(x, r, dev(d["gamma"]), dev(d["beta"]), d["eps"], out=x,
                          residual_out=r)
    torch.cuda.synchronize()
    check("in place odd rows", d, x, r, "bf16")


@pytest.mark.parametrize("has_res,affine,store", [(False, True, False), (True, False, True),
                                                  (True, True, False), (False, False, False)])
def test_optional_operands(has_res, affine, store):
    d = fd.layernorm_inputs(3, 33, 1024, "bf16")
    announce("layernorm optional", has_res, affine, store)
    y, ro = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]) if has_res else None,
                                  dev(d["gamma"]) if affine else None,
                                  dev(d["beta"]) if affine else None, d["eps"],
                                  store_residual=store)
    assert (ro is None) == (not (has_res and store))
    check("optional", d, y, ro, "bf16", has_res, affine)


def test_statistics_properties_fp32():
    # gamma = 1, beta = 0: each row has mean 0 and variance var/(var+eps)
    d = fd.layernorm_inputs(9, 16, 4096, "f32")
    y, _ = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]), None, None, 0.25)
    y = host64(y)
    h = d["x"].f64() + d["residual"].f64()
    var = h.var(axis=1)
    np.testing.assert_allclose(y.mean(axis=1), 0.0, atol=1e-6)
    np.testing.assert_allclose(y.var(axis=1), var / (var + 0.25), rtol=1e-5)


def test_constant_rows_give_beta():
    x = torch.full((4, 1024), 3.0, device="cuda")
    beta = torch.linspace(-1, 1, 1024, device="cuda")
    gamma = torch.ones(1024, device="cuda")
    y, _ = fs.layernorm_residual(x, None, gamma, beta, 1e-5)
    assert_close("constant rows", host64(y), np.broadcast_to(host64(beta), (4, 1024)), 1e-6, 0)


def test_in_place_outputs():
    d = fd.layernorm_inputs(4, 40, 4096, "bf16")
    x, r = dev(d["x"]), dev(d["residual"])
    fs.layernorm_residual(x, r, dev(d["gamma"]), dev(d["beta"]), d["eps"], out=x,
                          residual_out=r)             # y == x, residual_out == residual
    torch.cuda.synchronize()
    check("in place", d, x, r, "bf16")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_strided_misaligned_and_guards(dtype):
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rows, cols, ld = 13, 1500, 1536
    d = fd.layernorm_inputs(13, rows, cols, dtype)
    for offset in (0, 1):
        announce("layernorm guard", dtype, offset)
        xg = Guarded(rows, cols, ld, tdt, offset=offset)
        xg.view.copy_(dev(d["x"]))
        yg = Guarded(rows, cols, ld + 16, tdt, offset=offset)
        og = Guarded(rows, cols, ld + 32, tdt, offset=offset)
        fs.layernorm_residual(xg.view, dev(d["residual"]), dev(d["gamma"]), dev(d["beta"]),
                              d["eps"], out=yg.view, residual_out=og.view)
        torch.cuda.synchronize()
        check(f"strided offset {offset}", d, yg.view, og.view, dtype)
        yg.check_untouched("layernorm y")
        og.check_untouched("layernorm residual_out")


@pytest.mark.slow
def test_beyond_2_31_elements():
    rows, cols = (1 << 19) + 9, 4096
    d = fd.layernorm_inputs(6, 64, cols, "bf16")
    announce("layernorm > 2^31 elements", rows, cols)
    rep = (rows + 63) // 64
    x = dev(d["x"]).repeat(rep, 1)[:rows]
    r = dev(d["residual"]).repeat(rep, 1)[:rows]
    y, ro = fs.layernorm_residual(x, r, dev(d["gamma"]), dev(d["beta"]), d["eps"])
    idx = np.array([0, 5, 64, rows // 3, rows - 1])
    ti = torch.from_numpy(idx).cuda()
    sub = {"x": d["x"].rows(idx % 64), "residual": d["residual"].rows(idx % 64),
           "gamma": d["gamma"], "beta": d["beta"], "eps": d["eps"]}
    check("beyond 2^31", sub, y[ti], ro[ti], "bf16")


# ---------------------------------------------------------------------------
# RMSNorm + residual (the same kernel family)
# ---------------------------------------------------------------------------
def check_rms(name, d, y, ro, dtype, has_res=True, affine=True, eps=1e-6):
    ref_y, _ = oracle.rmsnorm_residual(d["x"].f64(), d["residual"].f64() if has_res else None,
                                       d["gamma"].f64() if affine else None, eps)
    got = host64(y)
    assert_close(name + " y", got, ref_y, *TOL[dtype])
    if dtype == "bf16":
        bf16_ulp_close(name + " y", got, ref_y, ulps=1.0, atol=2e-5)
    if ro is not None and dtype == "bf16":
        np.testing.assert_array_equal(host64(ro), oracle.residual_store_bf16(
            d["x"].f64(), d["residual"].f64()), err_msg=name + " residual_out")


@pytest.mark.parametrize("seed", SEEDS)
def test_rmsnorm_five_seeds(seed):
    d = fd.layernorm_inputs(seed, 80, 4096)
    announce("rmsnorm", seed)
    eps = float(np.float32(1e-6))
    y, ro = fs.rmsnorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]), eps)
    check_rms(f"seed {seed}", d, y, ro, "bf16", eps=eps)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cols", [1, 7, 64, 1024, 4099, 6001, 8192, 8195, 20000])
def test_rmsnorm_widths(dtype, cols):
    d = fd.layernorm_inputs(cols + 1, 9 if cols <= 8192 else 3, cols, dtype)
    announce("rmsnorm width", cols, dtype)
    eps = float(np.float32(1e-6))
    y, ro = fs.rmsnorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]), eps)
    check_rms(f"cols {cols}", d, y, ro, dtype, eps=eps)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cols", [1001, 12289])
def test_rmsnorm_odd_rows(dtype, cols):
    d = fd.layernorm_inputs(cols + 2, 9, cols, dtype)
    announce("rmsnorm odd rows", cols, dtype)
    eps = float(np.float32(1e-6))
    y, ro = fs.rmsnorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]), eps)
    check_rms(f"odd rows {cols}", d, y, ro, dtype, eps=eps)


def test_rmsnorm_without_residual_or_gamma():
    d = fd.layernorm_inputs(5, 16, 1024, "bf16")
    eps = float(np.float32(1e-6))
    y, ro = fs.rmsnorm_residual(dev(d["x"]), None, None, eps)
    assert ro is None
    check_rms("plain", d, y, None, "bf16", has_res=False, affine=False, eps=eps)


# rows that fill one wave's 16-byte slots exactly (fp32 256 / 512 / 1024,
# bf16 512 / 1024 columns) with gamma and beta take the one-wave kernel:
# LayerNorm and RMSNorm, with and without a residual (stored or not); row
# counts that leave the last wave partly empty, and one large enough that the
# grid loops
@pytest.mark.parametrize("dtype,cols", [("f32", 256), ("f32", 512), ("f32", 1024),
                                        ("bf16", 512), ("bf16", 1024)])
@pytest.mark.parametrize("rms", [False, True])
@pytest.mark.parametrize("has_res,store", [(False, False), (True, True), (True, False)])
def test_one_wave_rows(dtype, cols, rms, has_res, store):
    rows = 4099
    d = fd.layernorm_inputs(cols + 31, rows, cols, dtype)
    announce("one-wave rows", dtype, cols, rms, has_res, store)
    r = dev(d["residual"]) if has_res else None
    if rms:
        y, ro = fs.rmsnorm_residual(dev(d["x"]), r, dev(d["gamma"]), d["eps"],
                                    store_residual=store)
        check_rms(f"rms {cols}", d, y, ro, dtype, has_res, eps=d["eps"])
    else:
        y, ro = fs.layernorm_residual(dev(d["x"]), r, dev(d["gamma"]), dev(d["beta"]), d["eps"],
                                      store_residual=store)
        check(f"ln {cols}", d, y, ro, dtype, has_res)
    assert (ro is None) == (not (has_res and store))


@pytest.mark.parametrize("dtype,cols,rows_per_wave", [("bf16", 512, 2), ("f32", 256, 4)])
def test_one_wave_rows_grid_loops(dtype, cols, rows_per_wave):
    # twice the rows that the capped grid (8 * 16 / 4 four-wave blocks per
    # compute unit) covers in one trip: every wave loops
    cus = torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count
    rows = 2 * (cus * 8 * 16 // 4) * 4 * rows_per_wave + 5
    d = fd.layernorm_inputs(cols + 41, rows, cols, dtype)
    announce("one-wave rows looping", dtype, cols, rows)
    y, ro = fs.layernorm_residual(dev(d["x"]), dev(d["residual"]), dev(d["gamma"]),
                                  dev(d["beta"]), d["eps"])
    check(f"looping {cols}", d, y, ro, dtype)


def test_one_wave_rows_in_place_and_strided():
    # y == x and residual_out == residual; then rows 16-byte aligned with a
    # row stride above the width, guard bands around every output
    d = fd.layernorm_inputs(77, 301, 1024, "bf16")
    x, r = dev(d["x"]), dev(d["residual"])
    announce("one-wave rows in place")
    fs.layernorm_residual(x, r, dev(d["gamma"]), dev(d["beta"]), d["eps"], out=x, residual_out=r)
    torch.cuda.synchronize()
    check("one-wave in place", d, x, r, "bf16")
    rows, cols, ld = 301, 1024, 1032
    xg = Guarded(rows, cols, ld, torch.bfloat16)
    xg.view.copy_(dev(d["x"]))
    yg = Guarded(rows, cols, ld + 8, torch.bfloat16)
    og = Guarded(rows, cols, ld + 16, torch.bfloat16)
    announce("one-wave rows strided")
    fs.layernorm_residual(xg.view, dev(d["residual"]), dev(d["gamma"]), dev(d["beta"]), d["eps"],
                          out=yg.view, residual_out=og.view)
    torch.cuda.synchronize()
    check("one-wave strided", d, yg.view, og.view, "bf16")
    yg.check_untouched("y")
    og.check_untouched("residual_out")
