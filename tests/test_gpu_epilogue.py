"""GPU parity of fs_gemm_epilogue_reduce (and of the hipBLASLt GEMM that
feeds it) against the float64 oracle."""
import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
import paper_2609_30059_amd as fs
from gpu_util import SEEDS, TOL, announce, assert_close, dev, host64

pytestmark = pytest.mark.gpu

# fp32 tree sum of 8192 terms below 1: |error| <= log2(8192) * ulp(4096) ~ 5e-3
SUM_ATOL = 5e-3


@pytest.mark.parametrize("seed", SEEDS)
def test_epilogue_only_five_seeds(seed):
    d = fd.epilogue_inputs(seed, 128, 8192)
    announce("epilogue 8192 columns", seed)
    o = fs.gemm_epilogue_reduce(dev(d["c"]), dev(d["bias"]), dev(d["col_scale"]), "sigmoid", "sum")
    ref = oracle.gemm_epilogue_reduce(d["c"].f64(), d["bias"].f64(), d["col_scale"].f64(),
                                      "sigmoid", "sum")
    got = host64(o)
    assert_close(f"seed {seed}", got, ref, *TOL["bf16"])
    # the contract tolerance (~82 at 4096) cannot see a kernel that ignores C
    assert_close(f"seed {seed} supplementary", got, ref, SUM_ATOL, 0.0)


def test_zero_input_is_exactly_half_count():
    cm = torch.zeros(5, 8192, dtype=torch.bfloat16, device="cuda")
    o = fs.gemm_epilogue_reduce(cm, torch.zeros(8192, dtype=torch.bfloat16, device="cuda"),
                                torch.ones(8192, device="cuda"), "sigmoid", "sum")
    np.testing.assert_array_equal(host64(o), 4096.0)


def test_sign_flip_symmetry():
    d = fd.epilogue_inputs(7, 16, 8192)
    c, b, s = dev(d["c"]), dev(d["bias"]), dev(d["col_scale"])
    o1 = host64(fs.gemm_epilogue_reduce(c, b, s))
    o2 = host64(fs.gemm_epilogue_reduce(-c, -b, s))
    np.testing.assert_allclose(o1 + o2, 8192.0, atol=2 * SUM_ATOL)


def _saturating_c(cols, torch_dtype):
    """C whose sigmoid arguments reach far past the fp32 range of 2^u:
    row 0 all -300 (every term about 0), row 1 all +300 (every term 1),
    row 2 alternating, row 3 uniform in [-120, 120], the other rows N(0, 1)
    with one entry in ten replaced by +-U(40, 200)."""
    g = torch.Generator().manual_seed(11)
    rows = 24
    c = torch.randn(rows, cols, generator=g, dtype=torch.float64)
    c[0] = -300.0
    c[1] = 300.0
    c[2] = 300.0 * (1 - 2 * (torch.arange(cols) % 2))
    c[3] = torch.rand(cols, generator=g, dtype=torch.float64) * 240 - 120
    big = torch.rand(rows - 4, cols, generator=g) < 0.1
    mag = (torch.rand(rows - 4, cols, generator=g, dtype=torch.float64) * 160 + 40) * \
        torch.where(torch.rand(rows - 4, cols, generator=g) < 0.5, -1.0, 1.0).double()
    c[4:] = torch.where(big, mag, c[4:])
    return c.to(torch_dtype)


@pytest.mark.parametrize("c_dtype", ["bf16", "f32"])
# 4096: rows fill every lane's 16-byte slots; 4000: the last lanes' slots are masked
@pytest.mark.parametrize("cols", [4096, 4000])
def test_sigmoid_saturated_arguments(c_dtype, cols):
    """Arguments whose 2^u overflows fp32 (and every size in between): the
    four-term sum caps u at 31, which moves a term by less than 4.7e-10."""
    tdt = torch.bfloat16 if c_dtype == "bf16" else torch.float32
    c = _saturating_c(cols, tdt)
    g = torch.Generator().manual_seed(12)
    bias = (torch.rand(cols, generator=g) - 0.5).to(tdt)
    scale = torch.rand(cols, generator=g) + 0.5
    announce("epilogue saturated sigmoid", c_dtype, cols)
    got = host64(fs.gemm_epilogue_reduce(c.cuda(), bias.cuda(), scale.cuda(), "sigmoid", "sum"))
    with np.errstate(over="ignore"):
        ref = oracle.gemm_epilogue_reduce(c.double().numpy(), bias.double().numpy(),
                                          scale.double().numpy(), "sigmoid", "sum")
    assert np.isfinite(got).all()
    assert_close(f"saturated {c_dtype}", got, ref, SUM_ATOL * cols / 8192, 1e-6)
    assert 0.0 <= got[0] <= cols * 5e-10
    assert got[1] == cols


@pytest.mark.parametrize("c_dtype", ["bf16", "f32"])
def test_nan_and_infinities_in_c(c_dtype):
    """A NaN in C gives its row NaN and no other; +-inf give terms 1 and 0."""
    cols = 8192
    d = fd.epilogue_inputs(13, 9, cols, c_dtype)
    c = dev(d["c"])
    c[3, 17] = float("nan")
    c[5, 4000] = float("inf")
    c[6, 5] = float("-inf")
    c[7, 8191] = float("nan")
    announce("epilogue NaN and inf in C", c_dtype)
    got = host64(fs.gemm_epilogue_reduce(c, dev(d["bias"]), dev(d["col_scale"]), "sigmoid", "sum"))
    with np.errstate(over="ignore", invalid="ignore"):
        ref = oracle.gemm_epilogue_reduce(host64(c), d["bias"].f64(), d["col_scale"].f64(),
                                          "sigmoid", "sum")
    nan_rows = [3, 7]
    assert np.isnan(got[nan_rows]).all() and np.isnan(ref[nan_rows]).all()
    keep = [i for i in range(9) if i not in nan_rows]
    assert_close(f"{c_dtype} finite rows", got[keep], ref[keep], SUM_ATOL, 0.0)


@pytest.mark.parametrize("c_dtype,b_dtype", [("bf16", "bf16"), ("f32", "f32"), ("bf16", "f32"),
                                             ("f32", "bf16")])
# staged rungs up to 16384 columns; rows that are not whole vectors, from two
# vectors up (15, 17, 100, 1001, 4095, 16383, 16391: every rung, its edges and
# each row at another offset within a 16-byte unit); 512 (fp32) and 1024
# (bf16) fill the 2-vector rung exactly; the wide kernel with
# 16-byte loads (24000, 40000) and with element loads (1, 7, 16399, 24001)
@pytest.mark.parametrize("cols", [1, 7, 8, 15, 17, 100, 512, 1000, 1001, 1024, 4095, 4096, 8192,
                                  8200, 16383, 16384, 16391, 16399, 24000, 24001, 40000])
def test_widths_and_dtypes(c_dtype, b_dtype, cols):
    rows = 11 if cols <= 16384 else 3
    d = fd.epilogue_inputs(cols, rows, cols, c_dtype, bias_dtype=b_dtype)
    announce("epilogue width", cols, c_dtype, b_dtype)
    o = fs.gemm_epilogue_reduce(dev(d["c"]), dev(d["bias"]), dev(d["col_scale"]))
    ref = oracle.gemm_epilogue_reduce(d["c"].f64(), d["bias"].f64(), d["col_scale"].f64(),
                                      "sigmoid", "sum")
    tol = max(SUM_ATOL * cols / 8192, 1e-5)
    assert_close(f"cols {cols}", host64(o), ref, tol, 1e-6)


@pytest.mark.parametrize("act", ["none", "relu", "gelu_erf", "sigmoid"])
@pytest.mark.parametrize("reduce", ["sum", "mean"])
@pytest.mark.parametrize("with_bias,with_scale", [(True, True), (False, True), (True, False),
                                                  (False, False)])
def test_acts_reductions_optionals(act, reduce, with_bias, with_scale):
    d = fd.epilogue_inputs(3, 9, 2048, "f32", c_std=1.0, bias_dtype="f32")
    announce("epilogue options", act, reduce, with_bias, with_scale)
    o = fs.gemm_epilogue_reduce(dev(d["c"]), dev(d["bias"]) if with_bias else None,
                                dev(d["col_scale"]) if with_scale else None, act, reduce)
    ref = oracle.gemm_epilogue_reduce(d["c"].f64(), d["bias"].f64() if with_bias else None,
                                      d["col_scale"].f64() if with_scale else None, act, reduce)
    assert_close(f"{act} {reduce}", host64(o), ref, 2e-3 if reduce == "sum" else 1e-6, 1e-5)


@pytest.mark.parametrize("cols", [24000, 24001])
@pytest.mark.parametrize("act,reduce,with_bias,with_scale", [
    ("sigmoid", "sum", True, True), ("gelu_erf", "mean", False, True),
    ("relu", "sum", True, False), ("none", "mean", False, False)])
def test_wide_rows_options(cols, act, reduce, with_bias, with_scale):
    d = fd.epilogue_inputs(cols + 1, 5, cols, "bf16", c_std=1.0, bias_dtype="f32")
    announce("epilogue wide options", cols, act, reduce, with_bias, with_scale)
    o = fs.gemm_epilogue_reduce(dev(d["c"]), dev(d["bias"]) if with_bias else None,
                                dev(d["col_scale"]) if with_scale else None, act, reduce)
    ref = oracle.gemm_epilogue_reduce(d["c"].f64(), d["bias"].f64() if with_bias else None,
                                      d["col_scale"].f64() if with_scale else None, act, reduce)
    assert_close(f"{act} {reduce}", host64(o), ref, 2e-2 if reduce == "sum" else 1e-6, 1e-5)


@pytest.mark.parametrize("c_dtype,cols", [("bf16", 2051), ("f32", 2051), ("bf16", 9001)])
@pytest.mark.parametrize("act,reduce,with_bias,with_scale", [
    ("sigmoid", "sum", True, True), ("gelu_erf", "mean", False, True),
    ("relu", "sum", True, False), ("none", "mean", False, False)])
def test_odd_rows_options(c_dtype, cols, act, reduce, with_bias, with_scale):
    # rows of an odd width start at every offset within a 16-byte unit
    d = fd.epilogue_inputs(cols + 2, 13, cols, c_dtype, c_std=1.0, bias_dtype="bf16")
    announce("epilogue odd rows options", c_dtype, cols, act, reduce, with_bias, with_scale)
    o = fs.gemm_epilogue_reduce(dev(d["c"]), dev(d["bias"]) if with_bias else None,
                                dev(d["col_scale"]) if with_scale else None, act, reduce)
    ref = oracle.gemm_epilogue_reduce(d["c"].f64(), d["bias"].f64() if with_bias else None,
                                      d["col_scale"].f64() if with_scale else None, act, reduce)
    assert_close(f"{act} {reduce}", host64(o), ref, 1e-2 if reduce == "sum" else 1e-6, 1e-5)


def test_odd_rows_head_and_tail_columns():
    # one large value in the first or the last columns of each row: the head
    # and tail elements, read one per lane, must each count once
    rows, cols = 16, 4099
    c = torch.zeros(rows, cols, dtype=torch.bfloat16, device="cuda")
    for i, j in enumerate([0, 1, 6, 7, cols - 1, cols - 2, cols - 7, cols - 8]):
        c[2 * i, j] = 64.0
        c[2 * i + 1, j] = -64.0
    b = torch.zeros(cols, dtype=torch.float32, device="cuda")
    s = torch.ones(cols, dtype=torch.float32, device="cuda")
    announce("epilogue odd rows head and tail")
    got = host64(fs.gemm_epilogue_reduce(c, b, s, "relu", "sum"))
    np.testing.assert_array_equal(got, np.tile([64.0, 0.0], rows // 2))
    got = host64(fs.gemm_epilogue_reduce(c, b, s, "none", "sum"))
    np.testing.assert_array_equal(got, np.tile([64.0, -64.0], rows // 2))


def test_wide_rows_misaligned_coefficients():
    # bias and column scale one element off a 16-byte boundary: element loads
    # of the coefficients next to 16-byte loads of C
    cols = 24000
    d = fd.epilogue_inputs(8, 4, cols, "bf16", bias_dtype="bf16")
    bb = torch.empty(cols + 1, dtype=torch.bfloat16, device="cuda")
    sb = torch.empty(cols + 1, dtype=torch.float32, device="cuda")
    b, s = bb[1:], sb[1:]
    b.copy_(dev(d["bias"]))
    s.copy_(dev(d["col_scale"]))
    announce("epilogue misaligned coefficients")
    o = fs.gemm_epilogue_reduce(dev(d["c"]), b, s)
    ref = oracle.gemm_epilogue_reduce(d["c"].f64(), d["bias"].f64(), d["col_scale"].f64(),
                                      "sigmoid", "sum")
    assert_close("misaligned coefficients", host64(o), ref, SUM_ATOL * 3, 1e-6)


def test_strided_and_misaligned_c():
    d = fd.epilogue_inputs(4, 17, 3000, "bf16")
    base = torch.empty(17 * 3072 + 8, dtype=torch.bfloat16, device="cuda")
    for offset in (0, 1, 3):
        announce("epilogue strided", offset)
        view = base[offset:offset + 17 * 3072].view(17, 3072)[:, :3000]
        view.copy_(dev(d["c"]))
        o = fs.gemm_epilogue_reduce(view, dev(d["bias"]), dev(d["col_scale"]))
        ref = oracle.gemm_epilogue_reduce(d["c"].f64(), d["bias"].f64(), d["col_scale"].f64(),
                                          "sigmoid", "sum")
        assert_close(f"strided offset {offset}", host64(o), ref, SUM_ATOL, 0)


def test_zero_columns_sum_writes_zeros():
    out = torch.full((6,), 7.0, device="cuda")
    fs.gemm_epilogue_reduce(torch.empty(6, 0, dtype=torch.bfloat16, device="cuda"), out=out)
    np.testing.assert_array_equal(host64(out), 0.0)


@pytest.mark.slow
def test_beyond_2_31_elements():
    rows, cols = (1 << 18) + 3, 8192
    d = fd.epilogue_inputs(12, 64, cols)
    announce("epilogue > 2^31 elements", rows, cols)
    c = dev(d["c"]).repeat((rows + 63) // 64, 1)[:rows]
    o = fs.gemm_epilogue_reduce(c, dev(d["bias"]), dev(d["col_scale"]))
    idx = np.array([0, 1, 64, rows // 2, rows - 1])
    ref = oracle.gemm_epilogue_reduce(d["c"].rows(idx % 64).f64(), d["bias"].f64(),
                                      d["col_scale"].f64(), "sigmoid", "sum")
    assert_close("beyond 2^31", host64(o[torch.from_numpy(idx).cuda()]), ref, SUM_ATOL, 0)


# more rows than the staged kernels hold waves (two 16-wave blocks per compute
# unit): every wave reduces two or three rows, so the chunk pipeline carries
# from one row into the next (the next row's first chunk, the rotated chunk
# order, the last row's prefetch); 8192 bf16 and 4096 bf16 fill every slot
# (the variant without clamps), 1000 fp32 leaves slots empty, 1001 and 4095
# are rows that are not whole vectors (each row at another 16-byte phase)
@pytest.mark.parametrize("c_dtype,cols", [("bf16", 8192), ("bf16", 4096), ("f32", 1000),
                                          ("bf16", 1001), ("f32", 1001), ("bf16", 4095)])
def test_rows_beyond_the_resident_waves(c_dtype, cols):
    cus = torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count
    rows = 2 * (cus * 2 * 16) + 3
    d = fd.epilogue_inputs(cols + 13, rows, cols, c_dtype, bias_dtype=c_dtype)
    announce("epilogue looping rows", rows, cols, c_dtype)
    o = fs.gemm_epilogue_reduce(dev(d["c"]), dev(d["bias"]), dev(d["col_scale"]))
    ref = np.concatenate([
        oracle.gemm_epilogue_reduce(d["c"].rows(slice(r0, r0 + 2048)).f64(), d["bias"].f64(),
                                    d["col_scale"].f64(), "sigmoid", "sum")
        for r0 in range(0, rows, 2048)])
    tol = max(SUM_ATOL * cols / 8192, 1e-5)
    assert_close(f"looping rows {cols}", host64(o), ref, tol, 1e-6)


# max and log-sum-exp: the max is one of the fp32 values act((c + b) * s), so
# it is within the fp32 rounding of that expression (a few units of 2^-24,
# more through an activation's own error); log-sum-exp adds the relative
# error of a sum of fp32 exponentials to it (see the row reduction tests)
MAXLSE_ATOL, MAXLSE_RTOL = 2e-5, 2e-5


@pytest.mark.parametrize("seed", SEEDS)
@pytest.mark.parametrize("reduce", ["max", "logsumexp"])
def test_max_and_logsumexp_reductions_five_seeds(seed, reduce):
    d = fd.epilogue_inputs(seed, 128, 8192)
    announce("epilogue", reduce, seed)
    for act in ("none", "sigmoid", "gelu_erf", "relu"):
        o = fs.gemm_epilogue_reduce(dev(d["c"]), dev(d["bias"]), dev(d["col_scale"]), act, reduce)
        ref = oracle.gemm_epilogue_reduce(d["c"].f64(), d["bias"].f64(), d["col_scale"].f64(),
                                          act, reduce)
        assert_close(f"{reduce} {act} seed {seed}", host64(o), ref, MAXLSE_ATOL, MAXLSE_RTOL)


@pytest.mark.parametrize("reduce", ["max", "logsumexp"])
@pytest.mark.parametrize("c_dtype,b_dtype", [("bf16", "bf16"), ("f32", "f32"), ("bf16", "f32"),
                                             ("f32", "bf16")])
# the vector path, odd widths (element-wise), one column, long rows
@pytest.mark.parametrize("cols", [1, 7, 1000, 1003, 8192, 40000])
def test_max_and_logsumexp_widths_and_dtypes(reduce, c_dtype, b_dtype, cols):
    rows = 600 if cols <= 1003 else 40     # 600 rows: blocks loop over rows
    d = fd.epilogue_inputs(cols, rows, cols, c_dtype, c_std=2.0, bias_dtype=b_dtype)
    announce("epilogue width", reduce, c_dtype, b_dtype, cols)
    o = fs.gemm_epilogue_reduce(dev(d["c"]), dev(d["bias"]), dev(d["col_scale"]), "none", reduce)
    ref = oracle.gemm_epilogue_reduce(d["c"].f64(), d["bias"].f64(), d["col_scale"].f64(),
                                      "none", reduce)
    assert_close(f"{reduce} {c_dtype}/{b_dtype} {cols}", host64(o), ref, MAXLSE_ATOL, MAXLSE_RTOL)


def test_max_and_logsumexp_special_values():
    c = torch.zeros(6, 4096, device="cuda")
    c[0] = -float("inf")                     # a row of -inf
    c[1, 9] = float("inf")
    c[2, 100] = float("nan")
    c[3, :] = 50.0                           # all equal: max 50, LSE 50 + log 4096
    c[4, 17] = 1e30                          # one huge entry
    c[5, ::2] = -float("inf")                # half masked
    for reduce in ("max", "logsumexp"):
        o = host64(fs.gemm_epilogue_reduce(c, None, None, "none", reduce))
        ref = oracle.gemm_epilogue_reduce(host64(c), None, None, "none", reduce)
        assert o[0] == -np.inf and o[1] == np.inf and np.isnan(o[2]), (reduce, o[:3])
        assert_close(f"{reduce} finite rows", o[3:], ref[3:], MAXLSE_ATOL, MAXLSE_RTOL)
