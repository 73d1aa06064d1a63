"""GPU parity of fs_row_reduce (sum, mean, max) and fs_row_argmax against the
float64 oracle."""
import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
import paper_2609_30059_amd as fs
from gpu_util import SEEDS, Guarded, announce, assert_close, dev, host64

pytestmark = pytest.mark.gpu


def sum_tol(x64):
    # fp32 accumulation (sequential per lane, then a tree): a few fp32 units
    # of the sum of magnitudes
    return 1e-6 * np.abs(x64).sum(axis=1) + 1e-6


@pytest.mark.parametrize("seed", SEEDS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sum_mean_max_seeds(seed, dtype):
    x = fd.row_inputs(seed, 97, 4096, dtype, mean=0.25, std=2.0)
    t = dev(x)
    announce("row_reduce seeds", seed, dtype)
    x64 = x.f64()
    assert_close("sum", host64(fs.row_reduce(t, "sum")), oracle.row_reduce(x64, "sum"),
                 sum_tol(x64), 0)
    assert_close("mean", host64(fs.row_reduce(t, "mean")), oracle.row_reduce(x64, "mean"),
                 sum_tol(x64) / 4096, 0)
    np.testing.assert_array_equal(host64(fs.row_reduce(t, "max")), oracle.row_reduce(x64, "max"))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("rows,cols", [(5, 1), (9, 7), (33, 8), (17, 100), (8, 4099),
                                       (3, 65536 + 24), (2, (1 << 20) + 3)])
def test_widths(dtype, rows, cols):
    x = fd.row_inputs(cols, rows, cols, dtype)
    t = dev(x)
    announce("row_reduce width", rows, cols, dtype)
    x64 = x.f64()
    assert_close("sum", host64(fs.row_reduce(t, "sum")), oracle.row_reduce(x64, "sum"),
                 sum_tol(x64), 0)
    np.testing.assert_array_equal(host64(fs.row_reduce(t, "max")), oracle.row_reduce(x64, "max"))
    np.testing.assert_array_equal(fs.row_argmax(t).cpu().numpy(), oracle.row_argmax(x64))


@pytest.mark.parametrize("seed", SEEDS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cols", [64, 1000, 1001, 4096, 70000, 70001])
def test_argmax_bit_exact_with_ties(seed, dtype, cols):
    # small integers: every row is full of exact ties, so only the
    # lowest-index rule picks the right answer
    x = fd.integer_inputs(seed, 41, cols, dtype)
    announce("row_argmax ties", seed, dtype, cols)
    got = fs.row_argmax(dev(x)).cpu().numpy()
    np.testing.assert_array_equal(got, oracle.row_argmax(x.f64()))


def test_argmax_nan_inf_and_constant_rows():
    rows = np.zeros((6, 300), dtype=np.float32)
    rows[0, :] = 2.0                          # constant -> 0
    rows[1, 123] = np.nan                     # NaN wins
    rows[1, 200] = np.nan
    rows[1, 5] = 1e30
    rows[2, :] = -np.inf                      # all -inf -> 0
    rows[3, :] = -np.inf
    rows[3, 299] = -1.0                       # last element
    rows[4, 17] = np.inf                      # +inf
    rows[4, 250] = np.inf
    rows[5, :] = np.arange(300, dtype=np.float32)[::-1]   # first element
    t = torch.from_numpy(rows).cuda()
    got = fs.row_argmax(t).cpu().numpy()
    np.testing.assert_array_equal(got, oracle.row_argmax(rows.astype(np.float64)))
    np.testing.assert_array_equal(got, [0, 123, 0, 299, 17, 0])
    mx = host64(fs.row_reduce(t, "max"))
    assert np.isnan(mx[1]) and mx[2] == -np.inf and mx[4] == np.inf


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_head_and_tail_elements_of_odd_rows(dtype):
    # contiguous rows of 4099 columns start at every offset within a 16-byte
    # unit; their first and last few columns are loaded one at a time next
    # to the 16-byte body: put the maximum, NaNs and ties there
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rows, cols = 8, 4099
    x = np.zeros((rows, cols), dtype=np.float32)
    x[0, 0] = 5.0                                # first column (head)
    x[1, cols - 1] = 5.0                         # last column (tail)
    x[2, 1] = np.nan
    x[2, cols - 2] = np.nan                      # first NaN wins
    x[3, 2] = 7.0
    x[3, cols - 1] = 7.0                         # tie: head beats tail
    x[4, cols - 3] = 7.0
    x[4, 3000] = 7.0                             # tie: body beats tail
    x[5, 6] = -1.0
    x[5, :] = -2.0                               # constant row
    x[6, 3] = np.inf
    x[7, :] = np.arange(cols, dtype=np.float32)  # increasing: the last column
    t = torch.from_numpy(x).to(tdt).cuda()
    xr = t.float().cpu().numpy().astype(np.float64)
    announce("row_argmax head and tail", dtype)
    got = fs.row_argmax(t).cpu().numpy()
    np.testing.assert_array_equal(got, oracle.row_argmax(xr))
    np.testing.assert_array_equal(got[:5], [0, cols - 1, 1, 2, 3000])
    np.testing.assert_array_equal(host64(fs.row_reduce(t, "max")), oracle.row_reduce(xr, "max"))
    sums = host64(fs.row_reduce(t, "sum"))
    fin = [0, 1, 3, 4, 5, 7]
    assert_close("sum", sums[fin], oracle.row_reduce(xr[fin], "sum"), sum_tol(xr[fin]), 0)
    assert np.isnan(sums[2]) and sums[6] == np.inf


def test_zero_columns_sum_and_empty_rows():
    out = torch.full((4,), 3.0, device="cuda")
    fs.row_reduce(torch.empty(4, 0, device="cuda"), "sum", out=out)
    np.testing.assert_array_equal(host64(out), 0.0)
    assert fs.row_reduce(torch.empty(0, 9, device="cuda")).numel() == 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_strided_and_misaligned(dtype):
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rows, cols, ld = 13, 1500, 1536
    x = fd.integer_inputs(31, rows, cols, dtype, -50, 50)
    for offset in (0, 1):
        announce("row_reduce strided", dtype, offset)
        g = Guarded(rows, cols, ld, tdt, offset=offset)
        g.view.copy_(dev(x))
        np.testing.assert_array_equal(fs.row_argmax(g.view).cpu().numpy(), oracle.row_argmax(x.f64()))
        assert_close("sum", host64(fs.row_reduce(g.view, "sum")), oracle.row_reduce(x.f64(), "sum"),
                     sum_tol(x.f64()), 0)


# log-sum-exp: LSE = m + log S with S = sum_j exp(x_j - m) >= 1, so its
# absolute error is about the relative error of S -- fp32 terms from
# v_exp_f32 (a few units of 2^-24 each) summed in fp32, sequentially per lane
# and then in a tree -- plus the fp32 rounding of m + log S
LSE_ATOL, LSE_RTOL = 2e-5, 2e-6


@pytest.mark.parametrize("seed", SEEDS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_logsumexp_seeds(seed, dtype):
    x = fd.row_inputs(seed, 97, 4096, dtype, mean=0.25, std=2.0)
    announce("row_reduce logsumexp seeds", seed, dtype)
    got = host64(fs.row_reduce(dev(x), "logsumexp"))
    assert_close("logsumexp", got, oracle.row_reduce(x.f64(), "logsumexp"), LSE_ATOL, LSE_RTOL)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
# the vector path, the aligned body of odd rows, one element per lane, long rows
@pytest.mark.parametrize("rows,cols", [(5, 1), (5, 3), (9, 8), (33, 1000), (33, 1003), (7, 9001),
                                       (3, 70000), (2000, 64)])
def test_logsumexp_widths(dtype, rows, cols):
    x = fd.row_inputs(cols + rows, rows, cols, dtype, mean=-1.0, std=6.0)
    announce("row_reduce logsumexp width", rows, cols, dtype)
    got = host64(fs.row_reduce(dev(x), "logsumexp"))
    assert_close(f"logsumexp {rows}x{cols}", got, oracle.row_reduce(x.f64(), "logsumexp"),
                 LSE_ATOL, LSE_RTOL)


def test_logsumexp_special_rows():
    inf, nan = float("inf"), float("nan")
    x = torch.full((8, 1024), -3.0, device="cuda")
    x[0] = -inf                           # empty sum: -inf
    x[1, 500] = inf                       # +inf
    x[2, 7] = nan                         # NaN
    x[3, 100:200] = -inf                  # masked entries add nothing
    x[4] = 88.0                           # exp(88) near the fp32 limit: no overflow
    x[5, 0] = 1e30                        # one huge entry: the row is that entry
    x[6, :] = torch.arange(1024, device="cuda", dtype=torch.float32)   # rising maxima
    x[7, :] = -torch.arange(1024, device="cuda", dtype=torch.float32)  # falling
    got = host64(fs.row_reduce(x, "logsumexp"))
    ref = oracle.row_reduce(host64(x), "logsumexp")
    assert got[0] == -np.inf and got[1] == np.inf and np.isnan(got[2])
    assert_close("finite rows", got[3:], ref[3:], LSE_ATOL, LSE_RTOL)


def test_logsumexp_huge_magnitudes():
    # maxima far past the exponent range of exp2: the difference is taken
    # before the scaling, so the row's maximum contributes exactly 1
    x = torch.full((4, 2048), 0.0, device="cuda")
    x[0, 5] = 1e30
    x[1, :] = -1e30
    x[2, ::3] = 3e38
    x[3, :] = 2e9
    got = host64(fs.row_reduce(x, "logsumexp"))
    ref = oracle.row_reduce(host64(x), "logsumexp")
    assert_close("huge magnitudes", got, ref, LSE_ATOL, LSE_RTOL)
