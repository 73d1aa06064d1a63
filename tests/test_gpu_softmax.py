"""GPU parity of fs_row_softmax against the float64 oracle."""
import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
import paper_2609_30059_amd as fs
from gpu_util import (SEEDS, TOL, Guarded, announce, assert_close, bf16_ulp_close, dev, host64,
                      softmax_supplementary)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", SEEDS)
def test_4096_column_rows_five_seeds(seed):
    d = fd.softmax_inputs(seed, 96, 4096)
    announce("softmax 4096 columns", seed)
    y = fs.row_softmax(dev(d["x"]), dev(d["mask"]), d["scale"])
    got = host64(y)
    ref = oracle.row_softmax(d["x"].f64(), d["mask"].f64(), d["scale"])
    assert_close(f"seed {seed}", got, ref, *TOL["bf16"])
    softmax_supplementary(f"seed {seed}", got, ref, np.isinf(d["mask"].f64()))


@pytest.mark.parametrize("dtype,mask_dtype", [("f32", "f32"), ("f32", "bf16"), ("bf16", "bf16"),
                                              ("bf16", "f32"), ("bf16", None), ("f32", None)])
@pytest.mark.parametrize("cols", [1, 3, 8, 37, 511, 512, 513, 1000, 4095, 4096, 4104, 8192,
                                  16384 + 8, 65536])
def test_widths(dtype, mask_dtype, cols):
    rows = 7 if cols <= 16384 else 3
    d = fd.softmax_inputs(cols, rows, cols, dtype, mask_dtype=mask_dtype)
    announce("softmax width", cols, dtype, mask_dtype)
    y = fs.row_softmax(dev(d["x"]), dev(d["mask"]), d["scale"])
    got = host64(y)
    m = d["mask"].f64() if mask_dtype else None
    ref = oracle.row_softmax(d["x"].f64(), m, d["scale"])
    assert_close(f"cols {cols}", got, ref, *TOL[dtype])
    if dtype == "bf16":
        bf16_ulp_close(f"cols {cols}", got, ref, ulps=1.0, atol=1e-7)
    if m is not None:
        assert np.all(got[np.isinf(m)] == 0.0)


# rows that are not whole 16-byte vectors, with x, mask and y at one offset
# within a 16-byte unit per row (contiguous rows: a different one each row):
# every register rung's edges, one-wave rows batched several per trip
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("cols", [17, 63, 65, 1001, 2047, 4097, 8191, 12289, 16383])
def test_odd_rows_sharing_a_phase(dtype, cols):
    rows = 45 if cols <= 4097 else 9
    d = fd.softmax_inputs(cols + 3, rows, cols, dtype, mask_dtype=dtype, p_masked=0.3)
    announce("softmax odd rows", cols, dtype)
    got = host64(fs.row_softmax(dev(d["x"]), dev(d["mask"]), d["scale"]))
    m = d["mask"].f64()
    ref = oracle.row_softmax(d["x"].f64(), m, d["scale"])
    assert_close(f"odd rows {cols}", got, ref, *TOL[dtype])
    if dtype == "bf16":
        bf16_ulp_close(f"odd rows {cols}", got, ref, ulps=1.0, atol=1e-7)
    assert np.all(got[np.isinf(m)] == 0.0)


def test_odd_rows_head_and_tail_extremes():
    # the row maximum in the first or the last columns (read one per lane
    # next to the 16-byte body), masked heads and tails, an all-masked row
    rows, cols = 24, 2051
    x = torch.zeros(rows, cols, dtype=torch.bfloat16, device="cuda")
    m = torch.zeros(rows, cols, dtype=torch.bfloat16, device="cuda")
    for i, j in enumerate([0, 1, 6, 7, cols - 1, cols - 2, cols - 7, cols - 8]):
        x[i, j] = 30.0
        x[8 + i, j] = 30.0
        m[8 + i, j] = float("-inf")
        m[16 + i, :] = float("-inf")
        m[16 + i, j] = 0.0
    announce("softmax odd rows head and tail")
    got = host64(fs.row_softmax(x, m, 1.0))
    ref = oracle.row_softmax(host64(x), host64(m), 1.0)
    assert_close("head and tail", got, ref, *TOL["bf16"])
    for i, j in enumerate([0, 1, 6, 7, cols - 1, cols - 2, cols - 7, cols - 8]):
        assert got[i, j] > 0.99 and got[8 + i, j] == 0.0 and got[16 + i, j] == 1.0


@pytest.mark.parametrize("seed", SEEDS)
def test_causal_attention_scores(seed):
    # [2, 16, 512, 512] scores, causal, scale 1/8: the block's softmax shape
    b, h, s = 2, 16, 512
    d = fd.softmax_inputs(seed, b * h * s, s, "bf16", sigma=3.0, mask_dtype=None, scale=0.125)
    announce("softmax causal", seed)
    y = fs.row_softmax(dev(d["x"]), None, d["scale"], causal_q_len=s)
    got = host64(y)
    ref = oracle.row_softmax(d["x"].f64(), None, d["scale"], causal_q_len=s)
    assert_close(f"causal seed {seed}", got, ref, *TOL["bf16"])
    masked = oracle.causal_mask(b * h * s, s, s)
    softmax_supplementary(f"causal seed {seed}", got, ref, masked)
    one_hot = np.zeros(s)
    one_hot[0] = 1.0
    for r in range(0, b * h * s, s):          # row 0 of every head: exactly [1, 0, ...]
        np.testing.assert_array_equal(got[r], one_hot)


@pytest.mark.parametrize("q_len", [512, 64, 100, 48])
def test_causal_rows_beyond_one_trip_per_wave(q_len):
    """More rows than the one-wave grid covers in one trip, so waves advance
    their causal position by the grid step (power-of-two and other q_len)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    rows_per_trip = cus * 8 * 16 * 4 * 2       # grid cap x (4 waves x 2 rows) per block
    rows, cols = 2 * rows_per_trip + 13, 64
    d = fd.softmax_inputs(q_len, rows, cols, "bf16", mask_dtype=None)
    announce("softmax causal looping waves", q_len, rows)
    got = host64(fs.row_softmax(dev(d["x"]), None, d["scale"], causal_q_len=q_len))
    ref = oracle.row_softmax(d["x"].f64(), None, d["scale"], causal_q_len=q_len)
    assert_close(f"causal looping q_len {q_len}", got, ref, *TOL["bf16"])
    masked = oracle.causal_mask(rows, cols, q_len)
    softmax_supplementary(f"causal looping q_len {q_len}", got, ref, masked)


@pytest.mark.parametrize("q_len,cols", [(3, 10), (64, 512), (100, 4096), (512, 512), (37, 1001),
                                        (64, 4095), (9, 12289)])
def test_causal_offsets_and_widths(q_len, cols):
    rows = 3 * q_len
    d = fd.softmax_inputs(q_len + cols, rows, cols, "f32", mask_dtype="f32", p_masked=0.2)
    announce("softmax causal offset", q_len, cols)
    y = fs.row_softmax(dev(d["x"]), dev(d["mask"]), d["scale"], causal_q_len=q_len)
    ref = oracle.row_softmax(d["x"].f64(), d["mask"].f64(), d["scale"], causal_q_len=q_len)
    assert_close("causal offset", host64(y), ref, *TOL["f32"])


def test_fully_masked_rows_and_large_logits():
    # fp32 logits near 3e4 whose difference is ln 3: the exponent difference
    # must keep full relative accuracy
    x = torch.tensor([[1.0, 2.0, 3.0, 4.0], [3e4, 3e4 + float(np.log(3.0)), -3e4, 0.0],
                      [5.0, 5.0, 5.0, 5.0], [-3e4, -3e4, -3e4, -3e4 + 1.0]],
                     dtype=torch.float32, device="cuda")
    mask = torch.tensor([[-np.inf] * 4, [0, 0, -np.inf, -np.inf], [0, -np.inf, 0, -np.inf],
                         [-np.inf, -np.inf, 0, 0]], device="cuda", dtype=torch.float32)
    announce("softmax masked rows")
    y = host64(fs.row_softmax(x, mask, 1.0))
    np.testing.assert_array_equal(y[0], 0.0)
    assert not np.any(np.signbit(y[0]))
    x64 = host64(x)
    ref = oracle.row_softmax(x64, host64(mask), 1.0)
    assert_close("large and masked logits", y, ref, *TOL["f32"])
    np.testing.assert_allclose(y[2], [0.5, 0, 0.5, 0], rtol=1e-6)
    # very negative logits with an all-masked slice: no NaN, exact zeros where masked
    xs = torch.full((2, 4096), -3e4, dtype=torch.float32, device="cuda")
    xs[:, -1] = -2.9e4
    ms = torch.zeros_like(xs)
    ms[:, :2048] = float("-inf")
    ys = host64(fs.row_softmax(xs, ms, 1.0))
    assert not np.isnan(ys).any()
    assert np.all(ys[:, :2048] == 0.0)
    assert_close("negative logits", ys, oracle.row_softmax(host64(xs), host64(ms), 1.0),
                 *TOL["f32"])


def test_general_additive_mask():
    # a finite additive bias (not only 0/-inf)
    rng = np.random.default_rng(3)
    x = rng.standard_normal((9, 300)).astype(np.float32)
    m = (rng.standard_normal((9, 300)) * 2).astype(np.float32)
    y = fs.row_softmax(torch.from_numpy(x).cuda(), torch.from_numpy(m).cuda(), 0.5)
    ref = oracle.row_softmax(x.astype(np.float64), m.astype(np.float64), 0.5)
    assert_close("finite mask", host64(y), ref, *TOL["f32"])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_strided_misaligned_in_place_and_guards(dtype):
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rows, cols, ld = 21, 777, 800
    d = fd.softmax_inputs(21, rows, cols, dtype, mask_dtype=dtype)
    ref = oracle.row_softmax(d["x"].f64(), d["mask"].f64(), d["scale"])
    for offset in (0, 1):
        announce("softmax guard", dtype, offset)
        xg = Guarded(rows, cols, ld, tdt, offset=offset)
        xg.view.copy_(dev(d["x"]))
        mg = Guarded(rows, cols, ld + 8, tdt, offset=offset)
        mg.view.copy_(dev(d["mask"]))
        fs.row_softmax(xg.view, mg.view, d["scale"], out=xg.view)       # in place
        torch.cuda.synchronize()
        assert_close(f"strided in place offset {offset}", host64(xg.view), ref, *TOL[dtype])
        xg.check_untouched("softmax y")
        mg.check_untouched("softmax mask")


@pytest.mark.parametrize("offset", [0, 4, 8])
def test_bf16_mask_with_fp32_x_at_8_byte_offsets(offset):
    # fp32 x reads 4 mask elements (8 bytes of a bf16 mask) per 16-byte vector:
    # mask rows on 8-byte boundaries take the vector path, others the
    # element-wise one; both against the oracle, and bit for bit against the
    # same mask in a contiguous copy where both take the vector path
    rows, cols, ld = 19, 2048, 2048 + 4              # mask rows 4104 bytes apart
    d = fd.softmax_inputs(60 + offset, rows, cols, "f32", mask_dtype="bf16")
    announce("softmax fp32 x, bf16 mask offset", offset)
    buf = torch.zeros(rows * ld + 16, dtype=torch.bfloat16, device="cuda")
    e = offset // 2
    mview = buf[e:e + rows * ld].view(rows, ld)[:, :cols]
    mview.copy_(dev(d["mask"]))
    x = dev(d["x"])
    y = fs.row_softmax(x, mview, d["scale"])
    ref = oracle.row_softmax(d["x"].f64(), d["mask"].f64(), d["scale"])
    assert_close(f"offset {offset}", host64(y), ref, *TOL["f32"])
    if offset % 8 == 0:
        yc = fs.row_softmax(x, dev(d["mask"]), d["scale"])
        assert torch.equal(y.view(torch.int32), yc.view(torch.int32))


def test_repeatable():
    d = fd.softmax_inputs(5, 64, 4096)
    x, m = dev(d["x"]), dev(d["mask"])
    y1 = fs.row_softmax(x, m, d["scale"])
    y2 = fs.row_softmax(x, m, d["scale"])
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


@pytest.mark.slow
def test_beyond_2_31_elements():
    rows, cols = (1 << 19) + 5, 4096
    d = fd.softmax_inputs(8, 64, cols, "bf16")
    announce("softmax > 2^31 elements", rows, cols)
    rep = (rows + 63) // 64
    x = dev(d["x"]).repeat(rep, 1)[:rows]
    m = dev(d["mask"]).repeat(rep, 1)[:rows]
    y = fs.row_softmax(x, m, d["scale"])
    idx = np.array([0, 1, 64, rows // 2 + 7, rows - 1])
    got = host64(y[torch.from_numpy(idx).cuda()])
    ref = oracle.row_softmax(d["x"].rows(idx % 64).f64(), d["mask"].rows(idx % 64).f64(),
                             d["scale"])
    assert_close("beyond 2^31", got, ref, *TOL["bf16"])
    bf16_ulp_close("beyond 2^31", got, ref, atol=1e-7)


@pytest.mark.parametrize("q_len", [(1 << 30) - 1, 1 << 30, (1 << 40) + 5])
def test_huge_causal_q_len(q_len):
    # q_len at or above 2^30 takes the row cache (64-bit positions);
    # with q_len > cols every row here lies wholly above the diagonal shift,
    # so the oracle's rule masks it completely: all outputs are +0
    d = fd.softmax_inputs(5, 6, 64, "bf16", mask_dtype=None)
    announce("softmax huge causal q_len", q_len)
    got = host64(fs.row_softmax(dev(d["x"]), None, 0.5, causal_q_len=q_len))
    ref = oracle.row_softmax(d["x"].f64(), None, 0.5, causal_q_len=q_len)
    np.testing.assert_array_equal(ref, 0.0)
    np.testing.assert_array_equal(got, ref)


@pytest.mark.parametrize("cols", [64, 4096, 40000, 70000])
def test_extreme_finite_logits_and_lowest_value_masks(cols):
    # rows masked with the most negative finite value (a common padding
    # mask), rows whose maximum is far past 1e9, and a fully masked row: the
    # exponent differences are formed before the scaling, so every row stays
    # finite and matches the oracle (a fully lowest-masked row is uniform)
    low = float(np.finfo(np.float32).min)
    x = torch.zeros(6, cols, device="cuda")
    x[0, :] = low                                   # every position masked
    x[1, : cols // 2] = low
    x[2, :] = 1e30
    x[2, 1] = 1e30 * (1 - 2 ** -20)
    x[3, :] = 3e38
    x[4, :] = torch.linspace(-5e9, 5e9, cols, device="cuda")
    x[5, 3] = -3e9
    announce("softmax extreme logits", cols)
    y = host64(fs.row_softmax(x, None, 1.0))
    ref = oracle.row_softmax(host64(x), None, 1.0)
    assert np.isfinite(y).all()
    assert_close(f"extreme logits {cols}", y, ref, *TOL["f32"])
    np.testing.assert_allclose(y[0], 1.0 / cols, rtol=1e-5)
