"""GPU parity of fs_causal_softmax_trimmed: the written columns j < w(r)
match the float64 softmax, and every column from w(r) on keeps its previous
bits (a guard pattern), for square and rectangular causal rows, block sizes
from 1 to beyond the row, register and streamed rows, in place."""
import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
import paper_2609_30059_amd as fs
from gpu_util import TOL, announce, assert_close, bf16_ulp_close, dev, host64

pytestmark = pytest.mark.gpu

GUARD = {torch.bfloat16: 0x7FC3, torch.float32: 0x7FC00033}   # distinct quiet-NaN payloads


def guard_like(x):
    y = torch.empty_like(x)
    if x.dtype == torch.bfloat16:
        y.view(torch.int16).fill_(GUARD[x.dtype])
    else:
        y.view(torch.int32).fill_(GUARD[x.dtype])
    return y


def check(name, x_host, y, scale, q, block, dtype):
    rows, cols = x_host.shape
    ref = oracle.row_softmax(x_host, None, scale, causal_q_len=q)
    w = oracle.causal_written_width(rows, cols, q, block)
    written = np.arange(cols)[None, :] < w[:, None]
    got = host64(y)
    assert_close(name, np.where(written, got, 0.0), np.where(written, ref, 0.0), *TOL[dtype])
    if dtype == "bf16":
        bf16_ulp_close(name, got[written], ref[written], ulps=1.0, atol=1e-9)
    bits = (y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32)).cpu().numpy()
    untouched = bits[~written]
    assert np.all(untouched == np.array(GUARD[y.dtype]).astype(untouched.dtype)), \
        f"{name}: a column at or beyond w(r) was written"
    masked = oracle.causal_mask(rows, cols, q) & written
    assert np.all(got[masked] == 0.0) and not np.any(np.signbit(got[masked]))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("block", [1, 8, 64, 128, 512, 1024])
def test_square_attention_rows(dtype, block):
    q = 512
    rows = 3 * q                                      # three (head, sequence) pairs
    d = fd.softmax_inputs(block, rows, q, dtype, mask_dtype=None, sigma=3.0)
    announce("trimmed softmax", dtype, block)
    x = dev(d["x"])
    y = guard_like(x)
    fs.causal_softmax_trimmed(x, d["scale"], q, block, out=y)
    torch.cuda.synchronize()
    check(f"block {block}", d["x"].f64(), y, d["scale"], q, block, dtype)


# register rows, the 16-wave rung (20000), the row cache with element-wise
# loads (33333, 100001 with a streamed tail) and with 16-byte loads (50000,
# 70000 with a tail)
@pytest.mark.parametrize("rows,cols,q,block,dtype", [
    (37, 40, 10, 4, "f32"), (20, 3000, 2900, 256, "f32"), (16, 20000, 20000, 4096, "f32"),
    (9, 33333, 9, 1024, "f32"), (6, 50000, 40000, 2048, "bf16"), (6, 70000, 70000, 8192, "f32"),
    (5, 100001, 3, 16384, "f32"), (37, 1001, 1001, 64, "bf16"), (19, 4095, 300, 128, "bf16"),
    (11, 12289, 12289, 1024, "bf16"), (13, 2051, 2051, 16, "f32")])
def test_rectangular_ragged_and_streamed(rows, cols, q, block, dtype):
    d = fd.softmax_inputs(rows + cols, rows, cols, dtype, mask_dtype=None, sigma=2.0)
    announce("trimmed softmax rect", rows, cols, q, block, dtype)
    x = dev(d["x"])
    y = guard_like(x)
    fs.causal_softmax_trimmed(x, d["scale"], q, block, out=y)
    torch.cuda.synchronize()
    check(f"{rows}x{cols} q{q} b{block}", d["x"].f64(), y, d["scale"], q, block, dtype)


def test_in_place_keeps_the_unwritten_logits():
    q, block = 256, 64
    d = fd.softmax_inputs(4, 2 * q, q, "bf16", mask_dtype=None)
    announce("trimmed softmax in place")
    x = dev(d["x"])
    before = x.clone()
    fs.causal_softmax_trimmed(x, d["scale"], q, block, out=x)
    torch.cuda.synchronize()
    w = oracle.causal_written_width(2 * q, q, q, block)
    written = torch.from_numpy(np.arange(q)[None, :] < w[:, None]).cuda()
    assert torch.equal(x.view(torch.int16)[~written], before.view(torch.int16)[~written])
    ref = oracle.row_softmax(d["x"].f64(), None, d["scale"], causal_q_len=q)
    got = host64(x)
    wn = written.cpu().numpy()
    assert_close("in place", got[wn], ref[wn], *TOL["bf16"])


def test_full_block_equals_row_softmax():
    # a block covering the whole row writes everything: bit-identical to the
    # untrimmed causal softmax
    q = 512
    d = fd.softmax_inputs(77, 4 * q, q, "bf16", mask_dtype=None)
    x = dev(d["x"])
    a = fs.causal_softmax_trimmed(x, d["scale"], q, 512)
    b = fs.row_softmax(x, None, d["scale"], causal_q_len=q)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
