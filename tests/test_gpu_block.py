"""GPU parity of the stitched transformer block (fused sub-kernels between
hipBLASLt GEMMs) against the float64 block oracle, end to end and stage by
stage."""
import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
import paper_2609_30059_amd as fs
from gpu_util import SEEDS, TOL, announce, assert_close, dev, host64

pytestmark = pytest.mark.gpu

STAGES = ("a", "qkv", "probs", "o", "att", "h1", "m", "u", "g", "d", "out")


def run_block(d, heads, seqs, attn_block=None):
    params = {k: dev(d[k]) for k in fs.block.PARAM_NAMES}
    blk = fs.TransformerBlock(params, heads=heads, eps=d["eps"], attn_block=attn_block)
    x = dev(d["x"])
    buf = blk.forward(x)
    torch.cuda.synchronize()
    p64 = {k: d[k].f64() for k in fs.block.PARAM_NAMES}
    ref = oracle.block_forward(d["x"].f64(), p64, heads, d["eps"], sequences=seqs,
                               keep=STAGES + ("scores",))
    return buf, ref


# The block keeps its residual stream in bf16 (h1 is stored, then added to the
# MLP branch).  Where a residual add cancels, the exact result can be far
# smaller than its operands, so those two stages also allow one bf16 rounding
# (2^-8 relative, a bound on half a unit in the last place) of each operand.
RESIDUAL_OPERANDS = {"h1": ("x", "att"), "out": ("h1", "d")}


def compare(buf, ref, seqs, batch, seq, name, x64=None, block=None):
    atol, rtol = TOL["bf16"]
    for st in STAGES:
        if st == "probs":
            # device probs are head-major [heads, batch, seq, seq]; with
            # causal row blocks, columns beyond a row's block are unwritten
            got = host64(buf["probs"][:, seqs].transpose(0, 1))
            if block is not None:
                w = oracle.causal_written_width(seq, seq, seq, block)
                got = np.where(np.arange(seq)[None, :] < w[:, None], got, 0.0)
        else:
            got = host64(buf[st].view(batch, seq, -1)[seqs])
        want = ref[st]
        a = atol
        if st in RESIDUAL_OPERANDS:
            ops = [x64 if o == "x" else ref[o] for o in RESIDUAL_OPERANDS[st]]
            a = atol + 2.0 ** -8 * (np.abs(ops[0]) + np.abs(ops[1]))
        assert_close(f"{name} stage {st}", got, want, a, rtol)


@pytest.mark.parametrize("seed", SEEDS)
def test_small_block_all_stages(seed):
    d = fd.block_inputs(seed, batch=3, seq=64, hidden=256, heads=4, mlp=1024)
    announce("block small", seed)
    buf, ref = run_block(d, 4, [0, 1, 2])
    compare(buf, ref, [0, 1, 2], 3, 64, f"small seed {seed}", d["x"].f64()[[0, 1, 2]])


@pytest.mark.parametrize("attn_block", [1, 16, 32, 64])
def test_small_block_causal_row_blocks(attn_block):
    # the q k^T and P v products issued per causal row block, down to one row
    d = fd.block_inputs(attn_block, batch=2, seq=64, hidden=256, heads=4, mlp=1024)
    announce("block row blocks", attn_block)
    buf, ref = run_block(d, 4, [0, 1], attn_block=attn_block)
    compare(buf, ref, [0, 1], 2, 64, f"row block {attn_block}", d["x"].f64()[[0, 1]],
            block=attn_block)


def test_block_causality_on_gpu():
    d = fd.block_inputs(1, batch=2, seq=128, hidden=256, heads=4, mlp=512)
    params = {k: dev(d[k]) for k in fs.block.PARAM_NAMES}
    blk = fs.TransformerBlock(params, heads=4, eps=d["eps"])
    x = dev(d["x"])
    y1 = blk.forward(x)["out"].clone()
    x2 = x.clone()
    x2[:, 100:] = torch.randn_like(x2[:, 100:].float()).to(torch.bfloat16) * 4
    y2 = blk.forward(x2)["out"]
    y1 = y1.view(2, 128, -1)
    y2 = y2.view(2, 128, -1)
    assert torch.equal(y1[:, :100], y2[:, :100])
    assert not torch.equal(y1[:, 100:], y2[:, 100:])
