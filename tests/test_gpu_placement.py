"""GPU accuracy of the epilogue placements compared by the placement study:
the GEMM with hipBLASLt's own epilogues (per-column alpha, fp32 bias, GELU,
ReLU, beta * C residual) against the float64 definitions, next to the
separate libfusedsub epilogues."""
import math

import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
import paper_2609_30059_amd as fs
from gpu_util import TOL, announce, assert_close, dev, host64
from paper_2609_30059_amd.block import PARAM_NAMES
from paper_2609_30059_amd.placement import LibraryEpilogueBlock

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", [0, 1])
def test_sigmoid_row_sum_placements(seed):
    m, n, k = 256, 1024, 512
    h = fd.gemm_epilogue_inputs(seed, m, n, k)
    announce("placement sigmoid", seed)
    a, b, bias, scale = dev(h["a"]), dev(h["b"]), dev(h["bias"]), dev(h["col_scale"])
    c = fs.gemm(a, b)
    sep = fs.gemm_epilogue_reduce(c, bias, scale, "sigmoid", "sum")
    z = fs.gemm(a, b, bias=(bias.float() * scale).contiguous(), col_scale=scale)
    lib = fs.gemm_epilogue_reduce(z, None, None, "sigmoid", "sum")
    torch.cuda.synchronize()
    ref = oracle.gemm_epilogue_reduce(h["a"].f64() @ h["b"].f64(), h["bias"].f64(),
                                      h["col_scale"].f64(), "sigmoid", "sum")
    err_sep = np.abs(host64(sep) - ref).max()
    err_lib = np.abs(host64(lib) - ref).max()
    print(f"sigmoid row sum max |err|: separate {err_sep:.3e}  library {err_lib:.3e}", flush=True)
    # both round a GEMM output to bf16 before the sigmoid: C itself, or
    # (C + bias) * scale; sigma' <= 1/4 and the arguments stay below ~2
    assert_close("separate", host64(sep), ref, 1e-5 * n, 1e-4)
    assert_close("library affine", host64(lib), ref, 2.0 ** -9 * n, 1e-4)


def test_gemm_epilogue_options_against_float64():
    m, n, k = 192, 320, 256
    rng = np.random.default_rng(5)
    A = fd.Tensor(fd.f32_to_bf16_bits(rng.standard_normal((m, k)) * 0.1), "bf16")
    B = fd.Tensor(fd.f32_to_bf16_bits(rng.standard_normal((k, n)) * 0.1), "bf16")
    R = fd.Tensor(fd.f32_to_bf16_bits(rng.standard_normal((m, n))), "bf16")
    bias = fd.Tensor(fd.f32_to_bf16_bits(rng.standard_normal(n) * 0.5), "bf16")
    announce("placement gemm options")
    z = A.f64() @ B.f64() + bias.f64()[None, :]
    a, b, r, bb = dev(A), dev(B), dev(R), dev(bias)
    # residual as beta * C: one bf16 rounding of the exact sum
    y = fs.gemm(a, b, bias=bb, c_in=r, beta=1.0)
    assert_close("beta residual", host64(y), z + R.f64(), *TOL["bf16"])
    # relu and gelu epilogues
    y = fs.gemm(a, b, bias=bb, act="relu")
    assert_close("relu", host64(y), np.maximum(z, 0.0), *TOL["bf16"])
    y = fs.gemm(a, b, bias=bb, act="gelu")
    gelu = 0.5 * z * (1.0 + np.vectorize(math.erf)(z / math.sqrt(2.0)))
    err = np.abs(host64(y) - gelu).max()
    print(f"hipBLASLt GELU vs GELU_erf max |err| {err:.3e}", flush=True)
    assert_close("gelu", host64(y), gelu, *TOL["bf16"])


@pytest.mark.parametrize("seed", [0, 1])
def test_library_epilogue_block_matches_oracle(seed):
    d = fd.block_inputs(seed, batch=3, seq=64, hidden=256, heads=4, mlp=1024)
    announce("placement block", seed)
    params = {k: dev(d[k]) for k in PARAM_NAMES}
    blk = LibraryEpilogueBlock(params, heads=d["heads"], eps=d["eps"])
    buf = blk.forward(dev(d["x"]))
    torch.cuda.synchronize()
    ref = oracle.block_forward(d["x"].f64(), {k: d[k].f64() for k in PARAM_NAMES}, d["heads"],
                               d["eps"], sequences=[0, 1, 2], keep=("g", "out", "h1", "d"))
    atol, rtol = TOL["bf16"]
    got_g = host64(buf["g"]).reshape(3, 64, -1)
    assert_close("library gelu", got_g, ref["g"], atol, rtol)
    a = atol + 2.0 ** -8 * (np.abs(ref["h1"]) + np.abs(ref["d"]))
    assert_close("library out", host64(buf["out"]).reshape(3, 64, -1), ref["out"], a, rtol)


@pytest.mark.skip(reason="the timed hipBLASLt algorithm search was removed: a run that timed "
                         "16 heuristic candidates per GEMM shape of the block ended with "
                         "hipBLASLt's 'Could not initialize Tensile host' error, a segmentation "
                         "fault and a GPU fault whose cause inside the library was not found")
def test_algo_search_gives_the_same_product():
    raise AssertionError("not run: the feature it tested was removed")
