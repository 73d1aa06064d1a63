"""The hipBLASLt wrapper (the fixed library GEMMs) against float64 products
of the same bf16 operands: orientation, transposes, bias, strided batches."""
import numpy as np
import pytest
import torch

import fusedsub_data as fd
import paper_2609_30059_amd as fs
from gpu_util import announce, assert_close, dev, host64

pytestmark = pytest.mark.gpu


def bf(shape, seed, std=1.0):
    rng = np.random.default_rng(seed)
    return fd.Tensor(fd.f32_to_bf16_bits(rng.standard_normal(shape) * std), "bf16")


@pytest.mark.parametrize("m,n,k", [(1, 1, 1), (17, 33, 65), (256, 512, 128), (1000, 3072, 1024)])
@pytest.mark.parametrize("trans_b", [False, True])
@pytest.mark.parametrize("with_bias", [False, True])
def test_gemm(m, n, k, trans_b, with_bias):
    a = bf((m, k), 1, 0.1)
    b = bf((n, k) if trans_b else (k, n), 2, 0.1)
    bias = bf((n,), 3, 0.1) if with_bias else None
    announce("gemm", m, n, k, trans_b, with_bias)
    c = fs.gemm(dev(a), dev(b), bias=dev(bias) if bias else None, trans_b=trans_b)
    bm = b.f64().T if trans_b else b.f64()
    ref = a.f64() @ bm + (bias.f64()[None, :] if bias else 0.0)
    assert_close("gemm", host64(c), ref, 1e-2, 1e-2)


def test_strided_batched_head_views():
    # S[h] = q_h k_h^T over head views of a [tokens, 3H] buffer, batch over heads
    s, H, nh = 64, 256, 4
    dh = H // nh
    qkv = bf((s, 3 * H), 4, 0.5)
    out = torch.empty(nh, s, s, dtype=torch.bfloat16, device="cuda")
    t = dev(qkv)
    es = 2
    fs.gemm_strided_batched(t.data_ptr(), 3 * H, dh, t.data_ptr() + H * es, 3 * H, dh, True,
                            out.data_ptr(), s, s * s, s, s, dh, nh)
    q = qkv.f64()
    for h in range(nh):
        ref = q[:, h * dh:(h + 1) * dh] @ q[:, H + h * dh:H + (h + 1) * dh].T
        assert_close(f"head {h}", host64(out[h]), ref, 1e-2, 1e-2)
