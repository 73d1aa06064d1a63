"""GPU parity of fs_copy_strided against the oracle: bit-exact on random bit
patterns (NaN payloads included), head split / merge shapes of the block,
ragged and unaligned strides that take the element path, and guard bands
around the destination that must stay untouched."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_30059_amd as fs
from gpu_util import announce

pytestmark = pytest.mark.gpu


def bits(n, dtype, seed):
    rng = np.random.default_rng(seed)
    if dtype == torch.bfloat16:
        h = rng.integers(0, 1 << 16, size=n, dtype=np.uint16)
        return torch.from_numpy(h.view(np.int16)).view(torch.bfloat16).cuda(), h
    h = rng.integers(0, 1 << 32, size=n, dtype=np.uint32)
    return torch.from_numpy(h.view(np.int32)).view(torch.float32).cuda(), h


def as_bits(t):
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.view(torch.int32).cpu().numpy().view(np.uint32)


CASES = [
    # rows, cols, batch, ld_src, stride_src, ld_dst, stride_dst
    ("head split", 512, 64, 48, 3072, 64, 64, 512 * 64),
    ("head merge", 512, 64, 16, 64, 512 * 64, 1024, 64),
    ("ragged batch-outer", 37, 13, 5, 20, 13 * 37 + 3, 13, 13 * 37 + 1),
    ("odd strides", 9, 7, 3, 11, 101, 9, 80),
    ("single row", 1, 100, 4, 100, 100, 100, 128),
    ("broadcast", 16, 40, 6, 40, 0, 40, 640),
    ("wide rows", 3, 20000, 2, 20008, 60024, 20000, 60000),
]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_matches_oracle_bit_exact(dtype, case):
    name, rows, cols, batch, lds, sts, ldd, std = case
    announce("copy_strided", name, dtype)
    n_src = (batch - 1) * sts + (rows - 1) * lds + cols
    n_dst = (batch - 1) * std + (rows - 1) * ldd + cols
    guard = 64
    src, hsrc = bits(n_src, dtype, rows * 7 + cols)
    dst, hdst = bits(n_dst + 2 * guard, dtype, rows + cols * 3)
    body = dst[guard:guard + n_dst]
    fs.copy_strided(body, src, rows, cols, batch, lds, sts, ldd, std)
    torch.cuda.synchronize()
    want = oracle.strided_copy(hsrc, hdst[guard:guard + n_dst], rows, cols, batch, lds, sts,
                               ldd, std)
    got = as_bits(dst)
    np.testing.assert_array_equal(got[guard:guard + n_dst], want)
    np.testing.assert_array_equal(got[:guard], hdst[:guard])
    np.testing.assert_array_equal(got[guard + n_dst:], hdst[guard + n_dst:])


def test_block_head_split_at_full_shape():
    # [16384, 3072] -> [48, 16384, 64] bf16, as the block's attention uses it
    t, nh, dh = 16384, 16, 64
    announce("copy_strided full head split")
    x = torch.randn(t, 3 * nh * dh, device="cuda").to(torch.bfloat16)
    y = torch.empty(3 * nh, t, dh, dtype=torch.bfloat16, device="cuda")
    fs.copy_strided(y, x, t, dh, 3 * nh, 3 * nh * dh, dh, dh, t * dh)
    want = x.view(t, 3 * nh, dh).transpose(0, 1)
    assert torch.equal(y.view(torch.int16), want.contiguous().view(torch.int16))
    z = torch.empty(t, nh * dh, dtype=torch.bfloat16, device="cuda")
    fs.copy_strided(z, y[:nh].contiguous(), t, dh, nh, dh, t * dh, nh * dh, dh)
    assert torch.equal(z.view(torch.int16), x[:, :nh * dh].contiguous().view(torch.int16))


def test_rejects_too_small_tensors_on_the_host():
    x = torch.empty(100, dtype=torch.bfloat16, device="cuda")
    y = torch.empty(100, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError):
        fs.copy_strided(y, x, 10, 10, 2, 10, 100, 10, 50)
