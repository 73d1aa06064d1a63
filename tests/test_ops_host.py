"""Host tests of the binding's tensor marshalling (no GPU): the (rows, cols,
ld) view of a tensor, on CPU tensors of every layout the ops accept or refuse."""
import pytest
import torch

from paper_2609_30059_amd.ops import as_rows


@pytest.mark.parametrize("shape", [(2, 3, 4), (1, 5), (5, 1), (1, 1), (7, 9), (2, 1, 3, 8)])
def test_contiguous_tensors_are_dense_rows(shape):
    t = torch.empty(shape)
    cols = shape[-1]
    assert as_rows(t) == (t.numel() // cols, cols, cols)


def test_row_strided_and_degenerate_views():
    base = torch.empty(6, 10)
    assert as_rows(base[:, :7]) == (6, 7, 10)                 # ld > cols
    assert as_rows(base[2:3, :7]) == (1, 7, 7)                # one row: ld = cols
    assert as_rows(torch.empty(4, 3, 10)[:, :, :5]) == (12, 5, 10)
    assert as_rows(torch.empty(3, 0)) == (3, 0, 1)            # empty rows
    assert as_rows(torch.empty(0, 3)) == (0, 3, 3)
    assert as_rows(torch.empty(8)) == (1, 8, 8)
    assert as_rows(torch.empty(0)) == (1, 0, 1)
    # every other row of a [4, 6, 8] block: strides (48, 16, 1) still make
    # one row stride of 16 elements
    assert as_rows(torch.empty(4, 6, 8)[:, ::2, :]) == (12, 8, 16)


def test_layouts_that_are_refused():
    with pytest.raises(ValueError):
        as_rows(torch.tensor(1.0))                            # scalar
    with pytest.raises(ValueError):
        as_rows(torch.empty(4, 6).t())                        # last dim not contiguous
    with pytest.raises(ValueError):
        as_rows(torch.empty(4, 6, 8)[:, :3, :])               # rows 8 apart, batches 48 apart


def test_size_one_leading_dims_do_not_set_the_row_stride():
    # a size-1 dim between the rows and the columns may carry any stride
    t = torch.empty(3, 10).as_strided((3, 1, 5), (10, 999, 1))
    assert as_rows(t) == (3, 5, 10)


@pytest.mark.parametrize("make", [
    lambda: torch.randn(1, 5).expand(3, 5),                   # broadcast rows (stride 0)
    lambda: torch.empty(20).as_strided((3, 5), (2, 1)),       # overlapping rows
    lambda: torch.empty(10)[::2],                             # 1-D with stride 2
    lambda: torch.randn(1).expand(5),                         # 1-D broadcast
    lambda: torch.randn(1, 3, 5).expand(2, 3, 5),             # broadcast batch
])
def test_broadcast_and_overlapping_views_are_refused(make):
    with pytest.raises(ValueError):
        as_rows(make())
