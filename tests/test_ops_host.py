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
