"""The binding's reading of torch tensors as logical matrices (host only).

The C ABI reads a zero stride as "dense default", so the binding must turn
every real layout into explicit strides and refuse layouts whose rows,
blocks or planes overlap (expanded or broadcast tensors)."""
import pytest

torch = pytest.importorskip("torch")

from paper_2609_21594_amd.binding import RowBlocks, _view  # noqa: E402


def fields(x):
    return _view(x)[1:]  # (batch, rows, cols, ld, row_block, block_stride, plane_stride)


def test_dense_and_strided_views():
    W = torch.zeros(12, 8)
    assert fields(W) == (1, 12, 8, 8, 0, 0, 0)
    assert fields(W[:, 2:6]) == (1, 12, 4, 8, 0, 0, 0)
    assert fields(W.view(3, 4, 8)) == (3, 4, 8, 8, 0, 0, 32)
    assert fields(RowBlocks(W.view(2, 3, 2, 8)[:, 0])) == (1, 4, 8, 8, 2, 48, 0)
    assert fields(torch.zeros(4, 6, 10)[:, :, 5:]) == (4, 6, 5, 10, 0, 0, 60)


def test_singleton_dimensions_take_dense_strides():
    assert fields(torch.zeros(1, 5)) == (1, 1, 5, 5, 0, 0, 0)
    assert fields(torch.zeros(7, 1)) == (1, 7, 1, 1, 0, 0, 0)
    one_row_blocks = RowBlocks(torch.zeros(3, 1, 16))  # 3 blocks of 1 row
    assert fields(one_row_blocks) == (1, 3, 16, 16, 1, 16, 0)


@pytest.mark.parametrize("make", [
    lambda: torch.zeros(1, 8).expand(16, 8),               # rows share storage
    lambda: torch.zeros(8, 8).as_strided((8, 8), (4, 1)),  # rows overlap
    lambda: torch.zeros(1, 4, 8).expand(3, 4, 8),          # planes share storage
    lambda: RowBlocks(torch.zeros(1, 2, 8).expand(3, 2, 8)),  # blocks share storage
])
def test_overlapping_layouts_are_refused(make):
    with pytest.raises(ValueError):
        _view(make())


def test_columns_must_be_contiguous():
    with pytest.raises(ValueError):
        _view(torch.zeros(8, 8).t())


def test_tensors_off_the_handles_device_are_refused():
    from paper_2609_21594_amd.binding import _check_device
    W = torch.zeros(4, 8)
    with pytest.raises(ValueError, match="cuda:0"):
        _check_device([W], 0)
    with pytest.raises(ValueError):
        _check_device([RowBlocks(W.view(2, 2, 8))], 0)
    _check_device([], 0)


def test_coefficient_tables_must_match_the_step_count():
    # the library reads 3 * ns_steps values from the table
    from paper_2609_21594_amd.binding import make_hparams
    make_hparams(ns_coeffs=[(1.5, -0.5, 0.0)] * 3, ns_steps=3)
    with pytest.raises(ValueError):
        make_hparams(ns_coeffs=[(1.5, -0.5, 0.0)] * 2, ns_steps=3)
    with pytest.raises(ValueError):
        make_hparams(ns_coeffs=[(1.5, -0.5)] * 3, ns_steps=3)


def test_optimizer_needs_gpu_parameters():
    from paper_2609_21594_amd.optim import MuonAdamW
    with pytest.raises(ValueError, match="one GPU"):
        MuonAdamW([torch.nn.Parameter(torch.zeros(4, 4))])
