"""Host-side checks of the tile-major code layout helpers (no GPU): the
binding's untile() inverts the placement the header defines,
((r / 16) * (ld / 64) + k / 64) * 1024 + (r % 16) * 64 + k % 64."""
import numpy as np
import pytest


@pytest.mark.parametrize("rows,cols", [(1, 1), (16, 64), (17, 65), (100, 300), (33, 128)])
def test_untile_inverts_the_documented_placement(rows, cols):
    import torch
    from paper_2411_10948_amd import shiftquant as sq
    t = sq.code_matrix(rows, cols, True, "cpu")
    ld = t.stride(0)
    assert ld % 64 == 0 and ld >= cols
    assert t.untyped_storage().nbytes() >= sq.round_up(rows, 16) * ld
    rng = np.random.default_rng(rows * 1000 + cols)
    want = rng.integers(-127, 128, (rows, ld)).astype(np.int8)
    flat = np.zeros(sq.round_up(rows, 16) * ld, np.int8)
    r, k = np.meshgrid(np.arange(rows), np.arange(ld), indexing="ij")
    off = ((r // 16) * (ld // 64) + k // 64) * 1024 + (r % 16) * 64 + k % 64
    flat[off.ravel()] = want.ravel()
    assert len(np.unique(off)) == off.size          # a bijection onto the buffer
    buf = torch.from_numpy(flat).view(-1, ld)[:rows]
    np.testing.assert_array_equal(sq.untile(buf).numpy(), want)


def test_row_major_code_matrix():
    from paper_2411_10948_amd import shiftquant as sq
    t = sq.code_matrix(5, 20, False, "cpu")
    assert t.shape == (5, 32) and t.stride(0) == 32
