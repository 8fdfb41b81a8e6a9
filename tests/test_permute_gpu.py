"""GPU: gtr_scan_permute is bit-exact against the oracle's index gather, for all
four directions, three dtypes, square and non-square grids, and row widths that
take each copy width (16, 8, 4, 2, 1 bytes)."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

DTYPES = [torch.float16, torch.bfloat16, torch.float32]
GRIDS = [(1, 1), (3, 1), (1, 5), (7, 9), (40, 40), (80, 80)]


def as_bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    return (t.view(torch.int16) if t.element_size() == 2 else t.view(torch.int32)).numpy()


@pytest.mark.parametrize("dtype", DTYPES, ids=str)
@pytest.mark.parametrize("H,W", GRIDS)
@pytest.mark.parametrize("scan", ["row", "col", "row_rev", "col_rev"])
def test_permute_bit_exact(gtr, scan, H, W, dtype):
    g = torch.Generator().manual_seed(H * 100 + W)
    for E in (64, 3, 1):
        x = torch.randn((2, 3, H * W, E), generator=g).to(dtype)
        xd = x.cuda()
        y = gtr.gtr_scan_permute(xd, H, W, scan)
        ref = oracle.permute(as_bits(x), H, W, scan)
        np.testing.assert_array_equal(as_bits(y), ref)
        back = gtr.gtr_scan_permute(y, H, W, scan, inverse=True)
        np.testing.assert_array_equal(as_bits(back), as_bits(x))


def test_permute_col_is_grid_transpose(gtr):
    H, W, E = 6, 11, 8
    x = torch.arange(H * W * E, dtype=torch.float32).view(1, H * W, E).cuda()
    y = gtr.gtr_scan_permute(x, H, W, "col")
    want = x.view(H, W, E).transpose(0, 1).reshape(1, H * W, E)
    assert torch.equal(y, want)
