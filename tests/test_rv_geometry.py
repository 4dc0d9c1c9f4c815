"""Host-side checks of the row-major 16-byte update's geometry (the kernel
itself is covered by the GPU tests):

* tile widths: a matrix of m columns is cut into ceil(m / kRvMaxCols) tiles
  of equal width rounded up to a multiple of 8 -- every tile fits
  kRvMaxCols and the tiles cover the columns;
* the lane budget of a block's roles, for every tile width up to
  kRvMaxCols, every alignment of the tile's first unselected slot and
  every number of selected columns in the tile: the whole quads of the
  unselected range plus its edge slots (at most 6) leave at least one lane
  for the selected slots whenever there are any, and no Adam lane holds
  more than 4 of them;
* the padding helpers of the binding (16-byte rows for the row-major
  layout).

kRvMaxCols is read from the library's header, so a change there is checked
against the same invariants the kernel's static_assert summarises.
"""
import os
import re

import numpy as np
import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = os.path.join(ROOT, "paper_2505_12242_amd", "csrc", "zf_internal.hpp")
THREADS = 256


def rv_max_cols() -> int:
    m = re.search(r"constexpr int kRvMaxCols = (\d+);", open(HDR).read())
    assert m, "kRvMaxCols not found"
    return int(m.group(1))


def rv_width(m: int, maxc: int) -> int:
    tiles = max(1, -(-m // maxc))
    return 8 * -(-max(m, 1) // (8 * tiles))


def test_tile_widths_fit_and_cover():
    maxc = rv_max_cols()
    assert maxc % 8 == 0
    for m in list(range(1, 5000)) + [11008, 13824, 28672, 32000, 70001, 1 << 20]:
        w = rv_width(m, maxc)
        assert w % 8 == 0 and 8 <= w <= maxc, m
        tiles = -(-m // w)
        assert (tiles - 1) * w < m <= tiles * w, m


def test_role_lane_budget():
    maxc = rv_max_cols()
    worst_j = 0
    for width in range(1, maxc + 1):
        cs = np.arange(width + 1)            # selected columns in the tile
        cu = width - cs                      # unselected
        for us4 in range(4):                 # alignment of the first unselected slot
            qf0 = -(-us4 // 4)
            qf1 = (us4 + cu) // 4
            nqf = np.maximum(qf1 - qf0, 0)
            ne = np.where(nqf > 0, (4 * qf0 - us4) + (us4 + cu - 4 * qf1), cu)
            ne = np.where(cu > 0, ne, 0)
            nqf = np.where(cu > 0, nqf, 0)
            assert ne.max() <= 6
            lanes_a = THREADS - nqf - ne
            has_sel = cs > 0
            assert (lanes_a[has_sel] >= 1).all(), (width, us4)
            j = -(-cs[has_sel] // lanes_a[has_sel])
            if j.size:
                worst_j = max(worst_j, int(j.max()))
    assert worst_j <= 4


def test_alloc_stored_pads_row_major_rows():
    zf = pytest.importorskip("paper_2505_12242_amd")
    t = zf.alloc_stored(zf.ROW_MAJOR, 5, 7, torch.float32, "cpu")
    assert t.shape == (5, 7) and t.stride() == (8, 1)
    b = zf.alloc_stored(zf.ROW_MAJOR, 3, 9, torch.bfloat16, "cpu")
    assert b.shape == (3, 9) and b.stride() == (16, 1)
    c = zf.alloc_stored(zf.CHANNEL_MAJOR, 5, 7, torch.float32, "cpu")
    assert c.shape == (7, 5) and c.is_contiguous()
    from paper_2505_12242_amd._lib import padded_block
    blk = padded_block(t)
    assert blk.shape == (5, 8) and blk.is_contiguous() and blk.data_ptr() == t.data_ptr()
