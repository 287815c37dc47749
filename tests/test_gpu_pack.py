"""Packed weight layout (hpd_pack_weight / hpd_pack_gate_up): bit-exact
against a numpy permutation written from the layout's definition."""

import numpy as np
import pytest
import torch

from ._gpu import announce

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def packed_ref(w):
    """Tiles of 32 rows x 64 columns in (row tile, column tile) order; inside a
    tile, 16-byte piece (j, l) = row l % 32, columns 32 (l / 32) + 8 j .. + 7."""
    rows, cols = w.shape
    t = w.reshape(rows // 32, 32, cols // 64, 2, 4, 8)      # R, r, C, h, j, e
    return t.transpose(0, 2, 4, 3, 1, 5).reshape(rows, cols)  # R, C, j, l = 32 h + r, e


def _bits(rng, shape):
    return rng.integers(0, 1 << 16, size=shape, dtype=np.uint16)


def _dev(a):
    return torch.from_numpy(a.view(np.int16)).cuda()


@pytest.mark.parametrize("rows,cols", [(32, 64), (64, 192), (1792, 3072), (8960, 1536)])
def test_pack_weight_bit_exact(rows, cols):
    announce(f"pack weight {rows}x{cols}")
    from paper_2607_18839_amd import _lib
    rng = np.random.default_rng(rows + cols)
    w = _bits(rng, (rows, cols))
    assert _lib.hpd_packed_weight_bytes(rows, cols) == w.nbytes
    src, out = _dev(w), torch.full((rows, cols), -1, dtype=torch.int16, device="cuda")
    _lib.hpd_pack_weight(src.data_ptr(), rows, cols, out.data_ptr(), None)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint16)
    assert np.array_equal(got, packed_ref(w))
    assert np.array_equal(src.cpu().numpy().view(np.uint16), w)


@pytest.mark.parametrize("inter,hidden", [(16, 64), (48, 128), (8960, 1536)])
def test_pack_gate_up_bit_exact(inter, hidden):
    announce(f"pack gate/up {inter}x{hidden}")
    from paper_2607_18839_amd import _lib
    rng = np.random.default_rng(inter * 7 + hidden)
    g, u = _bits(rng, (inter, hidden)), _bits(rng, (inter, hidden))
    gd, ud = _dev(g), _dev(u)   # held until the kernel has run
    out = torch.full((2 * inter, hidden), -1, dtype=torch.int16, device="cuda")
    _lib.hpd_pack_gate_up(gd.data_ptr(), ud.data_ptr(), inter, hidden, out.data_ptr(), None)
    torch.cuda.synchronize()
    inter_rows = np.stack([g.reshape(-1, 16, hidden), u.reshape(-1, 16, hidden)], axis=1).reshape(2 * inter, hidden)
    assert np.array_equal(out.cpu().numpy().view(np.uint16), packed_ref(inter_rows))
