"""Packed weight layout (hpd_pack_weight, hpd_pack_weight_f16,
hpd_pack_gate_up): bit-exact against a numpy permutation written from the
layout's definition and numpy's fp16 rounding."""

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


def to_f16_bits(b):
    """bf16 bit patterns -> fp16 bit patterns, round to nearest even (numpy's
    float32 -> float16 conversion, subnormals included)."""
    f = (b.astype(np.uint32) << 16).view(np.float32)
    with np.errstate(over="ignore"):
        return f.astype(np.float16).view(np.uint16)


def _weights(rng, shape):
    """Finite bf16 weights spanning fp16's normal and subnormal ranges."""
    mag = np.exp2(rng.uniform(-30, 8, size=shape)).astype(np.float32)
    f = np.where(rng.random(shape) < 0.5, -mag, mag).astype(np.float32)
    return (f.view(np.uint32) >> 16).astype(np.uint16)


@pytest.mark.parametrize("f16", [False, True], ids=["bf16", "f16"])
@pytest.mark.parametrize("rows,cols", [(32, 64), (64, 192), (1792, 3072), (8960, 1536)])
def test_pack_weight_bit_exact(rows, cols, f16):
    announce(f"pack weight {rows}x{cols} f16 {f16}")
    from paper_2607_18839_amd import _lib
    rng = np.random.default_rng(rows + cols)
    w = _weights(rng, (rows, cols)) if f16 else _bits(rng, (rows, cols))
    assert _lib.hpd_packed_weight_bytes(rows, cols) == w.nbytes
    src, out = _dev(w), torch.full((rows, cols), -1, dtype=torch.int16, device="cuda")
    (_lib.hpd_pack_weight_f16 if f16 else _lib.hpd_pack_weight)(src.data_ptr(), rows, cols, out.data_ptr(), None)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint16)
    assert np.array_equal(got, packed_ref(to_f16_bits(w) if f16 else w))
    assert np.array_equal(src.cpu().numpy().view(np.uint16), w)


@pytest.mark.parametrize("inter,hidden", [(16, 64), (48, 128), (8960, 1536)])
def test_pack_gate_up_bit_exact(inter, hidden):
    announce(f"pack gate/up {inter}x{hidden}")
    from paper_2607_18839_amd import _lib
    rng = np.random.default_rng(inter * 7 + hidden)
    g, u = _weights(rng, (inter, hidden)), _weights(rng, (inter, hidden))
    gd, ud = _dev(g), _dev(u)   # held until the kernel has run
    out = torch.full((2 * inter, hidden), -1, dtype=torch.int16, device="cuda")
    _lib.hpd_pack_gate_up(gd.data_ptr(), ud.data_ptr(), inter, hidden, out.data_ptr(), None)
    torch.cuda.synchronize()
    inter_rows = np.stack([g.reshape(-1, 16, hidden), u.reshape(-1, 16, hidden)], axis=1).reshape(2 * inter, hidden)
    assert np.array_equal(out.cpu().numpy().view(np.uint16), packed_ref(to_f16_bits(inter_rows)))
