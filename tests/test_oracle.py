"""The fp64 oracle against its pins (CPU only)."""

import numpy as np
import pytest

import oracle
from oracle import attention as att, decode as dec, plan as pln

from . import _pins


@pytest.mark.parametrize("pin", _pins.ATTN_PINS + _pins.PLAN_PINS + _pins.DECODE_PINS,
                         ids=lambda f: f.__name__)
def test_pin(pin):
    err = pin(att, pln, dec)
    assert err <= _pins.TOLERANCE.get(pin, _pins.TOL), f"{pin.__name__}: error {err}"


def test_bf16_rounding_matches_torch():
    """The oracle's own bf16 rounding (used for the K/V cache writes) equals
    torch's fp32 -> bf16 conversion, including ties and carries."""
    import torch
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000),
                        # exact ties: bf16 values plus half an ulp
                        (np.arange(1, 2000) * 2.0 ** -7 + 2.0 ** -9),
                        (np.arange(1, 2000) * 2.0 ** -7 + 3 * 2.0 ** -9),
                        -(np.arange(1, 2000) * 2.0 ** -7 + 2.0 ** -9),
                        np.array([0.0, 1.0, -2.0, 255.5, 1.0 - 2.0 ** -10])])
    mine = dec._bf16_value(x)
    ref = torch.from_numpy(x).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(mine, ref)
    bits = dec._bf16_bits_of_value(mine)
    assert np.array_equal(dec._bits_value(bits), mine)


def test_oracle_header_says_test_infrastructure():
    assert "TEST INFRASTRUCTURE" in oracle.__doc__
