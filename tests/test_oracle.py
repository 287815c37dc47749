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


# ---------------------------------------------------------------- paged K/V rows

def test_paged_rows_identity_layout_is_the_packed_layout():
    """Blocks handed out in order to sequences laid end to end: the gather is
    the identity on the pool (closed form)."""
    from oracle.paged import gather_packed
    B = 64
    st = dict(prefix_len=np.array([130, 64]), past_len=np.array([3, 70]), num_new=np.array([4, 1]))
    # page 0: 3 blocks, page 1: 1 block, branch 0: 1 block, branch 1: 2 blocks
    paged = dict(block_rows=B, blocks=np.arange(7), page_block0=[0, 3], branch_block0=[4, 5])
    rng = np.random.default_rng(0)
    pool = rng.standard_normal((7 * B, 2, 8))
    sk, sv, pk, pv = gather_packed(pool, pool, pool, pool, st, paged)
    assert np.array_equal(sk[:130], pool[:130]) and np.array_equal(sk[130:], pool[192:256])
    assert np.array_equal(pk[:7], pool[256:263]) and np.array_equal(pk[7:], pool[320:391])


def test_paged_rows_match_a_per_row_loop_and_invert_a_scatter():
    """Brute force (pure-Python per-row address arithmetic) and a round trip:
    rows scattered into a scrambled pool by the test come back in order."""
    from oracle.paged import gather_packed, sequence_rows
    rng = np.random.default_rng(5)
    B = 64
    st = dict(prefix_len=np.array([200, 0, 65]), past_len=np.array([0, 130, 5, 63]),
              num_new=np.array([1, 4, 2, 1]))
    lens = list(st["prefix_len"]) + [L + k for L, k in zip(st["past_len"], st["num_new"])]
    nblk = [-(-int(n) // B) for n in lens]
    perm = rng.permutation(sum(nblk) + 5)[:sum(nblk)]
    first = np.concatenate([[0], np.cumsum(nblk)[:-1]])
    paged = dict(block_rows=B, blocks=perm, page_block0=first[:3], branch_block0=first[3:])
    for s, n in enumerate(lens):
        got = sequence_rows(perm, first[s], n, B)
        want = [int(perm[first[s] + i // B]) * B + i % B for i in range(int(n))]
        assert got.tolist() == want
    packed = rng.standard_normal((sum(int(n) for n in lens), 2, 8))
    pool = np.full(((sum(nblk) + 5) * B, 2, 8), np.nan)
    at = 0
    for s, n in enumerate(lens):          # scatter, written independently of the oracle
        for i in range(int(n)):
            pool[int(perm[first[s] + i // B]) * B + i % B] = packed[at + i]
        at += int(n)
    sk, sv, pk, pv = gather_packed(pool, pool, pool, pool, st, paged)
    n_sh = int(st["prefix_len"].sum())
    assert np.array_equal(sk, packed[:n_sh]) and np.array_equal(pk, packed[n_sh:])
