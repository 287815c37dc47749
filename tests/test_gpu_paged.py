"""GPU parity of paged K/V (rows through block tables built by hpd_kv_pool)
against the fp64 oracle on the gathered rows."""

import numpy as np
import pytest
import torch

from oracle.attention import attention_for_batch
from oracle.decode import decode_step
from oracle.paged import gather_packed
from paper_2607_18839_amd import _lib
from workloads import make_attn_batch
from workloads.gen import AttnBatch

from ._gpu import (LSE_ABS, BF16_MAX_ABS, BF16_REL_L2, announce, assert_cache_rows, assert_parity, errors,
                   run_batch, to_dev)
from .test_gpu_decode import c4_reference, small_inputs
from .test_kv_pool import _pool_layout

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _scatter(packed_rows, pool_rows, n_pool_rows, fill):
    """Pool array holding packed row i at pool row pool_rows[i] (test-side
    scatter; every other row is `fill`)."""
    out = np.full((n_pool_rows,) + packed_rows.shape[1:], fill, dtype=packed_rows.dtype)
    out[pool_rows] = packed_rows
    return out


def _pool_rows(st, pg):
    B = pg["block_rows"]
    seqs = [(pg["page_block0"][p], P) for p, P in enumerate(st["prefix_len"])]
    seqs += [(pg["branch_block0"][b], L + k) for b, (L, k) in enumerate(zip(st["past_len"], st["num_new"]))]
    rows = [np.asarray(pg["blocks"], np.int64)[f + np.arange(n) // B] * B + np.arange(n) % B for f, n in seqs]
    n_sh = len(st["prefix_len"])
    return np.concatenate(rows[:n_sh]), np.concatenate(rows[n_sh:])


@pytest.mark.parametrize("name,block_rows", [("c1", 64), ("c2", 128), ("c3", 64), ("c3f", 256), ("c5", 128)])
def test_paged_attention_parity(name, block_rows):
    announce(f"paged attention {name} block_rows {block_rows}")
    b = make_attn_batch(name, 2)
    st = dict(prefix_len=b.prefix_len, branch_page=b.branch_page, num_new=b.num_new, past_len=b.past_len,
              fork_len=b.fork_len)
    pool, pg = _pool_layout(st, block_rows, np.random.default_rng(4))
    n_pool = pg["num_blocks"] * block_rows
    sh_rows, pr_rows = _pool_rows(st, pg)
    nan = np.uint16(0x7FC0) if b.dtype == "bf16" else np.float32(np.nan)
    pools = [_scatter(getattr(b, f), r, n_pool, nan) for f, r in
             (("shared_k", sh_rows), ("shared_v", sh_rows), ("priv_k", pr_rows), ("priv_v", pr_rows))]
    O, lse = run_batch(b, fork_len=b.fork_len, paged=pg, shared_k=to_dev(pools[0], b.dtype),
                       shared_v=to_dev(pools[1], b.dtype), priv_k=to_dev(pools[2], b.dtype),
                       priv_v=to_dev(pools[3], b.dtype))
    sk, sv, pk, pv = gather_packed(*pools, st, pg)   # the oracle's own gather of the pool rows
    ref = AttnBatch(name=b.name, seed=b.seed, dtype=b.dtype, num_q_heads=b.num_q_heads,
                    num_kv_heads=b.num_kv_heads, head_dim=64, prefix_len=b.prefix_len, branch_page=b.branch_page,
                    num_new=b.num_new, past_len=b.past_len, is_layout=b.is_layout, q=b.q, shared_k=sk,
                    shared_v=sv, priv_k=pk, priv_v=pv, fork_len=b.fork_len)
    Oref, lref = attention_for_batch(ref)
    assert_parity(O, Oref, b.dtype, f"paged {name}")
    assert np.abs(lse - lref).max() <= LSE_ABS


def _paged_decode(inp, ref, nk, nv, block_rows, seed):
    """Decode step on paged K/V: the new K/V rows land in the branches' pool
    blocks (every other pool row keeps its bits) and the output matches the
    oracle."""
    from paper_2607_18839_amd.torch_api import DecodeStep
    st = dict(prefix_len=inp.prefix_len, branch_page=inp.branch_page, num_new=inp.num_new, past_len=inp.past_len)
    pool, pg = _pool_layout(st, block_rows, np.random.default_rng(seed))
    n_pool = pg["num_blocks"] * block_rows
    sh_rows, pr_rows = _pool_rows(st, pg)
    w = {k: [to_dev(a, "bf16") for a in getattr(inp, k)] for k in ("w_qkv", "w_o", "w_gate", "w_up", "w_down")}
    step = DecodeStep(inp.num_q_heads, inp.num_kv_heads, inp.prefix_len, inp.branch_page, inp.num_new,
                      inp.past_len, w, inp.hidden, inp.intermediate, inp.rms_eps, packed=True, paged=pg)
    fill = np.uint16(0x3F80)   # 1.0: rows outside the plan must keep it
    starts = np.concatenate([[0], np.cumsum(inp.past_len + inp.num_new)[:-1]])
    new = np.concatenate([np.arange(s + L, s + L + k) for s, L, k in zip(starts, inp.past_len, inp.num_new)])
    dest = pr_rows[new]

    def priv_pool(a):   # the slots the step must fill start as NaN
        out = _scatter(a, pr_rows, n_pool, fill)
        out[dest] = np.uint16(0x7FC0)
        return out
    sk = [to_dev(_scatter(a, sh_rows, n_pool, fill), "bf16") for a in inp.shared_k]
    sv = [to_dev(_scatter(a, sh_rows, n_pool, fill), "bf16") for a in inp.shared_v]
    pk = [to_dev(priv_pool(a), "bf16") for a in inp.priv_k]
    pv = [to_dev(priv_pool(a), "bf16") for a in inp.priv_v]
    h = step(torch.from_numpy(inp.hidden_in).cuda(), sk, sv, pk, pv)
    torch.cuda.synchronize()
    got = h.double().cpu().numpy()
    assert np.all(np.isfinite(got))
    mx, rl = errors(got, ref)
    back = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
    untouched = np.ones(n_pool, bool)
    untouched[dest] = False
    for l in range(inp.num_layers):
        got_k, got_v = back(pk[l]), back(pv[l])
        assert np.array_equal(got_k[untouched], priv_pool(inp.priv_k[l])[untouched])
        assert np.array_equal(got_v[untouched], priv_pool(inp.priv_v[l])[untouched])
        assert_cache_rows(got_k[dest], nk[l], f"layer {l} paged cache k rows")
        assert_cache_rows(got_v[dest], nv[l], f"layer {l} paged cache v rows")
    assert mx <= BF16_MAX_ABS and rl <= BF16_REL_L2, (mx, rl)
    return mx, rl


def test_paged_decode_step_parity():
    announce("paged decode small stack")
    inp = small_inputs(3)
    ref, nk, nv = decode_step(inp)
    _paged_decode(inp, ref, nk, nv, 64, 8)


def test_paged_decode_c4():
    """The c4 step (18 layers, 33 branches, 4096-token prefix) on paged K/V
    with 64-row blocks and a scrambled free list: the configuration
    the paged benchmark times; every branch and every appended row."""
    announce("paged decode c4, 64-row blocks")
    inp, (ref, nk, nv) = c4_reference()
    mx, rl = _paged_decode(inp, ref, nk, nv, 64, 11)
    print(f"paged c4: max abs {mx:.3e} rel L2 {rl:.3e}")
