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

from ._gpu import LSE_ABS, BF16_MAX_ABS, BF16_REL_L2, announce, assert_parity, errors, run_batch, to_dev
from .test_gpu_decode import small_inputs
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


def test_paged_decode_step_parity():
    """Decode step on paged K/V: the new K/V rows land in the branches' pool
    blocks (every other pool row keeps its bits) and the output matches the
    oracle."""
    announce("paged decode small stack")
    from paper_2607_18839_amd.torch_api import DecodeStep
    inp = small_inputs(3)
    st = dict(prefix_len=inp.prefix_len, branch_page=inp.branch_page, num_new=inp.num_new, past_len=inp.past_len)
    pool, pg = _pool_layout(st, 64, np.random.default_rng(8))
    n_pool = pg["num_blocks"] * 64
    sh_rows, pr_rows = _pool_rows(st, pg)
    w = {k: [to_dev(a, "bf16") for a in getattr(inp, k)] for k in ("w_qkv", "w_o", "w_gate", "w_up", "w_down")}
    step = DecodeStep(inp.num_q_heads, inp.num_kv_heads, inp.prefix_len, inp.branch_page, inp.num_new,
                      inp.past_len, w, inp.hidden, inp.intermediate, inp.rms_eps, packed=True, paged=pg)
    fill = np.uint16(0x3F80)   # 1.0: rows outside the plan must keep it
    sk = [to_dev(_scatter(a, sh_rows, n_pool, fill), "bf16") for a in inp.shared_k]
    sv = [to_dev(_scatter(a, sh_rows, n_pool, fill), "bf16") for a in inp.shared_v]
    pk = [to_dev(_scatter(a, pr_rows, n_pool, fill), "bf16") for a in inp.priv_k]
    pv = [to_dev(_scatter(a, pr_rows, n_pool, fill), "bf16") for a in inp.priv_v]
    h = step(torch.from_numpy(inp.hidden_in).cuda(), sk, sv, pk, pv)
    torch.cuda.synchronize()
    ref, nk, nv = decode_step(inp)
    mx, rl = errors(h.double().cpu().numpy(), ref)
    assert mx <= BF16_MAX_ABS and rl <= BF16_REL_L2, (mx, rl)
    back = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
    starts = np.concatenate([[0], np.cumsum(inp.past_len + inp.num_new)[:-1]])
    new = np.concatenate([np.arange(s + L, s + L + k) for s, L, k in zip(starts, inp.past_len, inp.num_new)])
    dest = pr_rows[new]
    untouched = np.ones(n_pool, bool)
    untouched[dest] = False
    val = lambda b: (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    for l in range(inp.num_layers):
        got_k, got_v = back(pk[l]), back(pv[l])
        want_k = _scatter(inp.priv_k[l], pr_rows, n_pool, fill)
        assert np.array_equal(got_k[untouched], want_k[untouched])
        for got, want in ((got_k[dest], nk[l]), (got_v[dest], nv[l])):
            mx, rl = errors(val(got), val(want))
            assert mx <= BF16_MAX_ABS * 5 and rl <= BF16_REL_L2
