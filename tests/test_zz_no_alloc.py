"""hpd_branch_attn_step_noalloc (the entry point that allocates nothing)
against hpd_branch_attn_step on the same plans, through the C ABI.

Two calls in a row share the library's static scratch: the first with the
largest workload (c5, about 19 MB of scratch), then smaller ones (fp32 c1,
bf16 c2), so the second call runs on whatever the first left there.  The
results must be bit-identical to the workspace entry point's, which itself
is held to the oracle's bar.  A plan needing more scratch than the library
holds is refused before anything is enqueued.
"""

import numpy as np
import pytest
import torch

from oracle.attention import attention_for_batch
from paper_2607_18839_amd import _lib
from workloads import make_attn_batch

from ._gpu import LSE_ABS, announce, assert_parity, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _plan(b):
    dt = _lib.HPD_BF16 if b.dtype == "bf16" else _lib.HPD_F32
    return _lib.hpd_plan_create(b.num_q_heads, b.num_kv_heads, b.prefix_len, b.branch_page, b.num_new,
                                b.past_len, dtype=dt, out_dtype=dt, fork_len=b.fork_len)


def _tensors(b):
    t = {n: to_dev(getattr(b, n), b.dtype) for n in ("q", "shared_k", "shared_v", "priv_k", "priv_v")}
    odt = torch.bfloat16 if b.dtype == "bf16" else torch.float32
    T, Hq = b.num_tokens, b.num_q_heads
    out = [torch.full((T, Hq, 64), float("nan"), dtype=odt, device="cuda") for _ in range(2)]
    lse = [torch.full((T, Hq), float("nan"), dtype=torch.float32, device="cuda") for _ in range(2)]
    return t, out, lse


def _both(b):
    """Runs the workspace entry point and the allocation-free one on batch b."""
    plan = _plan(b)
    t, out, lse = _tensors(b)
    stream = torch.cuda.current_stream().cuda_stream
    ws = torch.empty(max(plan.workspace_bytes, 256), dtype=torch.uint8, device="cuda")
    _lib.hpd_plan_upload(plan, ws.data_ptr(), plan.workspace_bytes, stream)
    args = [t[n].data_ptr() for n in ("q", "shared_k", "shared_v", "priv_k", "priv_v")]
    _lib.hpd_branch_attn_step(plan, *args, out[0].data_ptr(), lse[0].data_ptr(), ws.data_ptr(),
                              plan.workspace_bytes, stream)
    _lib.hpd_branch_attn_step_noalloc(plan, *args, out[1].data_ptr(), lse[1].data_ptr(), stream)
    torch.cuda.synchronize()
    return plan, [o.double().cpu().numpy() for o in out], [l.double().cpu().numpy() for l in lse]


@pytest.mark.parametrize("seq", [("c5", "c1", "c2")], ids=["c5-then-c1-then-c2"])
def test_noalloc_matches_workspace_entry_point(seq):
    sizes = []
    for name in seq:
        announce(f"noalloc attention {name}")
        b = make_attn_batch(name, 0)
        plan, (o_ws, o_na), (l_ws, l_na) = _both(b)
        sizes.append(plan.workspace_bytes)
        assert plan.workspace_bytes <= _lib.HPD_NOALLOC_SCRATCH_BYTES
        assert np.array_equal(o_ws, o_na, equal_nan=False), f"{name}: outputs differ"
        assert np.array_equal(l_ws, l_na), f"{name}: lse differ"
        ref, lref = attention_for_batch(b)
        assert_parity(o_na, ref, b.dtype, f"noalloc {name}")
        assert np.abs(l_na - lref).max() <= LSE_ABS
    assert sizes[0] > sizes[1] and sizes[0] > sizes[2], sizes   # later calls are smaller


def test_noalloc_refuses_a_plan_beyond_its_scratch():
    """48 pages of 4096 prefix rows with 32 branches each: the plan's
    scratch exceeds the static array, and the call fails before any launch
    (the output keeps its fill)."""
    announce("noalloc refuses an oversized plan")
    npg, nbr = 48, 33
    st = dict(prefix_len=np.full(npg, 4096, np.int32), branch_page=np.repeat(np.arange(npg), nbr).astype(np.int32),
              num_new=np.tile([1] + [4] * (nbr - 1), npg).astype(np.int32),
              past_len=np.full(npg * nbr, 64, np.int32))
    plan = _lib.hpd_plan_create(16, 2, st["prefix_len"], st["branch_page"], st["num_new"], st["past_len"],
                                dtype=_lib.HPD_BF16, out_dtype=_lib.HPD_BF16)
    assert plan.workspace_bytes > _lib.HPD_NOALLOC_SCRATCH_BYTES
    T = int(st["num_new"].sum())
    q = torch.zeros((T, 16, 64), dtype=torch.bfloat16, device="cuda")
    sk = torch.zeros((npg * 4096, 2, 64), dtype=torch.bfloat16, device="cuda")
    pk = torch.zeros((int((st["past_len"] + st["num_new"]).sum()), 2, 64), dtype=torch.bfloat16, device="cuda")
    out = torch.full((T, 16, 64), 7.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(_lib.HpdError, match="scratch"):
        _lib.hpd_branch_attn_step_noalloc(plan, q.data_ptr(), sk.data_ptr(), sk.data_ptr(), pk.data_ptr(),
                                          pk.data_ptr(), out.data_ptr(), None,
                                          torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
