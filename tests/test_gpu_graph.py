"""Graph capture of the library's launches (torch CUDAGraph = hipGraph).

Replays are interleaved with eager work and synchronisations, and every
replay is checked against the eager result bit for bit."""

import numpy as np
import pytest
import torch

from workloads import make_attn_batch

from ._gpu import announce, to_dev
from .test_gpu_decode import small_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _capture(fn):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return g


def test_attention_graph_replays():
    announce("graph: attention c2")
    from paper_2607_18839_amd.torch_api import BranchAttention
    b = make_attn_batch("c2", 3)
    layer = BranchAttention(b.num_q_heads, b.num_kv_heads, b.prefix_len, b.branch_page, b.num_new, b.past_len)
    ins = [to_dev(getattr(b, f), "bf16") for f in ("q", "shared_k", "shared_v", "priv_k", "priv_v")]
    eager = layer(*ins).clone()
    out = torch.empty_like(eager)
    g = _capture(lambda: layer(*ins, out=out))
    for r in range(4):
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        noise = torch.randn(1 << 20, device="cuda").sum()   # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {r} differs"
        assert torch.isfinite(noise)


@pytest.mark.parametrize("packed", [False, True], ids=["torch", "packed"])
def test_decode_graph_replays(packed):
    announce(f"graph: decode small stack, packed {packed}")
    from paper_2607_18839_amd.torch_api import DecodeStep
    inp = small_inputs(4, layers=2)
    w = {k: [to_dev(a, "bf16") for a in getattr(inp, k)] for k in ("w_qkv", "w_o", "w_gate", "w_up", "w_down")}
    step = DecodeStep(inp.num_q_heads, inp.num_kv_heads, inp.prefix_len, inp.branch_page, inp.num_new,
                      inp.past_len, w, inp.hidden, inp.intermediate, inp.rms_eps, packed=packed)
    sk = [to_dev(a, "bf16") for a in inp.shared_k]
    sv = [to_dev(a, "bf16") for a in inp.shared_v]
    pk = [to_dev(a, "bf16") for a in inp.priv_k]
    pv = [to_dev(a, "bf16") for a in inp.priv_v]
    h = torch.from_numpy(inp.hidden_in).cuda()
    eager = step(h, sk, sv, pk, pv).clone()
    eager_k = [t.clone() for t in pk]
    out = torch.empty_like(eager)
    starts = np.concatenate([[0], np.cumsum(inp.past_len + inp.num_new)[:-1]])
    dest = np.concatenate([np.arange(s + L, s + L + k) for s, L, k in zip(starts, inp.past_len, inp.num_new)])
    d = torch.from_numpy(dest).cuda()
    g = _capture(lambda: step(h, sk, sv, pk, pv, hidden_out=out))
    for r in range(4):
        out.fill_(float("nan"))
        for t in pk:          # clear the rows the step appends
            t[d] = 0
        torch.cuda.synchronize()
        g.replay()
        noise = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {r} differs"
        for l in range(len(pk)):
            assert torch.equal(pk[l], eager_k[l])
        assert torch.isfinite(noise)


def test_phase_isolation_is_bit_identical():
    """The phase-isolated launch order (shared-prefix items, then private
    items, as two launches) gives the same bits as the co-scheduled launch."""
    announce("phase isolation: attention c3 + decode small stack")
    from paper_2607_18839_amd import _lib
    from paper_2607_18839_amd.torch_api import BranchAttention, DecodeStep
    b = make_attn_batch("c3", 1)
    layer = BranchAttention(b.num_q_heads, b.num_kv_heads, b.prefix_len, b.branch_page, b.num_new, b.past_len)
    ins = [to_dev(getattr(b, f), "bf16") for f in ("q", "shared_k", "shared_v", "priv_k", "priv_v")]
    lse0 = torch.empty((layer.T, b.num_q_heads), dtype=torch.float32, device="cuda")
    lse1 = torch.empty_like(lse0)
    inp = small_inputs(6, layers=2)
    w = {k: [to_dev(a, "bf16") for a in getattr(inp, k)] for k in ("w_qkv", "w_o", "w_gate", "w_up", "w_down")}
    step = DecodeStep(inp.num_q_heads, inp.num_kv_heads, inp.prefix_len, inp.branch_page, inp.num_new,
                      inp.past_len, w, inp.hidden, inp.intermediate, inp.rms_eps, packed=True)
    sk = [to_dev(a, "bf16") for a in inp.shared_k]
    sv = [to_dev(a, "bf16") for a in inp.shared_v]
    h = torch.from_numpy(inp.hidden_in).cuda()
    outs = []
    try:
        for iso in (False, True):
            _lib.hpd_attn_phase_isolation(iso)
            o = layer(*ins, lse=lse1 if iso else lse0).clone()
            pk = [to_dev(a, "bf16") for a in inp.priv_k]
            pv = [to_dev(a, "bf16") for a in inp.priv_v]
            d = step(h, sk, sv, pk, pv).clone()
            torch.cuda.synchronize()
            outs.append((o, d, pk))
    finally:
        _lib.hpd_attn_phase_isolation(False)
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(lse0, lse1)
    assert torch.equal(outs[0][1], outs[1][1])
    assert all(torch.equal(x, y) for x, y in zip(outs[0][2], outs[1][2]))
