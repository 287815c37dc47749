"""Helpers of the GPU parity tests: move workload arrays to the device and
call the library through the C ABI (via the torch wrappers)."""

import sys

import numpy as np
import torch

from paper_2607_18839_amd.torch_api import BranchAttention

# Parity bars for bf16 inputs with fp32 accumulation (the workload statement).
BF16_MAX_ABS, BF16_REL_L2 = 1e-2, 5e-3
# fp32 inputs: fp32 products and sums; exp2 within 1e-7 relative.  The bar
# leaves two orders of magnitude over the expected ~1e-7 relative error.
F32_MAX_ABS, F32_REL_L2 = 2e-5, 1e-5
LSE_ABS = 1e-3


def announce(msg):
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def to_dev(a, dtype, device="cuda"):
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


def run_batch(b, out_dtype=None, fork_len=None, prefix_row=None, priv_row=None,
              shared_k=None, shared_v=None, priv_k=None, priv_v=None, with_lse=True, paged=None):
    """Runs one attention layer of a workload batch on the GPU.
    Returns (O float64 numpy [T][Hq][D], lse numpy [T][Hq])."""
    tdt = torch.bfloat16 if b.dtype == "bf16" else torch.float32
    odt = tdt if out_dtype is None else out_dtype
    layer = BranchAttention(b.num_q_heads, b.num_kv_heads, b.prefix_len, b.branch_page, b.num_new,
                            b.past_len, dtype=tdt, out_dtype=odt, fork_len=fork_len,
                            prefix_row=prefix_row, priv_row=priv_row, paged=paged)
    q = to_dev(b.q, b.dtype)
    sk = shared_k if shared_k is not None else to_dev(b.shared_k, b.dtype)
    sv = shared_v if shared_v is not None else to_dev(b.shared_v, b.dtype)
    pk = priv_k if priv_k is not None else to_dev(b.priv_k, b.dtype)
    pv = priv_v if priv_v is not None else to_dev(b.priv_v, b.dtype)
    lse = torch.empty((layer.T, b.num_q_heads), dtype=torch.float32, device="cuda") if with_lse else None
    out = layer(q, sk, sv, pk, pv, lse=lse)
    torch.cuda.synchronize()
    return out.double().cpu().numpy(), (lse.cpu().numpy().astype(np.float64) if with_lse else None)


def errors(got, want):
    d = got - want
    return float(np.abs(d).max()), float(np.linalg.norm(d) / max(np.linalg.norm(want), 1e-300))


def assert_parity(got, want, dtype, what=""):
    mx, rl = errors(got, want)
    if dtype == "bf16":
        assert mx <= BF16_MAX_ABS and rl <= BF16_REL_L2, f"{what}: max abs {mx:.3e}, rel L2 {rl:.3e}"
    else:
        assert mx <= F32_MAX_ABS and rl <= F32_REL_L2, f"{what}: max abs {mx:.3e}, rel L2 {rl:.3e}"
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    return mx, rl


def bf16_value(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def assert_cache_rows(got_bits, want_bits, what=""):
    """Appended K/V rows against the oracle's bf16 rows.

    Both sides round a projection to bf16.  The GPU's fp32 projection of a
    bf16-rounded input differs from the oracle's fp64 one by about 1e-3 of
    the value, so the two roundings agree or land on neighbouring bf16
    values: the bar is one bf16 ulp at the largest magnitude present,
    2^(floor(log2 max|v|) - 7), and rel L2 <= 5e-3 over the rows.
    """
    got, want = bf16_value(got_bits), bf16_value(want_bits)
    assert np.all(np.isfinite(got)), f"{what}: non-finite cache row (a slot was not written)"
    top = float(np.abs(want).max())
    bar = 2.0 ** (np.floor(np.log2(top)) - 7) if top > 0 else 0.0
    mx, rl = errors(got, want)
    assert mx <= bar and rl <= BF16_REL_L2, f"{what}: max abs {mx:.3e} (bar {bar:.3e}), rel L2 {rl:.3e}"
    return mx, rl, float(np.mean(got_bits != want_bits))

