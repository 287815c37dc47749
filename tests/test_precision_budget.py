"""Error budget of the decode step's 16-bit rounding points (CPU, fp64).

The GPU step rounds several intermediate values to 16 bits: q, the new K/V
rows (the cache dtype), the attention output, the attention-input norm, the
MLP-input norm and the SwiGLU product.  This test re-runs the 18-layer c4
step (section "Overview", paragraph "LLM Decoder") in fp64 with chosen
values rounded to bf16 or fp16, and measures the error each choice leaves in
the residual stream against the unrounded fp64 step.  It pins the choice the
kernels make: with bf16 MLP operands the step misses the 1e-2 max-abs bar,
and with fp16 MLP operands (the kernels' choice) it passes with room to spare.

The simulation is the decoder written with batched matrix products (fast
enough for the CPU suite); on a small stack, run without rounding, it is
checked against the oracle's decode step.
"""

import functools

import numpy as np
import pytest

from oracle.decode import decode_step
from workloads import get_config, make_decode_inputs

BAR = 1e-2


def _bits(b):
    return (np.asarray(b, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _bf16(x):
    """fp64 -> fp32 -> bf16, round to nearest even (8 significant bits)."""
    x32 = np.asarray(x, np.float64).astype(np.float32).astype(np.float64)
    m, e = np.frexp(x32)
    return np.ldexp(np.rint(m * 256.0), e - 8)


def _fp16(x):
    return np.asarray(x, np.float64).astype(np.float32).astype(np.float16).astype(np.float64)


ROUND = {None: lambda x: x, "bf16": _bf16, "fp16": _fp16}


def _rms(y, eps):
    return y / np.sqrt(np.mean(y * y, axis=-1, keepdims=True) + eps)


def simulate(inp, q=None, kv="bf16", attn_out=None, norm_attn=None, norm_mlp=None, swiglu=None):
    """The decode step in fp64 with each named value rounded as given
    (None = exact).  The new K/V rows are rounded to bf16 by default: the
    cache dtype is part of the step's definition, as in the oracle.
    Returns h after the last layer."""
    Hq, Hkv, D, Lyr = inp.num_q_heads, inp.num_kv_heads, inp.head_dim, inp.num_layers
    G = Hq // Hkv
    nb = len(inp.num_new)
    tq = np.concatenate([[0], np.cumsum(inp.num_new)])
    rp = np.concatenate([[0], np.cumsum(inp.past_len + inp.num_new)])
    ps = np.concatenate([[0], np.cumsum(inp.prefix_len)])
    h = inp.hidden_in.astype(np.float64)
    T = h.shape[0]
    for l in range(Lyr):
        x = ROUND[norm_attn](_rms(h, inp.rms_eps))
        qkv = x @ _bits(inp.w_qkv[l]).T
        qq = ROUND[q](qkv[:, :Hq * D]).reshape(T, Hkv, G, D)
        kn = ROUND[kv](qkv[:, Hq * D:(Hq + Hkv) * D]).reshape(T, Hkv, D)
        vn = ROUND[kv](qkv[:, (Hq + Hkv) * D:]).reshape(T, Hkv, D)
        sk, sv = _bits(inp.shared_k[l]), _bits(inp.shared_v[l])
        pk, pv = _bits(inp.priv_k[l]), _bits(inp.priv_v[l])
        a = np.zeros((T, Hkv, G, D))
        for b in range(nb):
            p, k, L = int(inp.branch_page[b]), int(inp.num_new[b]), int(inp.past_len[b])
            P = int(inp.prefix_len[p])
            K = np.concatenate([sk[ps[p]:ps[p] + P], pk[rp[b]:rp[b] + L], kn[tq[b]:tq[b + 1]]])   # [N, Hkv, D]
            V = np.concatenate([sv[ps[p]:ps[p] + P], pv[rp[b]:rp[b] + L], vn[tq[b]:tq[b + 1]]])
            Qb = qq[tq[b]:tq[b + 1]].transpose(1, 0, 2, 3).reshape(Hkv, k * G, D)            # [Hkv, kG, D]
            s = (Qb @ K.transpose(1, 2, 0)) / np.sqrt(D)                                      # [Hkv, kG, N]
            N = P + L + k
            j = np.repeat(np.arange(k), G)
            s = np.where(np.arange(N)[None, None, :] <= (P + L + j)[None, :, None], s, -np.inf)
            w = np.exp(s - s.max(axis=2, keepdims=True))
            w /= w.sum(axis=2, keepdims=True)
            a[tq[b]:tq[b + 1]] = (w @ V.transpose(1, 0, 2)).reshape(Hkv, k, G, D).transpose(1, 0, 2, 3)
        a = ROUND[attn_out](a.reshape(T, Hq * D))
        h = h + a @ _bits(inp.w_o[l]).T
        x = ROUND[norm_mlp](_rms(h, inp.rms_eps))
        g, u = x @ _bits(inp.w_gate[l]).T, x @ _bits(inp.w_up[l]).T
        m = ROUND[swiglu](g / (1.0 + np.exp(-g)) * u)
        h = h + m @ _bits(inp.w_down[l]).T
    return h


def test_simulation_without_rounding_is_the_oracle():
    cfg = get_config("c4", num_q_heads=4, num_kv_heads=2, num_pages=1, prefix=("fixed", 150),
                     layout=dict(k=1, past=("fixed", 20)), content_count=("fixed", 3), content_k=4,
                     content_past=("list", [0, 7, 30]),
                     model=dict(num_layers=3, hidden=128, intermediate=256, weight_std=0.05, rms_eps=1e-6))
    inp = make_decode_inputs(cfg, 4)
    ref, _, _ = decode_step(inp)
    assert np.abs(simulate(inp) - ref).max() <= 1e-10


@functools.lru_cache(maxsize=1)
def _c4():
    inp = make_decode_inputs("c4", 0)
    return inp, simulate(inp)


def _err(**rounding):
    inp, exact = _c4()
    return float(np.abs(simulate(inp, **rounding) - exact).max())


# what the kernels round to 16 bits besides the MLP operands and the cache
COMMON = dict(q="bf16", attn_out="bf16", norm_attn="bf16")


@pytest.mark.slow
def test_bf16_mlp_operands_miss_the_bar_and_fp16_meet_it():
    """c4, seed 0: the MLP-input norm or the SwiGLU product in bf16 each
    push the step past 1e-2 max abs (measured 1.6e-2 and 1.2e-2); with both
    in fp16 and everything else as the kernels round it, the step stays well
    inside the bar (2.5e-3).  q, the attention output and the
    attention-input norm cost about 4-6e-4 each."""
    assert _err(norm_mlp="bf16") > BAR
    assert _err(swiglu="bf16") > BAR
    assert _err(**COMMON, norm_mlp="fp16", swiglu="fp16") < BAR / 2
    # the other rounding points are small on their own
    for k in COMMON:
        assert _err(**{k: "bf16"}) < BAR / 10, k
