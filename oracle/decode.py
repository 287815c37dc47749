"""One branch-parallel decode step of the synthetic decoder stack, fp64.

Test infrastructure: see the package docstring.

The decoder is a pre-norm GQA transformer with RMSNorm and a SwiGLU MLP
(section "Overview", paragraph "LLM Decoder").  One step feeds the k_b new
tokens of every branch through every layer at once (Algorithm 1, the parallel
draft over the active pool).  For each layer l, with residual stream h
[T][hidden]:

  x = RMSNorm(h)                 y / sqrt(mean(y^2) + eps) * gamma
  [q | k | v] = x W_qkv^T        q: Hq heads, k and v: Hkv heads, head dim D
  k, v are stored in the bf16 cache: rounded to bf16 and written into the
  private rows L_b + j of branch b (the new tokens' slots)
  a = attention(q, shared KV of layer l, private KV of layer l)
  h = h + a W_o^T
  x = RMSNorm(h)
  h = h + (silu(x W_gate^T) * (x W_up^T)) W_down^T,  silu(u) = u / (1 + e^-u)

Optionally (a Qwen3-style decoder, the base the "Overview" section names):
right after the projection, q and k are RMS-normalised per head with their
own gains, then rotated by position (rotary embedding): dims i and i + 32 of
a head turn by the angle pos * theta^(-i / 32), pos = F_b + L_b + j the
token's position in its branch's sequence.

The step returns h after the last layer (no final norm, no LM head) and the
bf16 bits of the K/V rows it wrote.  Everything else is fp64.
"""

import numpy as np

from . import attention as attn_mod
from .plan import canonical_plan


def _bf16_value(x):
    """Round fp64 -> fp32 -> bf16 (nearest, ties to even); returns the fp64 value.

    bf16 keeps 8 significant bits: with x = m * 2^e, 0.5 <= |m| < 1, the
    rounded value is rint(m * 2^8) * 2^(e - 8) (np.rint rounds half to even).
    """
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)
    m, e = np.frexp(x32)
    return np.ldexp(np.rint(m * 256.0), e - 8)


def _bf16_bits_of_value(v):
    """Bit pattern of a value that is exactly representable in bf16."""
    f = np.asarray(v, dtype=np.float64).astype(np.float32)
    return (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def _bits_value(bits):
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def rms_norm(y, eps, gamma=None):
    r = y / np.sqrt(np.mean(y * y, axis=-1, keepdims=True) + eps)
    return r if gamma is None else r * gamma


def rope(x, pos, theta):
    """Rotary position embedding of the last axis (2 * half values) at
    positions pos (one per entry of the first axis): dims i and i + half turn
    by the angle pos * theta^(-i / half)."""
    half = x.shape[-1] // 2
    ang = np.asarray(pos, np.float64)[:, None] * float(theta) ** (-np.arange(half) / half)[None, :]
    shape = (ang.shape[0],) + (1,) * (x.ndim - 2) + (half,)
    c, s = np.cos(ang).reshape(shape), np.sin(ang).reshape(shape)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def qwen3_qk(inp, l, q, k, visible):
    """Qwen3-style attention inputs of layer l (identity when the inputs carry
    no q_norm / k_norm / rope_theta): per-head RMSNorm of q and k with their
    gains, then the rotary embedding at position visible - 1."""
    qn, kn = getattr(inp, "q_norm", None), getattr(inp, "k_norm", None)
    theta = float(getattr(inp, "rope_theta", 0.0) or 0.0)
    if qn is not None:
        q = rms_norm(q, inp.rms_eps, _bits_value(qn[l]))
    if kn is not None:
        k = rms_norm(k, inp.rms_eps, _bits_value(kn[l]))
    if theta > 0:
        pos = np.asarray(visible, np.float64) - 1
        q, k = rope(q, pos, theta), rope(k, pos, theta)
    return q, k


def silu(u):
    return u / (1.0 + np.exp(-u))


def decode_step(inp, num_layers=None):
    """Run the step on ``workloads.DecodeInputs`` (an optional ``fork_len``
    attribute gives per-branch fork points, section "Layout-Coordinated
    Parallel Decoding": a branch sees its page's prefix up to its fork).

    Returns (h_out [T][hidden] fp64, new_k, new_v) where new_k[l] and
    new_v[l] are uint16 arrays [T][Hkv][D] with the bf16 bits the step writes
    into layer l's private cache (token t = j-th new token of branch b goes to
    private row priv_row[b] + L_b + j).
    """
    Lyr = inp.num_layers if num_layers is None else num_layers
    Hq, Hkv, D = inp.num_q_heads, inp.num_kv_heads, inp.head_dim
    fork = getattr(inp, "fork_len", None)   # per-branch fork points; None = the whole prefix
    plan = canonical_plan(inp.prefix_len, inp.branch_page, inp.num_new, inp.past_len, fork)
    T = plan["T"]
    dest = (plan["priv_row"][plan["token_branch"]] +
            np.asarray(inp.past_len, np.int64)[plan["token_branch"]] + plan["token_j"])
    st = dict(prefix_len=inp.prefix_len, branch_page=inp.branch_page,
              num_new=inp.num_new, past_len=inp.past_len, fork_len=fork)
    h = np.asarray(inp.hidden_in, dtype=np.float64).copy()
    new_k, new_v = [], []
    for l in range(Lyr):
        Wqkv = _bits_value(inp.w_qkv[l])
        Wo = _bits_value(inp.w_o[l])
        Wg = _bits_value(inp.w_gate[l])
        Wu = _bits_value(inp.w_up[l])
        Wd = _bits_value(inp.w_down[l])
        x = rms_norm(h, inp.rms_eps)
        qkv = x @ Wqkv.T
        q = qkv[:, :Hq * D].reshape(T, Hq, D)
        q, k_raw = qwen3_qk(inp, l, q, qkv[:, Hq * D:(Hq + Hkv) * D].reshape(T, Hkv, D), plan["visible"])
        k_new = _bf16_value(k_raw)
        v_new = _bf16_value(qkv[:, (Hq + Hkv) * D:].reshape(T, Hkv, D))
        pk = _bits_value(inp.priv_k[l]).copy()
        pv = _bits_value(inp.priv_v[l]).copy()
        pk[dest] = k_new
        pv[dest] = v_new
        a, _ = attn_mod.attention(q, _bits_value(inp.shared_k[l]), _bits_value(inp.shared_v[l]),
                                  pk, pv, st, Hq, Hkv)
        h = h + a.reshape(T, Hq * D) @ Wo.T
        x = rms_norm(h, inp.rms_eps)
        h = h + (silu(x @ Wg.T) * (x @ Wu.T)) @ Wd.T
        new_k.append(_bf16_bits_of_value(k_new))
        new_v.append(_bf16_bits_of_value(v_new))
    return h, new_k, new_v
