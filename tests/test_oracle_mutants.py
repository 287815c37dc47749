"""Plant plausible mistakes in copies of the oracle and check that the pins catch each.

The mistakes are planted on the CPU, in throw-away module copies built from
the oracle's source text; the oracle files themselves are never modified.
"""

import importlib.util
import os
import sys
import types

import pytest

from . import _pins

ORACLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")


def _load(name, src, deps):
    mod = types.ModuleType(f"oracle_mutant_{name}")
    mod.__dict__.update(deps)
    src = src.replace("from .plan import canonical_plan", "")
    src = src.replace("from . import attention as attn_mod", "")
    exec(compile(src, f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


def _modules(target, old, new):
    import oracle.attention as A
    import oracle.decode as Dm
    import oracle.plan as P
    srcs = {m: open(os.path.join(ORACLE, f"{m}.py")).read() for m in ("plan", "attention", "decode")}
    assert srcs[target].count(old) >= 1, f"mutation anchor not found: {old!r}"
    srcs[target] = srcs[target].replace(old, new, 1)
    plan = _load("plan", srcs["plan"], {})
    att = _load("attention", srcs["attention"], {"canonical_plan": plan.canonical_plan})
    dec = _load("decode", srcs["decode"], {"canonical_plan": plan.canonical_plan, "attn_mod": att})
    return att, plan, dec


MUTANTS = [
    ("attention", "z = scale * np.einsum", "z = np.einsum"),                       # dropped scale
    ("attention", "scale = 1.0 / np.sqrt(D)", "scale = 1.0 / D"),                   # wrong scale
    ("attention", "min(npv, L + j + 1)", "min(npv, L + j)"),                        # misses itself
    ("attention", "min(npv, L + j + 1)", "min(npv, L + j + 2)"),                    # sees a future draft
    ("attention", "min(npv, L + j + 1)", "min(npv, L + 1)"),                        # top-left causal
    ("attention", "head_to_kv = np.arange(Hq) // G", "head_to_kv = np.arange(Hq) % num_kv_heads"),
    ("attention", "s0 = int(plan[\"prefix_row\"][p])", "s0 = 0"),                 # wrong page prefix
    ("attention", "r0 = int(plan[\"priv_row\"][b])", "r0 = int(plan[\"q_row\"][b])"),
    ("attention", "Vcat = np.concatenate([Vs, Vp], axis=0)", "Vcat = np.concatenate([Ks, Kp], axis=0)"),
    ("attention", "vis[:, :ns] = True", "vis[:, :ns] = False"),                    # drops the prefix
    ("attention", "e / np.where(finite, s, 1.0)[:, :, None]", "e"),                # unnormalised
    ("attention", "m_safe + np.log(np.where(finite, s, 1.0))", "m_safe - np.log(np.where(finite, s, 1.0))"),
    ("attention", "np.exp(zm - m_safe[:, :, None])", "np.exp(zm + m_safe[:, :, None])"),
    ("attention", "coef = np.where(finite[None], w / np.where(finite, s, 1.0)[None], 0.0)",
                  "coef = np.where(finite[None], w, 0.0)"),                        # merge unnormalised
    ("attention", "lse = np.where(finite, m_safe + np.log(np.where(finite, s, 1.0)), -np.inf)\n    coef",
                  "lse = np.where(finite, m_safe + np.log(np.where(finite, s, 1.0)) + 1.0, -np.inf)\n    coef"),
    ("plan", "out[1:] = np.cumsum(x[:-1])", "out[:] = np.cumsum(x)"),            # inclusive scan
    ("plan", "priv_row = exclusive_cumsum(past_len + num_new)", "priv_row = exclusive_cumsum(past_len)"),
    ("plan", "fork[token_branch] + past_len[token_branch] + token_j + 1",
             "fork[token_branch] + past_len[token_branch] + token_j"),
    ("decode", "h = h + a.reshape(T, Hq * D) @ Wo.T", "h = a.reshape(T, Hq * D) @ Wo.T"),  # lost residual
    ("decode", "return u / (1.0 + np.exp(-u))", "return u / (1.0 + np.exp(u))"),      # silu sign
    ("decode", "np.mean(y * y, axis=-1, keepdims=True) + eps", "np.mean(y * y, axis=0, keepdims=True) + eps"),
    ("decode", "k_new = _bf16_value(k_raw)", "k_new = k_raw"),                    # cache not bf16
    ("decode", "return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)",
               "return np.concatenate([x1 * c + x2 * s, x2 * c - x1 * s], axis=-1)"),   # rotation sign
    ("decode", "float(theta) ** (-np.arange(half) / half)", "float(theta) ** (-np.arange(half) / (2 * half))"),
    ("decode", "pos = np.asarray(visible, np.float64) - 1", "pos = np.asarray(visible, np.float64)"),  # off by one
    ("decode", "v_new = _bf16_value(qkv[:, (Hq + Hkv) * D:].reshape(T, Hkv, D))",
               "v_new = _bf16_value(qkv[:, Hq * D:(Hq + Hkv) * D].reshape(T, Hkv, D))"),  # v := k
    ("decode", "(silu(x @ Wg.T) * (x @ Wu.T)) @ Wd.T", "(silu(x @ Wu.T) * (x @ Wg.T)) @ Wd.T"),  # gate/up swapped
    ("decode", "np.ldexp(np.rint(m * 256.0), e - 8)", "np.ldexp(np.floor(m * 256.0), e - 8)"),  # truncation
    # fork offsets ignored somewhere on the path (a branch must see only its
    # page's prefix up to its fork point)
    ("attention", "F = int(plan[\"fork\"][b])", "F = int(prefix_len[p])"),
    ("plan", "fork = np.asarray(fork_len, dtype=np.int64)", "fork = prefix_len[branch_page]"),
    ("plan", "visible[:] = fork[token_branch] + past_len[token_branch] + token_j + 1",
             "visible[:] = prefix_len[branch_page][token_branch] + past_len[token_branch] + token_j + 1"),
    ("plan", "fork = np.asarray(fork_len, dtype=np.int64)", "fork = np.asarray(fork_len, dtype=np.int64) - 1"),
    ("decode", "fork = getattr(inp, \"fork_len\", None)", "fork = None"),
]


@pytest.mark.parametrize("target,old,new", MUTANTS, ids=[f"{t}:{i}" for i, (t, _, _) in enumerate(MUTANTS)])
def test_pins_catch_mutant(target, old, new):
    att, plan, dec = _modules(target, old, new)
    pins = {"attention": _pins.ATTN_PINS + _pins.DECODE_PINS, "plan": _pins.PLAN_PINS + _pins.ATTN_PINS,
            "decode": _pins.DECODE_PINS}[target]
    caught = []
    for pin in pins:
        try:
            err = pin(att, plan, dec)
        except Exception as exc:  # a crash also counts as caught
            caught.append(f"{pin.__name__} raised {type(exc).__name__}")
            continue
        if not err <= _pins.TOLERANCE.get(pin, _pins.TOL):
            caught.append(pin.__name__)
    assert caught, f"no pin caught mutant {old!r} -> {new!r}"


def test_unmutated_copy_passes_all_pins():
    att, plan, dec = _modules("attention", "import numpy as np", "import numpy as np")
    for pin in _pins.ATTN_PINS + _pins.PLAN_PINS + _pins.DECODE_PINS:
        assert pin(att, plan, dec) <= _pins.TOLERANCE.get(pin, _pins.TOL), pin.__name__
