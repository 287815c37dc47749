"""GPU parity of the full decode step (hpd_decode_step) against the fp64 oracle."""

import numpy as np
import pytest
import torch

import functools

from oracle.decode import decode_step
from workloads import get_config, make_decode_inputs

from ._gpu import BF16_MAX_ABS, BF16_REL_L2, announce, assert_cache_rows, errors, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def run_decode(inp, canary=True, packed=False):
    """Runs hpd_decode_step on the inputs; returns (h_out, priv_k list, priv_v list) as numpy."""
    from paper_2607_18839_amd.torch_api import DecodeStep
    w = {k: [to_dev(a, "bf16") for a in getattr(inp, k)] for k in ("w_qkv", "w_o", "w_gate", "w_up", "w_down")}
    for k in ("q_norm", "k_norm"):   # Qwen3-style inputs, when the workload has them
        if getattr(inp, k, None) is not None:
            w[k] = [to_dev(a, "bf16") for a in getattr(inp, k)]
    step = DecodeStep(inp.num_q_heads, inp.num_kv_heads, inp.prefix_len, inp.branch_page, inp.num_new,
                      inp.past_len, w, inp.hidden, inp.intermediate, inp.rms_eps, packed=packed,
                      fork_len=getattr(inp, "fork_len", None), rope_theta=getattr(inp, "rope_theta", 0.0))
    sk = [to_dev(a, "bf16") for a in inp.shared_k]
    sv = [to_dev(a, "bf16") for a in inp.shared_v]
    pk_np = [a.copy() for a in inp.priv_k]
    pv_np = [a.copy() for a in inp.priv_v]
    if canary:   # the slots the step must fill start as NaN
        rows = np.concatenate([np.arange(r + L, r + L + k) for r, L, k in
                               zip(np.concatenate([[0], np.cumsum(inp.past_len + inp.num_new)[:-1]]),
                                   inp.past_len, inp.num_new)])
        for a in pk_np + pv_np:
            a[rows] = np.uint16(0x7FC0)
    pk = [to_dev(a, "bf16") for a in pk_np]
    pv = [to_dev(a, "bf16") for a in pv_np]
    h = torch.from_numpy(inp.hidden_in).cuda()
    out = step(h, sk, sv, pk, pv)
    torch.cuda.synchronize()
    back = lambda ts: [t.view(torch.int16).cpu().numpy().view(np.uint16) for t in ts]
    return out.double().cpu().numpy(), back(pk), back(pv)


def small_inputs(seed, layers=2):
    cfg = get_config("c4", num_q_heads=4, num_kv_heads=2, num_pages=1, prefix=("fixed", 300),
                     layout=dict(k=1, past=("fixed", 70)), content_count=("fixed", 5), content_k=4,
                     content_past=("lognormal", 40.0, 1.0, 0, 200),
                     model=dict(num_layers=layers, hidden=256, intermediate=384, weight_std=0.05, rms_eps=1e-6))
    return make_decode_inputs(cfg, seed)


def _check_cache(inp, pk, pv, nk, nv):
    """New rows match the oracle's bf16 K/V (one bf16 ulp, see
    assert_cache_rows); every other row is bit-identical to the input.
    Returns the largest fraction of appended values whose bits differ."""
    starts = np.concatenate([[0], np.cumsum(inp.past_len + inp.num_new)[:-1]])
    dest = np.concatenate([np.arange(r + L, r + L + k) for r, L, k in zip(starts, inp.past_len, inp.num_new)])
    keep = np.ones(pk[0].shape[0], bool)
    keep[dest] = False
    flips = 0.0
    for l in range(inp.num_layers):
        assert np.array_equal(pk[l][keep], inp.priv_k[l][keep]) and np.array_equal(pv[l][keep], inp.priv_v[l][keep])
        for nm, got, want in (("k", pk[l][dest], nk[l]), ("v", pv[l][dest], nv[l])):
            flips = max(flips, assert_cache_rows(got, want, f"layer {l} cache {nm} rows")[2])
    return flips


@functools.lru_cache(maxsize=1)
def c4_reference():
    """The c4 inputs (seed 0) and the oracle's whole step on them, computed
    once per test session (about 10-40 s of fp64 on the host)."""
    inp = make_decode_inputs("c4", 0)
    return inp, decode_step(inp)


@pytest.mark.parametrize("packed", [False, True], ids=["torch", "packed"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_small_stack(seed, packed):
    announce(f"decode small seed {seed} packed {packed}")
    inp = small_inputs(seed)
    h, pk, pv = run_decode(inp, packed=packed)
    ref, nk, nv = decode_step(inp)
    mx, rl = errors(h, ref)
    print(f"small stack seed {seed}: max abs {mx:.3e} rel L2 {rl:.3e}")
    assert np.all(np.isfinite(h))
    assert mx <= BF16_MAX_ABS and rl <= BF16_REL_L2, (mx, rl)
    _check_cache(inp, pk, pv, nk, nv)


@pytest.mark.parametrize("packed", [True, False], ids=["packed", "torch"])
def test_full_c4_all_branches(packed):
    """c4 at full size (18 layers, 33 branches, 4096-token prefix); with
    packed weights this is the configuration the benchmark times.  Every
    branch's output and every appended K/V row of every layer (NaN canaries
    in the slots the step must fill) against the oracle's whole step."""
    announce(f"decode c4 full, all branches and cache rows, packed {packed}")
    inp, (ref, nk, nv) = c4_reference()
    h, pk, pv = run_decode(inp, canary=True, packed=packed)
    assert np.all(np.isfinite(h))
    mx, rl = errors(h, ref)
    flips = _check_cache(inp, pk, pv, nk, nv)
    print(f"c4 all 33 branches, packed {packed}: max abs {mx:.3e} rel L2 {rl:.3e}; "
          f"cache rows: at most {100 * flips:.2f}% of values one bf16 ulp off")
    assert mx <= BF16_MAX_ABS and rl <= BF16_REL_L2, (mx, rl)


def test_decode_deterministic_and_hidden_alias():
    announce("decode determinism + in-place")
    inp = small_inputs(5, layers=3)
    h1, pk1, _ = run_decode(inp)
    h2, pk2, _ = run_decode(inp)
    assert np.array_equal(h1, h2) and all(np.array_equal(a, b) for a, b in zip(pk1, pk2))
    h3, pk3, _ = run_decode(inp, packed=True)
    h4, pk4, _ = run_decode(inp, packed=True)
    assert np.array_equal(h3, h4) and all(np.array_equal(a, b) for a, b in zip(pk3, pk4))


def qwen3_inputs(seed, layers=2, theta=1e4):
    cfg = get_config("c4", num_q_heads=4, num_kv_heads=2, num_pages=1, prefix=("fixed", 300),
                     layout=dict(k=1, past=("fixed", 70)), content_count=("fixed", 5), content_k=4,
                     content_past=("lognormal", 40.0, 1.0, 0, 200),
                     model=dict(num_layers=layers, hidden=256, intermediate=384, weight_std=0.05, rms_eps=1e-6,
                                qwen3=dict(rope_theta=theta, qk_norm=True)))
    return make_decode_inputs(cfg, seed)


@pytest.mark.parametrize("seed,packed", [(0, True), (1, True), (0, False)], ids=["packed0", "packed1", "torch0"])
def test_qwen3_small_stack(seed, packed):
    """Per-head QK norm and rotary embedding (base 10^4) on the small stack,
    with random fork points for the content branches on the second seed,
    with packed and with torch-layout weights."""
    announce(f"decode qwen3 small seed {seed} packed {packed}")
    inp = qwen3_inputs(seed)
    if seed == 1:
        rng = np.random.default_rng(9)
        P = int(inp.prefix_len[0])
        inp.fork_len = np.array([P] + [int(rng.integers(100, P + 1)) for _ in inp.num_new[1:]], np.int64)
    h, pk, pv = run_decode(inp, packed=packed)
    ref, nk, nv = decode_step(inp)
    mx, rl = errors(h, ref)
    print(f"qwen3 small seed {seed} packed {packed}: max abs {mx:.3e} rel L2 {rl:.3e}")
    assert mx <= BF16_MAX_ABS and rl <= BF16_REL_L2, (mx, rl)
    _check_cache(inp, pk, pv, nk, nv)


def test_qwen3_c4q_full_step():
    """c4q: the 18-layer c4 step with QK norm and rotary embedding (base 10^6)."""
    announce("decode c4q")
    inp = make_decode_inputs("c4q", 0)
    h, pk, pv = run_decode(inp, packed=True)
    ref, nk, nv = decode_step(inp)
    mx, rl = errors(h, ref)
    print(f"c4q: max abs {mx:.3e} rel L2 {rl:.3e}")
    assert mx <= BF16_MAX_ABS and rl <= BF16_REL_L2, (mx, rl)


@pytest.mark.parametrize("packed", [False, True], ids=["torch", "packed"])
def test_many_token_tiles(packed):
    """322 tokens (two pages of 40 content branches, k = 4): 11 token tiles,
    the last holding 2 tokens.  Each projection's token tiles start their K
    walks at different steps, and with more tiles than K steps per wave
    (QKV 2, down 3, gate/up 8 at hidden 512, intermediate 768) several tiles
    share a start; the whole step is checked against the oracle."""
    announce(f"decode 322 tokens, 11 token tiles, packed {packed}")
    cfg = get_config("c4", num_q_heads=4, num_kv_heads=2, num_pages=2, prefix=("fixed", 200),
                     layout=dict(k=1, past=("fixed", 40)), content_count=("fixed", 40), content_k=4,
                     content_past=("lognormal", 30.0, 1.0, 0, 150),
                     model=dict(num_layers=2, hidden=512, intermediate=768, weight_std=0.05, rms_eps=1e-6))
    inp = make_decode_inputs(cfg, 3)
    h, pk, pv = run_decode(inp, packed=packed)
    assert len(h) == 322
    ref, nk, nv = decode_step(inp)
    mx, rl = errors(h, ref)
    print(f"322 tokens, packed {packed}: max abs {mx:.3e} rel L2 {rl:.3e}")
    assert mx <= BF16_MAX_ABS and rl <= BF16_REL_L2, (mx, rl)
    _check_cache(inp, pk, pv, nk, nv)


@pytest.mark.parametrize("seed", [0, 1])
def test_small_stack_multipage(seed):
    """Three pages of ragged prefixes and branch counts (the planner's general
    work lists, not the single-page computed items), packed weights."""
    announce(f"decode small multipage seed {seed}")
    cfg = get_config("c4", num_q_heads=4, num_kv_heads=2, num_pages=3, prefix=("uniform", 64, 300),
                     layout=dict(k=1, past=("uniform", 0, 90)), content_count=("uniform", 2, 5), content_k=4,
                     content_past=("lognormal", 40.0, 1.0, 0, 200),
                     model=dict(num_layers=2, hidden=256, intermediate=384, weight_std=0.05, rms_eps=1e-6))
    inp = make_decode_inputs(cfg, seed)
    assert len(inp.prefix_len) == 3
    h, pk, pv = run_decode(inp, packed=True)
    ref, nk, nv = decode_step(inp)
    mx, rl = errors(h, ref)
    print(f"multipage seed {seed}: T {len(h)} max abs {mx:.3e} rel L2 {rl:.3e}")
    assert mx <= BF16_MAX_ABS and rl <= BF16_REL_L2, (mx, rl)
    _check_cache(inp, pk, pv, nk, nv)


@pytest.mark.parametrize("packed", [True, False], ids=["packed", "torch"])
def test_large_residual_stream_stays_in_fp16_range(packed):
    """hidden_in scaled by 2^15 (exact): |h * gamma| reaches about 1.3e5,
    beyond fp16's 65504, so an fp16 MLP input written unscaled would be
    inf.  The O projection writes it times the power of two of the token's
    attention-norm factor, and the gate/up projection divides by it (both
    exact), so the step matches the oracle.  At |h| < 2^17 the fp32 residual
    stream has an ulp of 2^-7 and each of the 4 residual adds may round by
    half of it.  So the update h_out - h_in is held to 1e-2 + 4 * 2^-8 max
    abs and 1e-2 rel L2."""
    announce(f"decode with a residual stream beyond fp16 range, packed {packed}")
    inp = small_inputs(4)
    inp.hidden_in = (inp.hidden_in * np.float32(2 ** 15)).astype(np.float32)
    assert np.abs(inp.hidden_in).max() > 65504 * 1.5
    h, pk, pv = run_decode(inp, packed=packed)
    ref, nk, nv = decode_step(inp)
    assert np.all(np.isfinite(h)), "non-finite output: the fp16 norm input overflowed"
    h_in = inp.hidden_in.astype(np.float64)
    mx, rl = errors(h - h_in, ref - h_in)
    print(f"large residual stream, packed {packed}: update max abs {mx:.3e} rel L2 {rl:.3e}")
    assert mx <= 1e-2 + 4 * 2.0 ** -8 and rl <= 1e-2, (mx, rl)
    _check_cache(inp, pk, pv, nk, nv)
