"""GPU parity of P-MTP verification and drafting (hpd_verify_draft_step).

The step's inputs are the decode step's GPU hidden states; the oracle works on
the same values.  Argmax decisions: a GPU token must be the oracle's argmax
or a valid one within rounding (its oracle logit within TOL_REL of the row's
spread of the maximum).  Integer logic (acceptance, bonus token, which state
seeds the drafts) must follow the GPU's own tokens exactly, and drafting is
checked teacher-forced: the oracle continues from the GPU's tokens."""

import numpy as np
import pytest
import torch

from oracle.pmtp import accepted, draft, verify
from workloads import make_decode_inputs, make_pmtp_inputs

from ._gpu import announce, to_dev
from .test_gpu_decode import small_inputs

pytestmark = pytest.mark.gpu

# bf16 LM-head input and bf16 / fp16 draft activations move logits by a few
# 2^-9 of their scale; a wrong token sits far below the maximum
TOL_REL = 2.0 ** -5


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _valid_argmax(tokens, logits, what):
    logits = np.asarray(logits)
    mx = logits.max(axis=-1)
    spread = logits.std(axis=-1)
    got = logits[np.arange(len(tokens)), tokens]
    bad = np.nonzero(got < mx - TOL_REL * spread)[0]
    assert len(bad) == 0, f"{what}: rows {bad[:8]} took a token {((mx - got) / spread)[bad][:8]} spreads below the max"
    return float(np.mean(tokens == logits.argmax(axis=-1)))


def _run(inp, pm, plant_seed, window=0):
    from paper_2607_18839_amd.torch_api import DecodeStep, VerifyDraft
    w = {k: [to_dev(a, "bf16") for a in getattr(inp, k)] for k in ("w_qkv", "w_o", "w_gate", "w_up", "w_down")}
    step = DecodeStep(inp.num_q_heads, inp.num_kv_heads, inp.prefix_len, inp.branch_page, inp.num_new,
                      inp.past_len, w, inp.hidden, inp.intermediate, inp.rms_eps, packed=True)
    pw = {k: to_dev(getattr(pm, k), "bf16") for k in ("lm_head", "embed", "w_draft_gate", "w_draft_up",
                                                       "w_draft_down")}
    vd = VerifyDraft(step, pw, window=window)
    sk = [to_dev(a, "bf16") for a in inp.shared_k]
    sv = [to_dev(a, "bf16") for a in inp.shared_v]
    pk = [to_dev(a, "bf16") for a in inp.priv_k]
    pv = [to_dev(a, "bf16") for a in inp.priv_v]
    hid = step(torch.from_numpy(inp.hidden_in).cuda(), sk, sv, pk, pv)
    torch.cuda.synchronize()
    h64 = hid.double().cpu().numpy()
    # plant drafts that the oracle's verification accepts for a chosen count
    lm = lambda a: (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    W_lm = lm(pm.lm_head)
    ver_o, _, _, _, _ = verify(h64, np.zeros(len(h64), np.int64), inp.num_new, None, W_lm)
    rng = np.random.default_rng(plant_seed)
    tokens = rng.integers(0, pm.vocab, size=len(h64)).astype(np.int64)
    q0 = np.concatenate([[0], np.cumsum(inp.num_new)[:-1]])
    planted = []
    for q, k in zip(q0, inp.num_new):
        a = int(rng.integers(0, k))
        for i in range(1, a + 1):
            tokens[q + i] = ver_o[q + i - 1]
        if a + 1 < k and tokens[q + a + 1] == ver_o[q + a]:
            tokens[q + a + 1] = (tokens[q + a + 1] + 1) % pm.vocab
        planted.append(a)
    tin = torch.from_numpy(tokens.astype(np.int32)).cuda()
    ver, n_acc, drafts = vd(hid, tin)
    torch.cuda.synchronize()
    return h64, tokens, np.array(planted), ver.cpu().numpy(), n_acc.cpu().numpy(), drafts.cpu().numpy()


def _check(inp, pm, plant_seed, window=0):
    h64, tokens, planted, ver, n_acc, drafts = _run(inp, pm, plant_seed, window)
    f64 = lambda a: (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    W_lm, E = f64(pm.lm_head), f64(pm.embed)
    Wg, Wu, Wd = f64(pm.w_draft_gate), f64(pm.w_draft_up), f64(pm.w_draft_down)
    ver_o, _, _, _, logits = verify(h64, tokens, inp.num_new, None, W_lm)
    agree = _valid_argmax(ver, logits, "verified")
    q0 = np.concatenate([[0], np.cumsum(inp.num_new)[:-1]])
    nb = len(inp.num_new)
    for b, (q, k) in enumerate(zip(q0, inp.num_new)):   # integer logic on the GPU's own tokens
        assert n_acc[b] == accepted(ver[q:q + k], tokens[q:q + k]), b
        assert drafts[b, 0] == ver[q + n_acc[b]], b
        if np.array_equal(ver[q:q + k], ver_o[q:q + k]):
            assert n_acc[b] == planted[b], b
    W = window or int(inp.num_new.max())   # every branch gets a window of W tokens
    seed = q0 + n_acc
    forced = drafts[:, 1:W].astype(np.int64)
    _, step_logits = draft(h64[seed], drafts[:, 0].astype(np.int64), W - 1, E, Wg, Wu, Wd, None, W_lm,
                           inp.rms_eps, forced=forced)
    for s, lg in enumerate(step_logits):
        need = np.arange(nb)
        _valid_argmax(forced[need, s], lg[need], f"draft {s + 1}")
    print(f"verified tokens equal to the oracle argmax: {agree:.3f}; n_acc {n_acc.tolist()}")
    return agree


@pytest.mark.parametrize("seed", [0, 1])
def test_verify_draft_small(seed):
    announce(f"pmtp small seed {seed}")
    inp = small_inputs(seed)
    pm = make_pmtp_inputs(inp.hidden, 2048, 256, 0.05, seed)
    assert _check(inp, pm, seed) > 0.9


def test_verify_draft_window_longer_than_the_step():
    """window = 7 > every k_b: each branch, including those that fed one
    token, gets the bonus token and 6 drafts."""
    announce("pmtp small window 7")
    inp = small_inputs(2)
    pm = make_pmtp_inputs(inp.hidden, 1024, 128, 0.05, 2)
    assert _check(inp, pm, 2, window=7) > 0.9


def test_verify_draft_many_tokens():
    """T = 1 + 48 * 4 = 193 tokens (7 token tiles): the LM head runs two
    token-tile groups per weight slice, the second with a padding tile."""
    announce("pmtp 193 tokens")
    from workloads import get_config, make_decode_inputs
    cfg = get_config("c4", num_q_heads=4, num_kv_heads=2, num_pages=1, prefix=("fixed", 200),
                     layout=dict(k=1, past=("fixed", 30)), content_count=("fixed", 48), content_k=4,
                     content_past=("lognormal", 20.0, 1.0, 0, 80),
                     model=dict(num_layers=1, hidden=256, intermediate=384, weight_std=0.05, rms_eps=1e-6))
    inp = make_decode_inputs(cfg, 3)
    assert int(inp.num_new.sum()) == 193
    pm = make_pmtp_inputs(inp.hidden, 2048, 128, 0.05, 3)
    assert _check(inp, pm, 3) > 0.9


def test_verify_draft_c4_full_vocab():
    """c4 (18 layers, 33 branches) with the full 151,936-token vocabulary."""
    announce("pmtp c4 full vocab")
    inp = make_decode_inputs("c4", 0)
    from workloads import get_config
    c = get_config("c4")["pmtp"]
    pm = make_pmtp_inputs(inp.hidden, c["vocab"], c["draft_inner"], c["weight_std"], 0)
    assert _check(inp, pm, 0) > 0.9


def test_verify_draft_large_hidden_state():
    """Hidden states scaled by 2^15 (exact), past fp16's range: the draft
    input [f ; embed(t)] is written in fp16 times the power of two of its
    own norm factor and the draft GEMM divides it back out, so the drafts
    stay valid argmaxes of the oracle's logits."""
    announce("pmtp with hidden states beyond fp16 range")
    inp = small_inputs(1)
    inp.hidden_in = (inp.hidden_in * np.float32(2 ** 15)).astype(np.float32)
    pm = make_pmtp_inputs(inp.hidden, 2048, 256, 0.05, 1)
    assert _check(inp, pm, 1) > 0.9
