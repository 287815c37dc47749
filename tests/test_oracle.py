"""The fp64 oracle against its pins (CPU only)."""

import numpy as np
import pytest

import oracle
from oracle import attention as att, decode as dec, plan as pln

from . import _pins


@pytest.mark.parametrize("pin", _pins.ATTN_PINS + _pins.PLAN_PINS + _pins.DECODE_PINS,
                         ids=lambda f: f.__name__)
def test_pin(pin):
    err = pin(att, pln, dec)
    assert err <= _pins.TOLERANCE.get(pin, _pins.TOL), f"{pin.__name__}: error {err}"


def test_bf16_rounding_matches_torch():
    """The oracle's own bf16 rounding (used for the K/V cache writes) equals
    torch's fp32 -> bf16 conversion, including ties and carries."""
    import torch
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000),
                        # exact ties: bf16 values plus half an ulp
                        (np.arange(1, 2000) * 2.0 ** -7 + 2.0 ** -9),
                        (np.arange(1, 2000) * 2.0 ** -7 + 3 * 2.0 ** -9),
                        -(np.arange(1, 2000) * 2.0 ** -7 + 2.0 ** -9),
                        np.array([0.0, 1.0, -2.0, 255.5, 1.0 - 2.0 ** -10])])
    mine = dec._bf16_value(x)
    ref = torch.from_numpy(x).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(mine, ref)
    bits = dec._bf16_bits_of_value(mine)
    assert np.array_equal(dec._bits_value(bits), mine)


def test_oracle_header_says_test_infrastructure():
    assert "TEST INFRASTRUCTURE" in oracle.__doc__


# ---------------------------------------------------------------- paged K/V rows

def test_paged_rows_identity_layout_is_the_packed_layout():
    """Blocks handed out in order to sequences laid end to end: the gather is
    the identity on the pool (closed form)."""
    from oracle.paged import gather_packed
    B = 64
    st = dict(prefix_len=np.array([130, 64]), past_len=np.array([3, 70]), num_new=np.array([4, 1]))
    # page 0: 3 blocks, page 1: 1 block, branch 0: 1 block, branch 1: 2 blocks
    paged = dict(block_rows=B, blocks=np.arange(7), page_block0=[0, 3], branch_block0=[4, 5])
    rng = np.random.default_rng(0)
    pool = rng.standard_normal((7 * B, 2, 8))
    sk, sv, pk, pv = gather_packed(pool, pool, pool, pool, st, paged)
    assert np.array_equal(sk[:130], pool[:130]) and np.array_equal(sk[130:], pool[192:256])
    assert np.array_equal(pk[:7], pool[256:263]) and np.array_equal(pk[7:], pool[320:391])


def test_paged_rows_match_a_per_row_loop_and_invert_a_scatter():
    """Brute force (pure-Python per-row address arithmetic) and a round trip:
    rows scattered into a scrambled pool by the test come back in order."""
    from oracle.paged import gather_packed, sequence_rows
    rng = np.random.default_rng(5)
    B = 64
    st = dict(prefix_len=np.array([200, 0, 65]), past_len=np.array([0, 130, 5, 63]),
              num_new=np.array([1, 4, 2, 1]))
    lens = list(st["prefix_len"]) + [L + k for L, k in zip(st["past_len"], st["num_new"])]
    nblk = [-(-int(n) // B) for n in lens]
    perm = rng.permutation(sum(nblk) + 5)[:sum(nblk)]
    first = np.concatenate([[0], np.cumsum(nblk)[:-1]])
    paged = dict(block_rows=B, blocks=perm, page_block0=first[:3], branch_block0=first[3:])
    for s, n in enumerate(lens):
        got = sequence_rows(perm, first[s], n, B)
        want = [int(perm[first[s] + i // B]) * B + i % B for i in range(int(n))]
        assert got.tolist() == want
    packed = rng.standard_normal((sum(int(n) for n in lens), 2, 8))
    pool = np.full(((sum(nblk) + 5) * B, 2, 8), np.nan)
    at = 0
    for s, n in enumerate(lens):          # scatter, written independently of the oracle
        for i in range(int(n)):
            pool[int(perm[first[s] + i // B]) * B + i % B] = packed[at + i]
        at += int(n)
    sk, sv, pk, pv = gather_packed(pool, pool, pool, pool, st, paged)
    n_sh = int(st["prefix_len"].sum())
    assert np.array_equal(sk, packed[:n_sh]) and np.array_equal(pk, packed[n_sh:])


# ---------------------------------------------------------------- P-MTP

def test_pmtp_argmax_ties_go_to_the_smallest_id():
    from oracle.pmtp import argmax_first
    z = np.array([[1.0, 3.0, 3.0, -1.0], [0.0, 0.0, 0.0, 0.0], [-2.0, -1.0, -3.0, -1.0]])
    assert argmax_first(z).tolist() == [1, 0, 1]


def test_pmtp_acceptance_matches_its_definition_by_brute_force():
    """n_acc = the largest n such that drafts 1..n all equal the verified token
    one position earlier (brute force over every n)."""
    from oracle.pmtp import accepted
    rng = np.random.default_rng(0)
    for _ in range(500):
        k = int(rng.integers(1, 8))
        fed = rng.integers(0, 3, size=k)
        ver = rng.integers(0, 3, size=k)
        want = max(n for n in range(k) if all(ver[i - 1] == fed[i] for i in range(1, n + 1)))
        assert accepted(ver, fed) == want


def test_pmtp_verify_closed_form():
    """Unit-vector LM head: the argmax at a position is the coordinate where
    its hidden state peaks; planted drafts are accepted up to the first plant
    that disagrees."""
    from oracle.pmtp import verify
    V, H = 16, 8
    w_lm = np.zeros((V, H))
    w_lm[np.arange(H) * 2, np.arange(H)] = 1.0          # token 2c reads coordinate c
    num_new = np.array([4, 1, 3])
    peak = np.array([3, 5, 1, 0, 7, 2, 2, 6])            # per position
    hidden = np.full((8, H), 0.01) + np.eye(H)[peak] * 4.0
    tokens_in = np.array([9, 6, 10, 5, 3, 1, 4, 0])      # branch 0: drafts 6, 10 verified, 5 not
    ver, n_acc, bonus, seed, _ = verify(hidden, tokens_in, num_new, None, w_lm)
    assert ver.tolist() == (2 * peak).tolist()
    assert n_acc.tolist() == [2, 0, 1] and bonus.tolist() == [2, 14, 4] and seed.tolist() == [2, 4, 6]


def test_pmtp_draft_without_mlp_repeats_the_bonus_position():
    """A zero down projection leaves the draft state unchanged, so every
    drafted token is the LM head argmax of the seed state (closed form)."""
    from oracle.pmtp import argmax_first, draft, lm_logits
    rng = np.random.default_rng(1)
    V, H, I = 32, 16, 8
    f0 = rng.standard_normal((3, H))
    w_lm = rng.standard_normal((V, H))
    toks, logits = draft(f0, np.array([1, 2, 3]), 3, rng.standard_normal((V, H)), rng.standard_normal((I, 2 * H)),
                         rng.standard_normal((I, 2 * H)), np.zeros((H, I)), None, w_lm, 1e-6)
    base = argmax_first(lm_logits(f0, None, w_lm))
    assert all(np.array_equal(toks[:, s], base) for s in range(3))


def test_pmtp_draft_mlp_matches_torch():
    """One draft advance against torch's own RMSNorm and SiLU in fp64 (library
    routines)."""
    import torch
    from oracle.pmtp import draft_mlp
    rng = np.random.default_rng(2)
    V, H, I = 20, 16, 24
    f = rng.standard_normal((5, H))
    tok = rng.integers(0, V, size=5)
    E, Wg, Wu, Wd = (rng.standard_normal(s) for s in ((V, H), (I, 2 * H), (I, 2 * H), (H, I)))
    got = draft_mlp(f, tok, E, Wg, Wu, Wd, 1e-6)
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    d = torch.cat([t(f), t(E)[torch.from_numpy(tok)]], dim=-1)
    x = torch.nn.functional.rms_norm(d, (2 * H,), eps=1e-6)
    want = t(f) + (torch.nn.functional.silu(x @ t(Wg).T) * (x @ t(Wu).T)) @ t(Wd).T
    assert np.allclose(got, want.numpy(), rtol=1e-12, atol=1e-12)


def test_pmtp_lm_input_rounding_is_bf16():
    """The LM head's input rounding equals the generator's integer bf16
    rounding (round to nearest even on the bit pattern)."""
    from oracle.pmtp import lm_logits
    from workloads.gen import bf16_bits_to_f64, f64_to_bf16_bits
    rng = np.random.default_rng(3)
    h = rng.standard_normal((4, 64)) * 3
    g = rng.standard_normal(64)
    eye = np.eye(64)
    got = lm_logits(h, g, eye)
    want = bf16_bits_to_f64(f64_to_bf16_bits(h * g))
    assert np.array_equal(got, want)


# ---------------------------------------------------------------- Qwen3-style attention inputs

def test_qk_norm_matches_transformers_qwen3_rmsnorm():
    """The per-head q / k norm against transformers' Qwen3RMSNorm (library;
    it normalises in fp32, hence the tolerance)."""
    import torch
    from transformers.models.qwen3.modeling_qwen3 import Qwen3RMSNorm
    from oracle.decode import rms_norm
    rng = np.random.default_rng(5)
    x = rng.standard_normal((7, 3, 64)) * 2.0
    g = 1 + 0.1 * rng.standard_normal(64)
    m = Qwen3RMSNorm(64, eps=1e-6).double()
    with torch.no_grad():
        m.weight.copy_(torch.from_numpy(g))
        want = m(torch.from_numpy(x)).numpy()
    assert np.abs(rms_norm(x, 1e-6, g) - want).max() < 1e-5


def test_rope_matches_transformers_qwen3_rotary_embedding():
    """The rotary embedding against transformers' Qwen3RotaryEmbedding and
    apply_rotary_pos_emb (library; fp32 angles there, hence the tolerance)."""
    import torch
    from transformers import Qwen3Config
    from transformers.models.qwen3.modeling_qwen3 import Qwen3RotaryEmbedding, apply_rotary_pos_emb
    from oracle.decode import rope
    cfg = Qwen3Config(head_dim=64, hidden_size=1024, num_attention_heads=16, num_key_value_heads=2,
                      max_position_embeddings=8192, rope_theta=1e6)
    pos = np.array([0, 1, 5, 100, 2047])
    cos, sin = Qwen3RotaryEmbedding(cfg)(torch.zeros(1, len(pos), 64), torch.from_numpy(pos)[None])
    rng = np.random.default_rng(6)
    q, k = rng.standard_normal((5, 3, 64)), rng.standard_normal((5, 2, 64))
    qo, ko = apply_rotary_pos_emb(torch.from_numpy(q).permute(1, 0, 2)[None].float(),
                                  torch.from_numpy(k).permute(1, 0, 2)[None].float(), cos, sin)
    assert np.abs(qo[0].permute(1, 0, 2).double().numpy() - rope(q, pos, 1e6)).max() < 1e-4
    assert np.abs(ko[0].permute(1, 0, 2).double().numpy() - rope(k, pos, 1e6)).max() < 1e-4


def test_rope_scores_depend_only_on_the_position_difference():
    """<rope(q, m), rope(k, n)> = <rope(q, m - n), k> per head (closed form of
    a rotation), rope(x, 0) = x, and norms are kept."""
    from oracle.decode import rope
    rng = np.random.default_rng(7)
    q, k = rng.standard_normal((1, 64)), rng.standard_normal((1, 64))
    for m, n in ((5, 3), (4000, 17), (123, 123), (0, 900)):
        lhs = np.sum(rope(q, [m], 1e6) * rope(k, [n], 1e6))
        rhs = np.sum(rope(q, [m - n], 1e6) * k)
        assert abs(lhs - rhs) < 1e-9 * (1 + abs(rhs))
    x = rng.standard_normal((3, 2, 64))
    assert np.allclose(rope(x, [0, 0, 0], 1e4), x, rtol=0, atol=0)
    y = rope(x, [1, 70, 3000], 1e4)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)


def test_qwen3_options_off_leave_the_step_unchanged():
    """rope_theta = 0 and no gains: the step equals the plain one bit for bit."""
    from oracle.decode import decode_step
    from tests.test_gpu_decode import small_inputs
    inp = small_inputs(0, layers=1)
    h0, k0, _ = decode_step(inp)
    inp.rope_theta = 0.0
    h1, k1, _ = decode_step(inp)
    assert np.array_equal(h0, h1) and all(np.array_equal(a, b) for a, b in zip(k0, k1))
