"""The seeded input generator: determinism, structure and rounding (CPU only)."""

import json
import os

import numpy as np
import pytest
import torch

from workloads import get_config, make_attn_batch, make_structure
from workloads.gen import bf16_bits_to_f64, f64_to_bf16_bits

from .golden.make_gen_hashes import attn_digests, decode_digests

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "gen_sha256.json")


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c5"])
def test_generator_bits_are_stable(name):
    want = json.load(open(GOLDEN))
    assert attn_digests(name, 0) == want[f"{name}/seed0"]


@pytest.mark.slow
def test_decode_generator_bits_are_stable():
    want = json.load(open(GOLDEN))
    assert decode_digests(0) == want["c4_1layer/seed0"]


def test_generator_rounding_matches_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(50000) * 10.0 ** rng.integers(-8, 8, 50000)
    bits = f64_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.float32).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    assert np.array_equal(bits, ref)
    assert np.array_equal(bf16_bits_to_f64(bits),
                          torch.from_numpy(x).to(torch.float32).to(torch.bfloat16).double().numpy())


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_structure_follows_the_workload_statement(name):
    cfg = get_config(name)
    for seed in range(5):
        st = make_structure(cfg, np.random.default_rng(seed))
        npg = cfg["num_pages"]
        assert st["prefix_len"].shape == (npg,)
        assert np.all(np.diff(st["branch_page"]) >= 0)
        for p in range(npg):
            on = st["branch_page"] == p
            lay = st["is_layout"][on]
            if cfg["layout"] is not None:
                assert lay[0] and not lay[1:].any()
                assert st["num_new"][on][0] == cfg["layout"]["k"]
            nc = int((~lay).sum())
            kind = cfg["content_count"]
            if kind[0] == "fixed":
                assert nc == kind[1]
            else:
                assert kind[1] <= nc <= kind[2]
            assert np.all(st["num_new"][on][~lay] == cfg["content_k"])
        spec = cfg["content_past"]
        L = st["past_len"][~st["is_layout"]]
        if spec[0] == "lognormal":
            assert L.min() >= spec[3] and L.max() <= spec[4]
        if spec[0] == "uniform":
            assert L.min() >= spec[1] and L.max() <= spec[2]
        if cfg["prefix"][0] == "uniform":
            assert st["prefix_len"].min() >= cfg["prefix"][1] and st["prefix_len"].max() <= cfg["prefix"][2]


def test_lognormal_median_is_128():
    cfg = get_config("c3", content_count=("fixed", 20000))
    st = make_structure(cfg, np.random.default_rng(0))
    L = st["past_len"][~st["is_layout"]]
    assert abs(np.median(L) - 128) <= 3


def test_packing_shapes():
    b = make_attn_batch("c2", 0)
    T = int(b.num_new.sum())
    assert b.q.shape == (T, 16, 64) and b.q.dtype == np.uint16
    assert b.shared_k.shape == (1024, 2, 64)
    assert b.priv_k.shape == (int((b.past_len + b.num_new).sum()), 2, 64)
    c1 = make_attn_batch("c1", 0)
    assert c1.q.dtype == np.float32 and list(c1.past_len) == [8, 16, 32, 32]


def test_fork_workload_extends_c3():
    """c3f is c3 (same structure and values for a seed) plus fork offsets:
    the layout branch sees the whole prefix, content branches a uniform
    integer in [1024, P]."""
    for seed in (0, 1):
        a, b = make_attn_batch("c3", seed), make_attn_batch("c3f", seed)
        assert a.fork_len is None
        for f in ("prefix_len", "branch_page", "num_new", "past_len", "q", "shared_k", "shared_v", "priv_k",
                  "priv_v"):
            assert np.array_equal(getattr(a, f), getattr(b, f)), f
        P = int(b.prefix_len[0])
        assert b.fork_len.dtype == np.int32 and b.fork_len.shape == (b.num_branches,)
        assert b.fork_len[b.is_layout].tolist() == [P]
        c = b.fork_len[~b.is_layout]
        assert c.min() >= 1024 and c.max() <= P and len(set(c.tolist())) > 20
