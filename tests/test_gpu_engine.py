"""GPU run of the continuous-batching loop (paper_2607_18839_amd.engine): the
host scheduler's batches drive the embedding lookup, the paged decode step
and P-MTP verification; every step is checked against the fp64 oracle on the
rows gathered from the K/V pools through the batch's own tables.

Forks are planted: the test replaces a parent's bonus token by the fork
token before the commit (random weights almost never produce it), so
children are spawned, admitted and decoded against their page's prefix."""

import types

import numpy as np
import pytest
import torch

from oracle.decode import decode_step
from oracle.pmtp import accepted, verify
from workloads import make_pmtp_inputs

from ._gpu import BF16_MAX_ABS, BF16_REL_L2, announce, errors, to_dev
from .test_gpu_decode import small_inputs
from .test_gpu_pmtp import _valid_argmax

pytestmark = pytest.mark.gpu

FORK, CHILD, EOS = 5, 6, 7


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _oracle_inputs(eng, inp, pm, batch):
    """The step's inputs for the oracle: the pools' rows gathered through the
    batch tables (the page's first P_p rows; each branch's L_b past rows and
    k_b zero rows), the embedding rows of the fed tokens, the weights."""
    from paper_2607_18839_amd.engine import pool_rows
    pg = batch["paged"]
    B = pg["block_rows"]
    k_all = [_bits(t) for t in eng.k_pool]
    v_all = [_bits(t) for t in eng.v_pool]

    def page_rows(p, n):
        r = np.arange(n, dtype=np.int64)
        return pg["blocks"][pg["page_block0"][p] + r // B].astype(np.int64) * B + r % B

    sh = np.concatenate([page_rows(p, int(P)) for p, P in enumerate(batch["prefix_len"])] or [np.zeros(0, np.int64)])
    nb = batch["num_branches"]
    pr_parts, new_mask = [], []
    for b in range(nb):
        L, k = int(batch["past_len"][b]), int(batch["num_new"][b])
        pr_parts.append(pool_rows(batch, b, 0, L + k))
        new_mask.append(np.r_[np.zeros(L, bool), np.ones(k, bool)])
    pr, new_mask = np.concatenate(pr_parts), np.concatenate(new_mask)
    sk = [a[sh] for a in k_all]
    sv = [a[sh] for a in v_all]
    pk = [np.where(new_mask[:, None, None], np.uint16(0), a[pr]) for a in k_all]
    pv = [np.where(new_mask[:, None, None], np.uint16(0), a[pr]) for a in v_all]
    emb = (pm.embed.astype(np.uint32) << 16).view(np.float32)
    ns = types.SimpleNamespace(
        num_q_heads=inp.num_q_heads, num_kv_heads=inp.num_kv_heads, head_dim=64, num_layers=inp.num_layers,
        hidden=inp.hidden, intermediate=inp.intermediate, rms_eps=inp.rms_eps,
        prefix_len=batch["prefix_len"].astype(np.int64), branch_page=batch["branch_page"].astype(np.int64),
        num_new=batch["num_new"].astype(np.int64), past_len=batch["past_len"].astype(np.int64),
        fork_len=batch["fork_len"].astype(np.int64), hidden_in=emb[batch["tokens_in"]],
        shared_k=sk, shared_v=sv, priv_k=pk, priv_v=pv,
        w_qkv=inp.w_qkv, w_o=inp.w_o, w_gate=inp.w_gate, w_up=inp.w_up, w_down=inp.w_down)
    return ns, pr[new_mask]


def _engine(inp, pm, num_blocks, max_active):
    from paper_2607_18839_amd.engine import Engine
    w = {k: [to_dev(a, "bf16") for a in getattr(inp, k)] for k in ("w_qkv", "w_o", "w_gate", "w_up", "w_down")}
    pw = {k: to_dev(getattr(pm, k), "bf16") for k in ("lm_head", "embed", "w_draft_gate", "w_draft_up",
                                                       "w_draft_down")}
    return Engine(w, pw, inp.hidden, inp.intermediate, inp.num_q_heads, inp.num_kv_heads,
                  dict(num_blocks=num_blocks, block_rows=64, kv_threshold=1.0, window=3, max_active=max_active,
                       fork_token=FORK, child_token=CHILD, eos_token=EOS), rms_eps=inp.rms_eps)


def _inputs():
    inp = small_inputs(0)
    pm = make_pmtp_inputs(inp.hidden, 1024, 128, 0.05, 0)
    # the embedding rows are the step's hidden input: give them the decode
    # workloads' N(0, 1) scale, the regime the parity bars are stated for
    # (at 0.05 the bf16 roundings of the layer updates dominate the output)
    from workloads.gen import f64_to_bf16_bits
    pm.embed = f64_to_bf16_bits(np.random.default_rng([0, 21]).standard_normal(pm.embed.shape))
    return inp, pm


def _checker(eng, inp, pm, seen, plant_at):
    """The per-step hook: every check against the oracle, then the planted forks."""
    W_lm = (pm.lm_head.astype(np.uint32) << 16).view(np.float32).astype(np.float64)

    def check(batch):
        T = batch["num_tokens"]
        # the embedding lookup is exact
        emb = (pm.embed.astype(np.uint32) << 16).view(np.float32)
        h_in = eng._buf["h_in"][:T * inp.hidden].view(T, inp.hidden).cpu().numpy()
        assert np.array_equal(h_in, emb[batch["tokens_in"]])
        ns, new_rows = _oracle_inputs(eng, inp, pm, batch)
        h_o, nk, nv = decode_step(ns)
        got = batch["hidden_out"][:T * inp.hidden].view(T, inp.hidden).double().cpu().numpy()
        mx, rl = errors(got, h_o)
        assert mx <= BF16_MAX_ABS and rl <= BF16_REL_L2, f"step {eng.steps}: max abs {mx:.3e}, rel L2 {rl:.3e}"
        seen["worst"] = (max(seen["worst"][0], mx), max(seen["worst"][1], rl))
        for l in range(inp.num_layers):   # the appended rows landed at the pool rows of the tables
            for pool, want in ((eng.k_pool[l], nk[l]), (eng.v_pool[l], nv[l])):
                g = _bits(pool)[new_rows]
                gv = (g.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
                wv = (want.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
                # bf16 values: a rounding flip costs one ulp (2^-5 at |v| < 4), the
                # decode tests' bar for appended rows
                cmx, crl = errors(gv, wv)
                assert cmx <= BF16_MAX_ABS * 5 and crl <= BF16_REL_L2, (l, cmx, crl)
        # verification: valid argmax tokens; acceptance on the GPU's own tokens
        _, _, _, _, logits = verify(got, batch["tokens_in"], batch["num_new"], None, W_lm)
        _valid_argmax(batch["verified"], logits, f"step {eng.steps} verified")
        q = 0
        for b, k in enumerate(batch["num_new"]):
            assert batch["n_acc"][b] == accepted(batch["verified"][q:q + k], batch["tokens_in"][q:q + k])
            q += k
        seen["children"] = max(seen["children"], int(np.sum(batch["fork_len"] > 0)))
        seen["prefill"] += int(np.sum(batch["prefill_to"] > batch["prefill_from"]))
        # plant a fork at the chosen page's parent bonus token
        if eng.steps in plant_at:
            p = plant_at[eng.steps]
            q = 0
            for b, k in enumerate(batch["num_new"]):
                if batch["branch_page"][b] == p and batch["fork_len"][b] == 0:
                    batch["verified"][q + batch["n_acc"][b]] = FORK   # emitted, and fed next
                    batch["draft_out"][b, 0] = FORK
                    seen["forks"] += 1
                q += k
        # a request admitted after a preemption resumes with its dropped rows to refill
        out = seen.setdefault("out", set())
        out.update(int(r) for r in batch["preempted"])
        for b, r in enumerate(batch["request"]):
            if int(r) in out and int(r) in set(int(a) for a in batch["admitted"]):
                seen["resumed"] += 1
                out.discard(int(r))
        seen["preempted"] += len(batch["preempted"])
    return check


def test_engine_steps_match_the_oracle_with_planted_forks():
    announce("engine: 2 pages, planted forks, oracle every step")
    inp, pm = _inputs()
    eng = _engine(inp, pm, num_blocks=48, max_active=4)
    eng.submit(150, 11, 14)
    eng.submit(90, 12, 14)
    seen = dict(children=0, forks=0, prefill=0, worst=(0.0, 0.0), preempted=0, resumed=0)
    eng.on_results = _checker(eng, inp, pm, seen, {1: 0, 3: 1, 4: 0})   # step -> page whose parent forks
    pages = []
    for _ in range(40):
        b = eng.step()
        pages += eng.outputs()
        if b["num_branches"] == 0 and len(pages) == 2:
            break
    print(f"engine: {eng.steps} steps, worst max abs {seen['worst'][0]:.2e}, rel L2 {seen['worst'][1]:.2e}, "
          f"forks {seen['forks']}, children in a step {seen['children']}")
    assert seen["forks"] >= 2 and seen["children"] >= 1 and seen["prefill"] >= 2
    assert sorted(p for p, _ in pages) == [0, 1]
    assert eng.sched.counts() == dict(waiting=0, active=0, free_blocks=48)


def test_engine_preempts_and_resumes_in_a_tight_pool():
    """8 blocks of 64 rows for three pages (prompts 100, 80 and 60 rows, up
    to 60 tokens each, a fork planted on the first page): growing requests
    preempt the youngest, whose dropped rows are refilled when it resumes;
    every step still matches the oracle and every page is output."""
    announce("engine: tight pool, preemption and resume, oracle every step")
    inp, pm = _inputs()
    eng = _engine(inp, pm, num_blocks=8, max_active=8)
    for prompt, tok in ((100, 11), (80, 12), (60, 13)):
        eng.submit(prompt, tok, 60)
    seen = dict(children=0, forks=0, prefill=0, worst=(0.0, 0.0), preempted=0, resumed=0)
    eng.on_results = _checker(eng, inp, pm, seen, {2: 0})
    pages = []
    for _ in range(400):
        b = eng.step()
        pages += eng.outputs()
        if b["num_branches"] == 0 and len(pages) == 3:
            break
    print(f"engine (tight pool): {eng.steps} steps, preempted {seen['preempted']}, resumed {seen['resumed']}, "
          f"worst max abs {seen['worst'][0]:.2e}")
    assert seen["preempted"] >= 1 and seen["resumed"] >= 1 and seen["forks"] >= 1
    assert sorted(p for p, _ in pages) == [0, 1, 2]
    assert eng.sched.counts() == dict(waiting=0, active=0, free_blocks=8)
