"""C ABI without a GPU: symbols, host planner bookkeeping and validation."""

import ctypes

import numpy as np
import pytest

from oracle.plan import canonical_plan
from paper_2607_18839_amd import _lib
from workloads import get_config, make_structure

from ._pins import tiny_structures


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_library_exports_every_declared_symbol(lib):
    names = _lib.declared_symbols()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
        assert n in _lib.SIGNATURES, n


def _structures():
    out = [("tiny%d" % i, st) for i, st in enumerate(tiny_structures())]
    for name in ("c1", "c2", "c3", "c5"):
        for seed in (0, 1, 2):
            out.append((f"{name}/{seed}", make_structure(get_config(name), np.random.default_rng(seed))))
    return out


def _plan(st, Hq=16, Hkv=2, **kw):
    return _lib.hpd_plan_create(Hq, Hkv, st["prefix_len"], st["branch_page"], st["num_new"],
                                st["past_len"], **kw)


@pytest.mark.parametrize("name,st", _structures(), ids=lambda x: x if isinstance(x, str) else "")
def test_bookkeeping_bit_exact_vs_oracle(name, st):
    info = _lib.hpd_plan_query(_plan(st))
    cp = canonical_plan(st["prefix_len"], st["branch_page"], st["num_new"], st["past_len"])
    assert info["T"] == cp["T"]
    for k in ("q_row", "priv_row", "prefix_row", "page_q_row", "page_T", "visible"):
        got = info[k].astype(np.int64)
        assert got.dtype == cp[k].dtype and np.array_equal(got, cp[k]), k
    assert info["priv_rows"] == cp["priv_rows_total"]
    assert info["shared_rows"] == cp["shared_rows_total"]


@pytest.mark.parametrize("name,st", _structures(), ids=lambda x: x if isinstance(x, str) else "")
@pytest.mark.parametrize("Hq,Hkv", [(16, 2), (8, 2), (4, 4)])
def test_work_lists_cover_every_key_once(name, st, Hq, Hkv):
    """Each (token, query head) row meets each visible shared key and each of
    its branch's private keys in exactly one work item, and each of its
    partial slots is written by exactly one item."""
    G = Hq // Hkv
    info = _lib.hpd_plan_query(_plan(st, Hq, Hkv))
    T = info["T"]
    P = st["prefix_len"].astype(np.int64)
    cp = canonical_plan(st["prefix_len"], st["branch_page"], st["num_new"], st["past_len"])
    slot_writes = np.zeros((info["num_partial_slots"], Hq), np.int64)
    shared_cov = [np.zeros((Hq, P[cp["token_branch"][t] * 0 + st["branch_page"][cp["token_branch"][t]]]), np.int64)
                  for t in range(T)]
    S, Pi = _lib.SI, _lib.PI
    # without fork offsets position t holds token t
    assert np.array_equal(info["pos_token"][:, 0], np.arange(T))
    for it in info["shared_items"]:
        p, g = it[S["page"]], it[S["kvh"]]
        assert it[S["page_q_row"]] == cp["page_q_row"][p] and it[S["prefix_row"]] == cp["prefix_row"][p]
        for r in range(it[S["row0"]], it[S["row0"]] + it[S["nrows"]]):
            t = cp["page_q_row"][p] + r // G
            h = g * G + r % G
            assert st["branch_page"][cp["token_branch"][t]] == p
            shared_cov[t][h, it[S["key0"]]:it[S["key1"]]] += 1
            first, cnt = info["token_slots"][t]
            assert 0 <= it[S["slot"]] < cnt
            slot_writes[first + it[S["slot"]], h] += 1
    priv_cov = [np.zeros((Hq, st["past_len"][cp["token_branch"][t]] + st["num_new"][cp["token_branch"][t]]), np.int64)
                for t in range(T)]
    for it in info["private_items"]:
        b, g = it[Pi["branch"]], it[Pi["kvh"]]
        assert it[Pi["priv_row"]] == cp["priv_row"][b] and it[Pi["q_row"]] == cp["q_row"][b]
        assert it[Pi["past"]] == st["past_len"][b] and it[Pi["num_new"]] == st["num_new"][b]
        for r in range(it[Pi["row0"]], it[Pi["row0"]] + it[Pi["nrows"]]):
            t = cp["q_row"][b] + r // G
            h = g * G + r % G
            priv_cov[t][h, it[Pi["key0"]]:it[Pi["key1"]]] += 1
            first, cnt = info["token_slots"][t]
            assert 0 <= it[Pi["slot"]] < cnt
            slot_writes[first + it[Pi["slot"]], h] += 1
    for t in range(T):
        assert np.all(shared_cov[t] == 1) and np.all(priv_cov[t] == 1)
    assert np.all(slot_writes == 1)
    first = info["token_slots"][:, 0]
    assert first[0] == 0 and np.all(first[1:] == first[:-1] + info["token_slots"][:-1, 1])


BAD = [
    (dict(num_kv_heads=3), "multiple"),
    (dict(head_dim=128), "head_dim"),
    (dict(num_new=[0, 4, 4]), "num_new"),
    (dict(num_new=[17, 4, 4]), "num_new"),
    (dict(past_len=[-1, 4, 4]), "past_len"),
    (dict(branch_page=[0, 1, 0], prefix_len=[8, 8]), "non-decreasing"),
    (dict(branch_page=[0, 0, 5]), "branch_page"),
    (dict(prefix_len=[-5]), "prefix_len"),
    (dict(fork_len=[9, 0, 0]), "fork_len"),
    (dict(fork_len=[-1, 0, 0]), "fork_len"),
    (dict(dtype=7), "dtype"),
    (dict(num_q_heads=128, num_kv_heads=2), "num_q_heads"),
    (dict(num_q_heads=64, num_kv_heads=1), "HPD_MAX_GROUP"),
    (dict(priv_row=[0, 5, -3]), "priv_row"),
    (dict(priv_row=[0, 5, 2 ** 31]), "2^31"),
    (dict(softmax_scale=float("nan")), "finite"),
]


@pytest.mark.parametrize("over,needle", BAD, ids=[n for _, n in BAD])
def test_validation_errors(over, needle):
    kw = dict(num_q_heads=16, num_kv_heads=2, prefix_len=[8], branch_page=[0, 0, 0],
              num_new=[1, 4, 4], past_len=[3, 0, 5])
    kw.update(over)
    with pytest.raises(_lib.HpdError) as e:
        _lib.hpd_plan_create(**kw)
    assert needle in str(e.value)
    assert e.value.status in (1, 2)


def test_null_arguments_are_rejected(lib):
    assert lib.hpd_plan_create(None, None, None) == 1
    assert lib.hpd_plan_query(None, None) == 1
    plan = _plan(tiny_structures()[0])
    assert lib.hpd_branch_attn_step(plan.handle, None, None, None, None, None, None, None, None, 0, None) == 1
    assert b"NULL" in lib.hpd_last_error_message()
    # a workspace that is too small is reported before anything is launched
    fake = ctypes.c_void_p(256)
    assert lib.hpd_branch_attn_step(plan.handle, fake, fake, fake, fake, fake, fake, None, fake, 16, None) == 3
    assert lib.hpd_status_string(3) == b"HPD_ERR_WORKSPACE_TOO_SMALL"
    assert lib.hpd_plan_upload(plan.handle, fake, 16, None) == 3


def test_custom_row_offsets_are_kept():
    st = tiny_structures()[1]
    pr = np.array([100, 7, 40], np.int64)
    vr = np.array([0, 30, 60, 90], np.int64)
    info = _lib.hpd_plan_query(_plan(st, 4, 2, prefix_row=pr, priv_row=vr))
    assert np.array_equal(info["prefix_row"], pr) and np.array_equal(info["priv_row"], vr)
    assert info["shared_rows"] == max(pr + st["prefix_len"])
    assert info["priv_rows"] == max(vr + st["past_len"] + st["num_new"])


def test_pack_entry_points_validate_before_launching(lib):
    assert _lib.hpd_packed_weight_bytes(32, 64) == 4096
    assert _lib.hpd_packed_weight_bytes(8960, 1536) == 8960 * 1536 * 2
    assert _lib.hpd_packed_weight_bytes(0, 64) == 0
    fake = ctypes.c_void_p(4096)
    assert lib.hpd_pack_weight(None, 32, 64, fake, None) == 1
    assert lib.hpd_pack_weight(fake, 48, 64, fake, None) == 1          # rows % 32
    assert lib.hpd_pack_weight(fake, 32, 96, fake, None) == 1          # cols % 64
    assert lib.hpd_pack_weight(ctypes.c_void_p(4098), 32, 64, fake, None) == 1   # alignment
    assert b"16-byte" in lib.hpd_last_error_message()
    assert lib.hpd_pack_gate_up(fake, None, 16, 64, fake, None) == 1
    assert lib.hpd_pack_gate_up(fake, fake, 24, 64, fake, None) == 1   # intermediate % 16
    assert b"intermediate" in lib.hpd_last_error_message()


def test_decode_step_checks_weight_format():
    st = tiny_structures()[1]
    plan = _plan(st, 4, 2)
    fake = 4096
    one = [fake]
    for fmt, w_up, status, needle in ((7, one, 1, "weight_format"), (0, [None], 1, "NULL weight"),
                                      (0, [fake + 2], 1, "16-byte aligned"),
                                      (1, [None], 3, "workspace too small")):
        model = _lib.model_desc(1, 256, 384, 1e-6, one, one, one, w_up, one, weight_format=fmt)
        with pytest.raises(_lib.HpdError) as e:
            _lib.hpd_decode_step(model, plan, fake, fake, one, one, one, one, 4096, 0)
        assert e.value.status == status and needle in str(e.value), str(e.value)


@pytest.mark.parametrize("name,st", _structures(), ids=lambda x: x if isinstance(x, str) else "")
@pytest.mark.parametrize("Hq,Hkv", [(16, 2), (12, 2), (4, 4)])
def test_single_page_items_follow_the_index_formula(name, st, Hq, Hkv):
    """For one page without fork offsets the kernels compute a shared item's
    fields from its index (kv head, split, row group nesting) instead of
    reading the table: the table must be exactly that formula."""
    if len(st["prefix_len"]) != 1 or st["prefix_len"][0] == 0:
        pytest.skip("not a single-page plan")
    G = Hq // Hkv
    info = _lib.hpd_plan_query(_plan(st, Hq, Hkv))
    items = info["shared_items"]
    S = _lib.SI
    rows = info["T"] * G
    groups = -(-rows // 128)
    split_keys = items[0][S["key1"]] - items[0][S["key0"]] if len(items) > 1 else st["prefix_len"][0]
    splits = len(items) // (Hkv * groups)
    assert len(items) == Hkv * splits * groups
    P = int(st["prefix_len"][0])
    for i, it in enumerate(items):
        rgi, rest = i % groups, i // groups
        s, g = rest % splits, rest // splits
        k0 = s * split_keys
        want = dict(page=0, kvh=g, row0=128 * rgi, nrows=min(128, rows - 128 * rgi), key0=k0,
                    key1=min(P, k0 + split_keys), slot=s, flags=0, prefix_row=info["prefix_row"][0],
                    page_q_row=0)
        for k, v in want.items():
            assert it[S[k]] == v, (i, k, it[S[k]], v)


@pytest.mark.parametrize("name,st", _structures(), ids=lambda x: x if isinstance(x, str) else "")
@pytest.mark.parametrize("Hq,Hkv", [(16, 2), (4, 4)])
def test_fork_work_lists_cover_visible_keys_once(name, st, Hq, Hkv):
    """With fork offsets: each (token, head) row meets each of its F_b visible
    shared keys in exactly one item, and each of its partial slots is written
    exactly once, a row writing a shared split's partial only when it sees
    the split's first key (the kernels' rule)."""
    G = Hq // Hkv
    rng = np.random.default_rng(len(st["num_new"]) * 7 + Hq)
    P_b = st["prefix_len"][st["branch_page"]]
    fork = np.array([rng.integers(0, P + 1) for P in P_b], np.int32)
    if len(fork) > 1:
        fork[0], fork[1] = 0, P_b[1]
    info = _lib.hpd_plan_query(_plan(st, Hq, Hkv, fork_len=fork))
    T = info["T"]
    cp = canonical_plan(st["prefix_len"], st["branch_page"], st["num_new"], st["past_len"], fork)
    tb = cp["token_branch"]
    S, Pi = _lib.SI, _lib.PI
    slot_writes = np.zeros((info["num_partial_slots"], Hq), np.int64)
    cov = [np.zeros((Hq, int(fork[tb[t]])), np.int64) for t in range(T)]
    pos = info["pos_token"]
    # each page's positions hold a permutation of its tokens, by descending
    # fork point (ties in token order), each with its own fork point
    for p in range(len(st["prefix_len"])):
        q0, n = cp["page_q_row"][p], cp["page_T"][p]
        toks = pos[q0:q0 + n, 0]
        assert sorted(toks) == list(range(q0, q0 + n))
        assert np.array_equal(pos[q0:q0 + n, 1], fork[tb[toks]])
        key = [(-int(fork[tb[t]]), int(t)) for t in toks]
        assert key == sorted(key)
    for it in info["shared_items"]:
        p, g, k0, k1 = it[S["page"]], it[S["kvh"]], it[S["key0"]], it[S["key1"]]
        assert k0 < k1
        rows = range(it[S["row0"]], it[S["row0"]] + it[S["nrows"]])
        # the item ends at its split's end or at the largest fork point of its rows
        max_f = max(int(pos[cp["page_q_row"][p] + r // G, 1]) for r in rows)
        assert k1 <= max_f and (k1 == max_f or k1 % 128 == 0 or k1 == st["prefix_len"][p])
        sorted_page = not np.array_equal(pos[cp["page_q_row"][p]:cp["page_q_row"][p] + cp["page_T"][p], 0],
                                         np.arange(cp["page_q_row"][p], cp["page_q_row"][p] + cp["page_T"][p]))
        assert bool(it[S["flags"]] & 2) == sorted_page
        for r in rows:
            t = int(pos[cp["page_q_row"][p] + r // G, 0])
            h = g * G + r % G
            F = int(fork[tb[t]])
            cov[t][h, k0:min(k1, F)] += 1
            if F > k0:
                first, cnt = info["token_slots"][t]
                assert 0 <= it[S["slot"]] < cnt
                slot_writes[first + it[S["slot"]], h] += 1
    for it in info["private_items"]:
        b, g = it[Pi["branch"]], it[Pi["kvh"]]
        for r in range(it[Pi["row0"]], it[Pi["row0"]] + it[Pi["nrows"]]):
            t = cp["q_row"][b] + r // G
            first, cnt = info["token_slots"][t]
            assert 0 <= it[Pi["slot"]] < cnt
            slot_writes[first + it[Pi["slot"]], g * G + r % G] += 1
    for t in range(T):
        assert np.all(cov[t] == 1), t
    assert np.all(slot_writes == 1)


@pytest.mark.timeout(60)
def test_plan_with_more_row_groups_than_the_item_target():
    """48 pages x 33 branches: even one key split per page gives 864 shared
    items, more than the planner's target of about one per CU, so growing the
    split cannot reach the target.  The planner must stop at one split per
    page (it once looped forever here) and still cover every (page, kv
    head, row group) prefix range [0, P_p) exactly once."""
    npg, nbr, G = 48, 33, 8
    rng = np.random.default_rng(3)
    st = dict(prefix_len=rng.integers(1024, 4097, npg).astype(np.int32),
              branch_page=np.repeat(np.arange(npg), nbr).astype(np.int32),
              num_new=np.tile([1] + [4] * (nbr - 1), npg).astype(np.int32),
              past_len=rng.integers(0, 300, npg * nbr).astype(np.int32))
    info = _lib.hpd_plan_query(_plan(st))
    S = _lib.SI
    spans = {}
    for it in info["shared_items"]:
        key = (it[S["page"]], it[S["kvh"]], it[S["row0"]])
        spans.setdefault(key, []).append((it[S["key0"]], it[S["key1"]]))
    page_T = np.bincount(st["branch_page"], weights=st["num_new"], minlength=npg).astype(int)
    assert len(spans) == sum(2 * -(-int(T) * G // 128) for T in page_T)
    for (p, g, r0), iv in spans.items():
        iv.sort()
        assert iv[0][0] == 0 and iv[-1][1] == st["prefix_len"][p]
        assert all(a[1] == b[0] for a, b in zip(iv, iv[1:])), (p, g, r0, iv)
    assert len(info["shared_items"]) == len(spans)    # one split per page


def test_embed_and_pmtp_entry_points_validate_before_launching(lib):
    """hpd_embed_tokens and hpd_verify_draft_step reject bad arguments on the
    host, before any launch (fake device addresses are never touched)."""
    fake = 4096
    assert lib.hpd_embed_tokens(None, 1024, 256, fake, 4, fake, None) == 1
    assert lib.hpd_embed_tokens(fake, 1024, 250, fake, 4, fake, None) == 1          # hidden % 4
    assert lib.hpd_embed_tokens(fake + 2, 1024, 256, fake, 4, fake, None) == 1     # 8-byte alignment
    assert lib.hpd_embed_tokens(fake, 1024, 256, fake, 4, fake + 4, None) == 1     # out 16-byte aligned
    assert b"hpd_embed_tokens" in lib.hpd_last_error_message()
    st = tiny_structures()[1]
    plan = _plan(st, 4, 2)
    one = [fake]
    model = _lib.model_desc(1, 256, 384, 1e-6, one, one, one, one, one, weight_format=1)
    ok = dict(vocab=1024, draft_inner=128, lm_head=fake, g_final=None, embed=fake, w_draft_gate_up=fake,
              w_draft_down=fake, window=0)
    cases = [(dict(window=HPD_MAX_K + 1), "window"), (dict(window=-1), "window"),
             (dict(vocab=1000), "multiples of 128"), (dict(lm_head=fake + 8), "misaligned"),
             (dict(embed=None), "misaligned")]
    for over, needle in cases:
        d = dict(ok, **over)
        desc = _lib.hpd_pmtp_desc(d["vocab"], d["draft_inner"], d["lm_head"], d["g_final"], d["embed"],
                                  d["w_draft_gate_up"], d["w_draft_down"], d["window"])
        with pytest.raises(_lib.HpdError) as e:
            _lib.hpd_verify_draft_step(model, desc, plan, fake, fake, fake, fake, fake, fake, 1 << 30)
        assert needle in str(e.value), (over, str(e.value))
    small = _lib.model_desc(1, 128, 384, 1e-6, one, one, one, one, one, weight_format=1)   # hidden % 256
    desc = _lib.hpd_pmtp_desc(1024, 128, fake, None, fake, fake, fake, 0)
    with pytest.raises(_lib.HpdError) as e:
        _lib.hpd_verify_draft_step(small, desc, plan, fake, fake, fake, fake, fake, fake, 1 << 30)
    assert "multiple of 256" in str(e.value)


def test_qwen3_options_are_validated():
    st = tiny_structures()[1]
    plan = _plan(st, 4, 2)
    fake = 4096
    one = [fake]
    for kw, needle in ((dict(rope_theta=-1.0), "rope_theta"), (dict(rope_theta=float("nan")), "rope_theta"),
                       (dict(q_norm=[None]), "q_norm"), (dict(k_norm=[fake + 2]), "k_norm")):
        model = _lib.model_desc(1, 256, 384, 1e-6, one, one, one, one, one, weight_format=1, **kw)
        with pytest.raises(_lib.HpdError) as e:
            _lib.hpd_decode_step(model, plan, fake, fake, one, one, one, one, 4096, 1 << 30)
        assert needle in str(e.value), (kw, str(e.value))


HPD_MAX_K = _lib.HPD_MAX_K
