"""Host paged-KV block manager (hpd_kv_pool) and paged plans, on the CPU."""

import numpy as np
import pytest

from oracle.plan import canonical_plan
from paper_2607_18839_amd import _lib
from workloads import get_config, make_structure


def test_reserve_truncate_release_account_for_every_block():
    pool = _lib.KvPool(10, 64)
    a = pool.new()
    pool.reserve(a, 1)
    assert pool.info(a) == dict(len=1, num_blocks=1, parent=-1, fork_len=0)
    pool.reserve(a, 128)
    assert pool.info(a)["num_blocks"] == 2 and pool.free_blocks() == 8
    pool.reserve(a, 129)
    assert pool.info(a)["num_blocks"] == 3
    pool.truncate(a, 64)   # rollback: whole blocks past the new length return
    assert pool.info(a)["num_blocks"] == 1 and pool.free_blocks() == 9
    pool.truncate(a, 0)
    assert pool.info(a)["num_blocks"] == 0 and pool.free_blocks() == 10
    pool.release(a)
    with pytest.raises(_lib.HpdError):
        pool.info(a)


def test_exhaustion_changes_nothing():
    pool = _lib.KvPool(4, 128)
    a, b = pool.new(), pool.new()
    pool.reserve(a, 300)                   # 3 blocks
    before = (pool.free_blocks(), pool.blocks(a).tolist())
    with pytest.raises(_lib.HpdError) as e:
        pool.reserve(b, 257)               # needs 3, 1 free
    assert e.value.status == 6 and "HPD_ERR_OUT_OF_BLOCKS" in str(e.value)
    assert (pool.free_blocks(), pool.blocks(a).tolist()) == before and pool.info(b)["num_blocks"] == 0
    pool.reserve(b, 128)                   # exactly the last block
    assert pool.free_blocks() == 0
    with pytest.raises(_lib.HpdError):
        pool.reserve(a, 385)


def test_fork_is_zero_copy_and_keeps_the_prefix_alive():
    pool = _lib.KvPool(16, 64)
    root = pool.new()
    pool.reserve(root, 200)                # 4 blocks
    prefix = pool.blocks(root).tolist()
    kids = [pool.new(root, f) for f in (0, 64, 200)]
    assert pool.free_blocks() == 12        # forking copies nothing
    for k in kids:
        pool.reserve(k, 70)                # private rows only: 2 blocks each
    assert pool.free_blocks() == 6
    with pytest.raises(_lib.HpdError):
        pool.truncate(root, 150)           # a branch sees 200 rows
    with pytest.raises(_lib.HpdError):
        pool.new(kids[0], 0)               # branches of branches are not sequences here
    with pytest.raises(_lib.HpdError):
        pool.new(root, 201)                # beyond the root's length
    pool.release(root)                     # kept while branches see it
    assert pool.free_blocks() == 6
    with pytest.raises(_lib.HpdError):
        pool.new(root, 0)
    pool.release(kids[0])
    pool.release(kids[2])                  # the 2 private blocks each, and the root
    assert pool.free_blocks() == 13        # blocks past the last fork (64 rows: 1 kept)
    pool.release(kids[1])                  # last branch: the prefix blocks return too
    assert pool.free_blocks() == 16
    r2 = pool.new()
    pool.reserve(r2, 64 * 16)
    assert sorted(pool.blocks(r2).tolist()) == list(range(16))
    assert set(prefix) <= set(pool.blocks(r2).tolist())


def test_random_operations_match_a_reference_model():
    """Random reserve / truncate / fork / release against a plain Python model
    of the block accounting: every block is owned by exactly one sequence or
    free, at every step."""
    rng = np.random.default_rng(3)
    B, NB = 64, 40
    pool = _lib.KvPool(NB, B)
    model = {}   # seq -> dict(len, parent, fork, live)
    for step in range(600):
        live = [s for s, m in model.items() if m["live"]]
        roots = [s for s in live if model[s]["parent"] == -1]
        op = rng.integers(0, 5)
        if op == 0 or not live:
            if roots and rng.random() < 0.6:
                r = int(rng.choice(roots))
                f = int(rng.integers(0, model[r]["len"] + 1))
                s = pool.new(r, f)
                model[s] = dict(len=0, parent=r, fork=f, live=True)
            else:
                s = pool.new()
                model[s] = dict(len=0, parent=-1, fork=0, live=True)
        elif op in (1, 2):
            s = int(rng.choice(live))
            n = model[s]["len"] + int(rng.integers(0, 300))
            free = pool.free_blocks()
            need = -(-n // B) - -(-model[s]["len"] // B)
            if need > free:
                with pytest.raises(_lib.HpdError) as e:
                    pool.reserve(s, n)
                assert e.value.status == 6
            else:
                pool.reserve(s, n)
                model[s]["len"] = n
        elif op == 3:
            s = int(rng.choice(live))
            n = int(rng.integers(0, model[s]["len"] + 1))
            forks = [m["fork"] for m in model.values() if m["live"] and m["parent"] == s]
            if forks and max(forks) > n:
                with pytest.raises(_lib.HpdError):
                    pool.truncate(s, n)
            else:
                pool.truncate(s, n)
                model[s]["len"] = n
        else:
            s = int(rng.choice(live))
            pool.release(s)
            model[s]["live"] = False
        # accounting: blocks held = live sequences + released roots with live branches
        held = []
        for s, m in model.items():
            alive_kids = any(k["live"] and k["parent"] == s for k in model.values())
            if m["live"]:
                info = pool.info(s)
                assert info["len"] == m["len"] and info["num_blocks"] == -(-m["len"] // B)
                held += pool.blocks(s).tolist()
            elif m["parent"] == -1 and alive_kids:   # released root: the blocks its branches see
                fmax = max(k["fork"] for k in model.values() if k["live"] and k["parent"] == s)
                held += [None] * -(-fmax // B)
        assert len(held) + pool.free_blocks() == NB
        ids = [b for b in held if b is not None]
        assert len(set(ids)) == len(ids) and all(0 <= b < NB for b in ids)
    # released sequence ids are reused; nothing leaks
    for s, m in model.items():
        if m["live"]:
            pool.release(s)
    assert pool.free_blocks() == NB


def _pool_layout(st, block_rows, rng, num_blocks=None):
    """Roots for the pages and branches for the branches of a structure, with
    the free list scrambled first; returns (pool, paged tables)."""
    nb = len(st["num_new"])
    need = sum(-(-int(P) // block_rows) for P in st["prefix_len"]) + \
        sum(-(-int(L + k) // block_rows) for L, k in zip(st["past_len"], st["num_new"]))
    pool = _lib.KvPool(num_blocks or need + 8, block_rows)
    junk = [pool.new() for _ in range(6)]
    for j in junk:
        pool.reserve(j, int(rng.integers(1, 3)) * block_rows)
    for j in rng.permutation(len(junk)):
        pool.release(junk[int(j)])
    roots = []
    for P in st["prefix_len"]:
        r = pool.new()
        pool.reserve(r, int(P))
        roots.append(r)
    kids = []
    for i in range(nb):
        p = int(st["branch_page"][i])
        f = int(st["prefix_len"][p]) if st.get("fork_len") is None else int(st["fork_len"][i])
        k = pool.new(roots[p], f)
        pool.reserve(k, int(st["past_len"][i] + st["num_new"][i]))
        kids.append(k)
    return pool, pool.batch_tables(roots, kids)


@pytest.mark.parametrize("name", ["c2", "c3", "c5"])
def test_paged_plan_maps_rows_through_the_blocks(name):
    rng = np.random.default_rng(11)
    st = make_structure(get_config(name), rng)
    B = 128
    pool, pg = _pool_layout(st, B, rng)
    plan = _lib.hpd_plan_create(16, 2, st["prefix_len"], st["branch_page"], st["num_new"], st["past_len"],
                                paged=pg)
    info = _lib.hpd_plan_query(plan)
    cp = canonical_plan(st["prefix_len"], st["branch_page"], st["num_new"], st["past_len"])
    for k in ("q_row", "page_q_row", "page_T", "visible"):
        assert np.array_equal(info[k].astype(np.int64), cp[k]), k
    assert info["shared_rows"] == info["priv_rows"] == pg["num_blocks"] * B
    # the same work lists as the contiguous plan, apart from the row field
    flat = _lib.hpd_plan_query(_lib.hpd_plan_create(16, 2, st["prefix_len"], st["branch_page"], st["num_new"],
                                                    st["past_len"]))
    S, Pi = _lib.SI, _lib.PI
    si, fi = info["shared_items"].copy(), flat["shared_items"].copy()
    si[:, S["prefix_row"]] = fi[:, S["prefix_row"]] = 0
    assert np.array_equal(si, fi)
    pi, fp = info["private_items"].copy(), flat["private_items"].copy()
    pi[:, Pi["priv_row"]] = fp[:, Pi["priv_row"]] = 0
    assert np.array_equal(pi, fp)
    assert np.array_equal(info["token_slots"], flat["token_slots"])


BAD_PAGED = [
    (dict(block_rows=96), "multiple of 64"),
    (dict(num_blocks=0), "num_blocks"),
    (dict(blocks_add=10 ** 6), "block id"),
    (dict(page_block0_add=10 ** 6), "page_block0"),
    (dict(branch_block0_add=10 ** 6), "branch_block0"),
    (dict(with_rows=True), "must be NULL"),
]


@pytest.mark.parametrize("over,needle", BAD_PAGED)
def test_paged_validation(over, needle):
    rng = np.random.default_rng(2)
    st = make_structure(get_config("c2"), rng)
    pool, pg = _pool_layout(st, 128, rng)
    pg = dict(pg)
    for k in ("block_rows", "num_blocks"):
        if k in over:
            pg[k] = over[k]
    for k in ("blocks", "page_block0", "branch_block0"):
        if k + "_add" in over:
            pg[k] = pg[k] + over[k + "_add"]
    kw = dict(paged=pg)
    if over.get("with_rows"):
        kw["prefix_row"] = np.zeros(len(st["prefix_len"]), np.int64)
    with pytest.raises(_lib.HpdError) as e:
        _lib.hpd_plan_create(16, 2, st["prefix_len"], st["branch_page"], st["num_new"], st["past_len"], **kw)
    assert needle in str(e.value)
