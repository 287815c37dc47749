"""GPU parity of one branch-parallel attention layer against the fp64 oracle.

Every call goes through the C ABI (hpd_plan_create / hpd_plan_upload /
hpd_branch_attn_step in libhpd.so)."""

import numpy as np
import pytest
import torch

from oracle.attention import attention_for_batch
from workloads import make_attn_batch
from workloads.gen import attn_batch_from_structure

from ._gpu import LSE_ABS, announce, assert_parity, run_batch, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c3f", "c5"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_workload_parity(name, seed):
    announce(f"workload {name} seed {seed}")
    b = make_attn_batch(name, seed)
    O, lse = run_batch(b, fork_len=b.fork_len)
    Oref, lref = attention_for_batch(b)
    mx, rl = assert_parity(O, Oref, b.dtype, f"{name}/{seed}")
    assert np.abs(lse - lref).max() <= LSE_ABS
    print(f"{name} seed {seed}: max abs {mx:.3e} rel L2 {rl:.3e}")


def _custom(prefix_len, branch_page, num_new, past_len, Hq, Hkv, dtype="bf16", seed=0):
    st = dict(prefix_len=np.array(prefix_len, np.int32), branch_page=np.array(branch_page, np.int32),
              num_new=np.array(num_new, np.int32), past_len=np.array(past_len, np.int32))
    return attn_batch_from_structure(st, Hq, Hkv, 64, dtype, seed)


EDGE = {
    # empty prefix on one page, L = 0, ragged tails everywhere
    "empty_prefix": ([0, 70], [0, 0, 1], [1, 3, 2], [0, 5, 63], 16, 2),
    # maximum draft window, keys crossing several chunks, G = 1
    "max_k_g1": ([129], [0, 0], [16, 16], [300, 0], 4, 4),
    # large group (G = 32) -> 32 stacked rows per token
    "group32": ([65], [0, 0], [2, 1], [1, 200], 32, 1),
    # Hq = 64 heads, single branch, prefix of exactly one tile
    "many_heads": ([64], [0], [3], [64], 64, 8),
    # one key per branch at L = 0 and k = 1 (private part is the token itself)
    "tiny": ([1], [0, 0, 0], [1, 1, 1], [0, 0, 0], 8, 2),
    # a page with no branches between two pages with branches
    "idle_page": ([33, 500, 257], [0, 2, 2], [4, 4, 1], [10, 127, 128], 16, 2),
    # a prefix ten times the workloads' longest: many splits per row group
    "long_prefix": ([40000], [0] * 5, [1, 4, 4, 4, 3], [512, 7, 130, 0, 64], 16, 2),
    # private histories far beyond the workloads' 1024 clip: 40 private chunks
    # and more than 16 partial slots per token (several merge batches)
    "long_private": ([64], [0, 0, 0], [4, 1, 4], [5000, 3071, 129], 16, 2),
    # more than 4,096 (token, head) rows: the merge's wide form
    "many_rows": ([300, 200], [0] * 40 + [1] * 37, [1] + [4] * 39 + [1] + [4] * 36,
                  [(7 * i) % 90 for i in range(77)], 16, 2),
}


@pytest.mark.parametrize("case", list(EDGE))
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_edge_cases(case, dtype):
    announce(f"edge {case} {dtype}")
    b = _custom(*EDGE[case], dtype=dtype, seed=11)
    O, lse = run_batch(b)
    Oref, lref = attention_for_batch(b)
    assert_parity(O, Oref, dtype, case)
    assert np.abs(lse - lref).max() <= LSE_ABS


def test_fp32_output_of_bf16_inputs():
    announce("bf16 in, fp32 out")
    b = make_attn_batch("c2", 4)
    O, _ = run_batch(b, out_dtype=torch.float32)
    Oref, _ = attention_for_batch(b)
    assert_parity(O, Oref, "bf16", "c2 fp32 out")


def test_fork_lengths():
    """Per-branch visible prefix F_b < P_p (tree-shaped prefix)."""
    announce("fork lengths")
    b = make_attn_batch("c2", 5)
    rng = np.random.default_rng(5)
    fork = rng.integers(0, int(b.prefix_len[0]) + 1, size=b.num_branches).astype(np.int32)
    fork[0] = 0
    fork[1] = int(b.prefix_len[0])
    b.fork_len = fork
    O, lse = run_batch(b, fork_len=fork)
    Oref, lref = attention_for_batch(b)
    assert_parity(O, Oref, "bf16", "fork")
    assert np.abs(lse - lref).max() <= LSE_ABS


FORK_CASES = {
    # three pages, ragged k and L, forks drawn per branch
    "three_pages": ([700, 1500, 333], [0, 0, 0, 1, 1, 2, 2, 2], [1, 4, 4, 1, 4, 2, 3, 4],
                    [10, 50, 0, 5, 200, 64, 1, 9], 16, 2),
    # G = 12: a token's 12 rows straddle 32-row waves and 128-row items
    "g12": ([900], [0, 0, 0, 0, 0], [1, 4, 4, 3, 2], [30, 7, 0, 100, 12], 12, 1),
    # G = 1 and 24 branches: waves of sorted rows that skip most key tiles
    "g1_many": ([2048], [0] * 24, [1] + [4] * 23, list(range(0, 240, 10)), 4, 4),
}


@pytest.mark.parametrize("case", list(FORK_CASES))
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_fork_sorted_rows(case, dtype):
    """Fork offsets: the planner stacks each page's tokens by descending fork
    point and the kernels skip the key tiles a wave's rows do not see."""
    announce(f"fork sorted {case} {dtype}")
    b = _custom(*FORK_CASES[case], dtype=dtype, seed=13)
    rng = np.random.default_rng(len(case))
    P_b = b.prefix_len[b.branch_page]
    fork = np.array([rng.integers(0, int(P) + 1) for P in P_b], np.int32)
    fork[0], fork[-1] = P_b[0], 0
    b.fork_len = fork
    O, lse = run_batch(b, fork_len=fork)
    Oref, lref = attention_for_batch(b)
    assert_parity(O, Oref, dtype, case)
    assert np.abs(lse - lref).max() <= LSE_ABS


def test_custom_offsets_and_canaries():
    """Rows live at caller-chosen offsets; every row outside the plan is NaN
    and must never be read."""
    announce("custom offsets + NaN canaries")
    b = make_attn_batch("c5", 7)
    nb, D = b.num_branches, 64
    rng = np.random.default_rng(1)
    gaps_p = rng.integers(1, 9, size=b.num_pages)
    pr = np.cumsum(np.concatenate([[gaps_p[0]], (b.prefix_len[:-1] + gaps_p[1:])])).astype(np.int64)
    rows = (b.past_len + b.num_new).astype(np.int64)
    gaps_b = rng.integers(1, 5, size=nb)
    vr = np.cumsum(np.concatenate([[gaps_b[0]], (rows[:-1] + gaps_b[1:])])).astype(np.int64)
    sh_rows = int(pr[-1] + b.prefix_len[-1] + 3)
    pv_rows = int(vr[-1] + rows[-1] + 3)
    nan = np.uint16(0x7FC0)

    def place(src, starts, lens, total):
        dst = np.full((total, b.num_kv_heads, D), nan, np.uint16)
        off = 0
        for s, n in zip(starts, lens):
            dst[s:s + n] = src[off:off + n]
            off += n
        return to_dev(dst, "bf16")
    sk = place(b.shared_k, pr, b.prefix_len, sh_rows)
    sv = place(b.shared_v, pr, b.prefix_len, sh_rows)
    pk = place(b.priv_k, vr, rows, pv_rows)
    pv = place(b.priv_v, vr, rows, pv_rows)
    O, lse = run_batch(b, prefix_row=pr, priv_row=vr, shared_k=sk, shared_v=sv, priv_k=pk, priv_v=pv)
    Oref, lref = attention_for_batch(b)
    assert_parity(O, Oref, "bf16", "offsets")


def test_deterministic_and_isolated():
    """Two runs agree bit for bit; changing one branch's private K/V leaves
    every other branch's output bit-identical."""
    announce("determinism + isolation")
    b = make_attn_batch("c3", 3)
    O1, l1 = run_batch(b)
    O2, l2 = run_batch(b)
    assert np.array_equal(O1, O2) and np.array_equal(l1, l2)
    victim = 5
    r0 = int(np.sum(b.past_len[:victim] + b.num_new[:victim]))
    r1 = r0 + int(b.past_len[victim] + b.num_new[victim])
    pk = b.priv_k.copy()
    pk[r0:r1] = pk[r0:r1] ^ np.uint16(0x0040)      # perturb the victim's keys
    O3, _ = run_batch(b, priv_k=to_dev(pk, "bf16"))
    t0 = int(np.sum(b.num_new[:victim]))
    t1 = t0 + int(b.num_new[victim])
    keep = np.ones(O1.shape[0], bool)
    keep[t0:t1] = False
    assert np.array_equal(O1[keep], O3[keep])
    assert not np.array_equal(O1[t0:t1], O3[t0:t1])
