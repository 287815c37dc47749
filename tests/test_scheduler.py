"""Host scheduler of the inference workflow (Algorithm 1): the oracle pinned
by hand-traced scenarios, and the C++ scheduler (hpd_sched_*) against the
oracle on the same scenarios and on seeded random token streams.  CPU only.

The hand traces follow the algorithm's steps with the readings of the
oracle's docstring; each expected value is derived in the comments."""

import numpy as np
import pytest

from oracle.scheduler import Scheduler as OracleSched
from paper_2607_18839_amd import _lib

MAXK = _lib.HPD_MAX_K


class Cpp:
    """The C++ scheduler behind the oracle's interface."""

    def __init__(self, **cfg):
        self.s = _lib.Sched(cfg["num_blocks"], cfg["block_rows"], cfg["tau"], cfg["window"], cfg["max_active"],
                            cfg["fork_token"], cfg["child_token"], cfg["eos_token"])
        self.finished = []

    def submit(self, prompt_len, first_token, max_new):
        return self.s.submit(prompt_len, first_token, max_new)

    def schedule(self):
        b = self.s.schedule()
        return dict(requests=b["request"].tolist(), branch_page=b["branch_page"].tolist(),
                    num_new=b["num_new"].tolist(), past_len=b["past_len"].tolist(), fork_len=b["fork_len"].tolist(),
                    prefix_len=b["prefix_len"].tolist(), tokens_in=b["tokens_in"].tolist(),
                    prefill=list(zip(b["prefill_from"].tolist(), b["prefill_to"].tolist())),
                    preempted=b["preempted"].tolist(), admitted=b["admitted"].tolist(), _raw=b)

    def commit(self, verified, n_acc, draft_out):
        d = np.zeros((len(n_acc), MAXK), np.int32)
        for i, row in enumerate(draft_out):
            d[i, :len(row)] = row
        self.s.commit(np.asarray(verified, np.int32), np.asarray(n_acc, np.int32), d)
        while (o := self.s.next_output()) is not None:
            self.finished.append((o[0], o[1].tolist()))

    def free_blocks(self):
        return self.s.counts()["free_blocks"]


class Orc(OracleSched):
    def __init__(self, **cfg):
        super().__init__(cfg["num_blocks"], cfg["block_rows"], cfg["tau"], cfg["window"], cfg["max_active"],
                         cfg["fork_token"], cfg["child_token"], cfg["eos_token"])

    def free_blocks(self):
        return len(self.free)


BATCH_KEYS = ("requests", "branch_page", "num_new", "past_len", "fork_len", "prefix_len", "tokens_in", "prefill",
              "preempted", "admitted")


def _pad(rows):
    return [list(r) + [0] * (MAXK - len(r)) for r in rows]


def _expect(batch, **want):
    for k, v in want.items():
        assert list(batch[k]) == v, (k, batch[k], v)


IMPLS = [pytest.param(Orc, id="oracle"), pytest.param(Cpp, id="cpp")]


@pytest.mark.parametrize("impl", IMPLS)
def test_scenario_gate_fork_rollback_interleave(impl):
    """N_max = 1, 64-row blocks, K = 3; fork token 7, child token 8, eos 9."""
    s = impl(num_blocks=100, block_rows=64, tau=1.0, window=3, max_active=1, fork_token=7, child_token=8,
             eos_token=9)
    assert s.submit(100, 1, 50) == 0 and s.submit(10, 2, 50) == 1
    # 1: request 0 is admitted (prompt 100 + 1 fed token -> 2 blocks); 1 waits on N_max
    b = s.schedule()
    _expect(b, requests=[0], num_new=[1], past_len=[100], fork_len=[0], prefix_len=[0], tokens_in=[1],
            prefill=[(0, 100)], admitted=[0], preempted=[])
    assert s.free_blocks() == 98
    s.commit([5], [0], _pad([[5, 6, 7]]))            # emits 5; len 101; next window 5 6 7
    # 2: feeds its window of 3
    b = s.schedule()
    _expect(b, requests=[0], num_new=[3], past_len=[101], tokens_in=[5, 6, 7], prefill=[(101, 101)], admitted=[])
    # drafts 6, 7 verified (y*_0 = 6, y*_1 = 7), bonus 4: emits 6 7 4, len 104;
    # the fork token 7 is y*_1, at position 101 + 1 + 1: the child sees 103 rows
    s.commit([6, 7, 4], [2], _pad([[4, 1, 1]]))
    # 3: the queue was dirtied: child 2 (key (0, 0, -1, 2)) before parent 1
    # (key (1, 1)); the child bypasses N_max and takes 1 block
    b = s.schedule()
    _expect(b, requests=[0, 2], branch_page=[0, 0], num_new=[3, 1], past_len=[104, 0], fork_len=[0, 103],
            prefix_len=[103], tokens_in=[4, 1, 1, 8], prefill=[(104, 104), (0, 0)], admitted=[2])
    assert s.free_blocks() == 97
    # request 0: y*_0 = 1 verifies draft 1, bonus 9 = eos -> done after 5 6 7 4 1;
    # the child emits 11 (len 1).  The page's 2 blocks stay: the child sees 103 rows.
    s.commit([1, 9, 3, 11], [1, 0], _pad([[9, 0, 0], [11, 12, 13]]))
    assert s.free_blocks() == 97 and s.finished == []
    # 4: only the child is active; parent 1 still waits on N_max
    b = s.schedule()
    _expect(b, requests=[2], branch_page=[0], num_new=[3], past_len=[1], fork_len=[103], prefix_len=[103],
            tokens_in=[11, 12, 13], admitted=[])
    s.commit([12, 9, 0], [1], _pad([[0, 0, 0]]))    # emits 12, then eos
    # every block returns; the page is output with the child after its fork token
    assert s.free_blocks() == 100
    assert s.finished == [(0, [5, 6, 7, 11, 12, 4, 1])]
    # 5: parent 1 is admitted with its prefill
    b = s.schedule()
    _expect(b, requests=[1], past_len=[10], prefill=[(0, 10)], tokens_in=[2], admitted=[1])
    assert s.free_blocks() == 99


@pytest.mark.parametrize("impl", IMPLS)
def test_scenario_preempt_youngest_and_resume(impl):
    """5 blocks of 64 rows, K = 4; two pages of 120 prompt rows."""
    s = impl(num_blocks=5, block_rows=64, tau=1.0, window=4, max_active=10, fork_token=100, child_token=101,
             eos_token=102)
    s.submit(120, 1, 1000)
    s.submit(120, 2, 1000)
    b = s.schedule()                                 # 2 blocks each (121 rows)
    _expect(b, requests=[0, 1], branch_page=[0, 1], num_new=[1, 1], past_len=[120, 120], prefix_len=[0, 0],
            prefill=[(0, 120), (0, 120)], admitted=[0, 1])
    assert s.free_blocks() == 1
    s.commit([3, 4], [0, 0], _pad([[3] * 4, [4] * 4]))             # len 121 each
    b = s.schedule()                                 # 125 rows: still 2 blocks each
    _expect(b, num_new=[4, 4], past_len=[121, 121], preempted=[])
    s.commit([3] * 4 + [4] * 4, [3, 3], _pad([[3] * 4, [4] * 4]))  # len 125 each
    # 3: request 0 needs 129 rows = 3 blocks and takes the last free one;
    # request 1 then fails, is the youngest, and is preempted (its 2 blocks
    # return); it cannot be readmitted (3 blocks needed, 2 free)
    b = s.schedule()
    _expect(b, requests=[0], num_new=[4], past_len=[125], preempted=[1], admitted=[])
    assert s.free_blocks() == 2
    s.commit([3] * 4, [3], _pad([[3] * 4]))          # len 129
    b = s.schedule()
    _expect(b, requests=[0], past_len=[129], admitted=[])
    s.commit([102, 0, 0, 0], [0], _pad([[0] * 4]))   # eos: done, page 0 output
    assert s.free_blocks() == 5 and s.finished == [(0, [3] * 9)]
    # 5: request 1 resumes and recomputes all its 125 rows
    b = s.schedule()
    _expect(b, requests=[1], past_len=[125], prefill=[(0, 125)], tokens_in=[4, 4, 4, 4], admitted=[1])
    assert s.free_blocks() == 2


@pytest.mark.parametrize("impl", IMPLS)
def test_scenario_kv_threshold_gates_parents_not_children(impl):
    """tau = 0.3 of 10 blocks: parents wait while more than 3 blocks are used."""
    s = impl(num_blocks=10, block_rows=64, tau=0.3, window=2, max_active=10, fork_token=7, child_token=8,
             eos_token=9)
    for _ in range(3):
        s.submit(127, 5, 100)                        # 2 blocks each at admission
    b = s.schedule()                                 # 0 used -> admit, 2 used -> admit, 4 > 3 -> stop
    _expect(b, requests=[0, 1], admitted=[0, 1])
    s.commit([7, 5], [0, 0], _pad([[5, 5], [5, 5]]))  # page 0 forks at 127 + 0 + 1
    # 2: 0 and 1 grow to 3 blocks (130 rows); child 3 bypasses the gate (6 used)
    b = s.schedule()
    _expect(b, requests=[0, 3, 1], branch_page=[0, 0, 1], num_new=[2, 1, 2], past_len=[128, 0, 128],
            fork_len=[0, 128, 0], prefix_len=[128, 0], tokens_in=[5, 5, 8, 5, 5], admitted=[3])
    assert s.free_blocks() == 3


def test_scheduler_batch_builds_a_paged_plan():
    """The C++ batch (tables included) is a valid paged plan whose visible
    counts are F_b + L_b + j + 1."""
    s = Cpp(num_blocks=10, block_rows=64, tau=0.3, window=2, max_active=10, fork_token=7, child_token=8,
            eos_token=9)
    for _ in range(3):
        s.submit(127, 5, 100)
    s.schedule()
    s.commit([7, 5], [0, 0], _pad([[5, 5], [5, 5]]))
    b = s.schedule()["_raw"]
    plan = _lib.hpd_plan_create(16, 2, b["prefix_len"], b["branch_page"], b["num_new"], b["past_len"],
                                fork_len=b["fork_len"], paged=b["paged"])
    info = _lib.hpd_plan_query(plan)
    want = [f + L + j + 1 for f, L, k in zip(b["fork_len"], b["past_len"], b["num_new"]) for j in range(k)]
    assert info["visible"].tolist() == want
    # the parent branch reads the page's blocks as its own rows
    p0, b0 = b["paged"]["page_block0"], b["paged"]["branch_block0"]
    blocks = b["paged"]["blocks"]
    assert blocks[b0[0]:b0[0] + 3].tolist() == blocks[p0[0]:p0[0] + 3].tolist()


def test_commit_and_schedule_misuse_change_nothing():
    s = _lib.Sched(8, 64, 1.0, 2, 4, 7, 8, 9)
    with pytest.raises(_lib.HpdError):
        s.commit(None, None, None)                   # nothing scheduled
    s.submit(10, 1, 5)
    s.schedule()
    with pytest.raises(_lib.HpdError):
        s.schedule()                                 # the batch awaits its commit
    with pytest.raises(_lib.HpdError):
        s.commit([1], [1], np.zeros((1, MAXK), np.int32))   # n_acc must be < num_new = 1
    s.commit([1], [0], np.zeros((1, MAXK), np.int32))
    assert s.request(0) == dict(state="active", len=11, kept=11, recorded=1)
    with pytest.raises(_lib.HpdError):
        _lib.Sched(8, 64, 1.5, 2, 4, 7, 8, 9)        # tau out of [0, 1]
    with pytest.raises(_lib.HpdError):
        _lib.Sched(8, 64, 1.0, MAXK + 1, 4, 7, 8, 9)


# ---------------------------------------------------------------- random streams

FORK, CHILD, EOS = 1, 2, 3


def _tokens(rng, n, p_fork, p_eos):
    u = rng.random(n)
    t = rng.integers(10, 60, size=n)
    t[u < p_fork + p_eos] = EOS
    t[u < p_fork] = FORK
    return t


def _step_outputs(rng, batch, window, p_fork, p_eos):
    """Verification results of one step: random acceptance counts, the
    accepted drafts verified by the token one position earlier, random
    tokens elsewhere, random next windows."""
    nb = len(batch["requests"])
    n_acc, verified, q = [], [], 0
    toks = batch["tokens_in"]
    for k in batch["num_new"]:
        n = int(rng.integers(0, k))
        v = _tokens(rng, k, p_fork, p_eos).tolist()
        for i in range(n):
            v[i] = toks[q + i + 1]
        n_acc.append(n)
        verified += v
        q += k
    drafts = _pad(rng.integers(10, 60, size=(nb, window)).tolist())
    return verified, n_acc, drafts


def _check_oracle_invariants(o):
    refs = [0] * o.num_blocks
    for r in o.reqs:
        for blk in r.blocks + r.shared:
            refs[blk] += 1
    assert refs == o.ref
    assert sorted(o.free) == [b for b in range(o.num_blocks) if refs[b] == 0]
    for r in o.P:
        assert len(r.blocks) == -(-r.len // o.B) or r.status != "active"
        if r.is_child:
            assert r.fork_len <= o.reqs[r.parent].len


CASES = [
    # num_blocks, block_rows, tau, window, max_active, p_fork, p_eos, arrivals, max_new
    (40, 64, 0.9, 4, 6, 0.08, 0.02, 12, 60),
    (12, 64, 1.0, 4, 8, 0.10, 0.005, 10, 300),   # tight pool: preemption
    (30, 128, 0.5, 3, 4, 0.15, 0.03, 16, 60),
    (9, 64, 0.8, 6, 16, 0.05, 0.005, 8, 300),    # tight pool, long windows
    (200, 64, 1.0, 1, 3, 0.10, 0.05, 20, 60),    # K = 1: no drafts
]


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_cpp_scheduler_matches_the_oracle_on_random_streams(case, seed):
    nblk, brows, tau, K, nmax, pf, pe, arrivals, max_new = CASES[case]
    cfg = dict(num_blocks=nblk, block_rows=brows, tau=tau, window=K, max_active=nmax, fork_token=FORK,
               child_token=CHILD, eos_token=EOS)
    o, c = Orc(**cfg), Cpp(**cfg)
    rng = np.random.default_rng([seed, case])
    submitted, stats = 0, dict(preempted=0, forks=0, steps=0)
    for it in range(3000):
        if submitted < arrivals and rng.random() < 0.3:
            prompt = int(rng.integers(1, 3 * brows))
            args = (prompt, int(rng.integers(10, 60)), int(rng.integers(4, max_new)))
            assert o.submit(*args) == c.submit(*args)
            submitted += 1
        bo, bc = o.schedule(), c.schedule()
        for k in BATCH_KEYS:
            assert list(bo[k]) == list(bc[k]), (it, k, bo[k], bc[k])
        # the C++ tables give each page and branch the blocks its rows need
        raw = bc["_raw"]
        if raw["num_branches"]:
            pg = raw["paged"]
            ends = np.concatenate([pg["page_block0"], pg["branch_block0"], [len(pg["blocks"])]])
            assert np.all(np.diff(np.sort(ends)) >= 0)
            _lib.hpd_plan_create(16, 2, raw["prefix_len"], raw["branch_page"], raw["num_new"], raw["past_len"],
                                 fork_len=raw["fork_len"], paged=pg)
        stats["preempted"] += len(bo["preempted"])
        if bo["requests"]:
            stats["steps"] += 1
        out = _step_outputs(rng, bo, K, pf, pe)
        o.commit(*out)
        c.commit(*out)
        assert o.free_blocks() == c.free_blocks(), it
        _check_oracle_invariants(o)
        assert o.finished == c.finished, it
        if submitted == arrivals and not o.P:
            # drained, or stalled: nothing active and the queue's head does not
            # fit next to the blocks that waiting requests hold (both sides
            # report the same state)
            cw = c.s.counts()
            assert (cw["waiting"], cw["active"]) == (len(o.Q), 0)
            break
    assert submitted == arrivals
    if case in (1, 3):
        assert stats["preempted"] > 0, "a tight pool must preempt"
        if o.Q:
            return   # stalled
    assert not o.Q, "the stream did not drain"
    assert o.free_blocks() == nblk == c.free_blocks()
    parents = [r for r in o.reqs if not r.is_child]
    assert sorted(p for p, _ in o.finished) == [r.id for r in parents]
    for pid, toks in o.finished:   # a page holds its parent's and its children's tokens
        kids = [r for r in o.reqs if r.is_child and r.parent == pid]
        assert len(toks) == len(o.reqs[pid].out) + sum(len(k.out) for k in kids)
    assert any(r.is_child for r in o.reqs)


@pytest.mark.parametrize("impl", IMPLS)
def test_scenario_kv_threshold_is_strict(impl):
    """tau = 0.4 of 10 blocks: a parent is still admitted at exactly 4 used
    blocks (the gate is usage > tau), not at 6."""
    s = impl(num_blocks=10, block_rows=64, tau=0.4, window=2, max_active=10, fork_token=7, child_token=8,
             eos_token=9)
    for _ in range(4):
        s.submit(127, 5, 100)
    b = s.schedule()
    _expect(b, requests=[0, 1, 2], admitted=[0, 1, 2])
    assert s.free_blocks() == 4


@pytest.mark.parametrize("impl", IMPLS)
def test_scenario_preempted_request_goes_to_the_front(impl):
    """N_max = 2 keeps page 2 waiting; the preempted page 1 is put in front
    of it and, not fitting, blocks it (FCFS: no overtaking)."""
    s = impl(num_blocks=5, block_rows=64, tau=1.0, window=4, max_active=2, fork_token=100, child_token=101,
             eos_token=102)
    s.submit(120, 1, 1000)
    s.submit(120, 2, 1000)
    s.submit(10, 3, 1000)
    _expect(s.schedule(), requests=[0, 1], admitted=[0, 1])
    s.commit([3, 4], [0, 0], _pad([[3] * 4, [4] * 4]))
    _expect(s.schedule(), requests=[0, 1], admitted=[])
    s.commit([3] * 4 + [4] * 4, [3, 3], _pad([[3] * 4, [4] * 4]))   # len 125 each
    # request 0 takes the last block; 1 is preempted to the queue's front and
    # needs 3 blocks with 2 free: admission stops before page 2 (1 block)
    _expect(s.schedule(), requests=[0], preempted=[1], admitted=[])
    assert s.free_blocks() == 2


# ---------------------------------------------------------------- planted mistakes

SCHED_MUTANTS = [
    ("v = max(self.P, key=lambda x: x.arrival)", "v = min(self.P, key=lambda x: x.arrival)"),   # preempt oldest
    ("self._spawn(r, base + i + 1)", "self._spawn(r, base + i)"),                              # fork off by one
    ("if not r.is_child and (self.used_blocks()", "if (self.used_blocks()"),                    # children gated
    ("self.used_blocks() > self.tau", "self.used_blocks() >= self.tau"),                        # gate not strict
    ("r.len = base + n + 1", "r.len = base + n"),                                              # bonus row lost
    ("return (0, self.reqs[r.parent].arrival", "return (2, self.reqs[r.parent].arrival"),     # parents first
    ("if t == self.eos:", "if t == self.eos and False:"),                                      # eos ignored
    ("out += self.reqs[spawned[i]].out", "out[-1:-1] = self.reqs[spawned[i]].out"),            # child before fork
    ("need = ceil_div(r.len + len(r.window), self.B)", "need = ceil_div(r.len + 1, self.B)"),  # window not reserved
    ("r.window = [int(t) for t in draft_out[b][:self.K]]", "r.window = [int(t) for t in draft_out[b][:1]]"),
    ("self.Q.insert(0, v)", "self.Q.append(v)"),                                               # preempted to the back
]


def _mutant_class(old, new):
    import os
    import types
    src = open(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                            "scheduler.py")).read()
    assert src.count(old) == 1, f"mutation anchor not found once: {old!r}"
    mod = types.ModuleType("oracle_scheduler_mutant")
    exec(compile(src.replace(old, new), "<scheduler mutant>", "exec"), mod.__dict__)

    class M(mod.Scheduler):
        def __init__(self, **cfg):
            super().__init__(cfg["num_blocks"], cfg["block_rows"], cfg["tau"], cfg["window"], cfg["max_active"],
                             cfg["fork_token"], cfg["child_token"], cfg["eos_token"])

        def free_blocks(self):
            return len(self.free)
    return M


PINS = [test_scenario_gate_fork_rollback_interleave, test_scenario_preempt_youngest_and_resume,
        test_scenario_kv_threshold_gates_parents_not_children, test_scenario_kv_threshold_is_strict,
        test_scenario_preempted_request_goes_to_the_front]


@pytest.mark.parametrize("old,new", SCHED_MUTANTS)
def test_scheduler_pins_catch_planted_mistakes(old, new):
    M = _mutant_class(old, new)
    caught = []
    for pin in PINS:
        try:
            pin(M)
        except Exception:
            caught.append(pin.__name__)
    assert caught, f"no pin catches {new!r}"
