"""Algorithm 1 (section "Inference Workflow"): FCFS scheduling with
hierarchical parallel decoding, in plain Python (oracle side).

Test infrastructure: see the package docstring.

The algorithm's steps, in its order, with the readings recorded in the
design notes (the paper names the operations, not their bookkeeping):

* Requests.  A parent is a page: its layout branch decodes after a prefill of
  prompt_len rows (visual tokens + prompt, computed outside the decode step)
  that also yields its first token.  A child is a content branch spawned when
  its parent emits the fork token; it sees the parent's rows before that
  token (fork_ptr, no copy) and starts from the child token.  Ids and arrival
  times are one counter, in order of submission or spawn.
* KV.  Blocks of block_rows rows with per-block reference counts.  A parent
  holds the blocks of its page sequence (prompt + accepted tokens); a child
  references the parent's first ceil(F / block_rows) blocks and holds its own
  for its private rows.  AllocKV for a step makes room for len + k rows (k =
  the tokens the request feeds); PartialFree drops a request's references to
  the blocks nobody else references (a parent keeps those its live children
  see, a child keeps its reference to the parent's prefix) and marks the
  dropped rows for recomputation.
* One iteration = schedule() (sort the queue if dirty; AllocKV for every
  active request, preempting the youngest active request while it fails;
  admission: parents gated by KV usage > tau or |P| >= N_max, children
  bypass the gate, and an admitted request must get its KV, else admission
  stops), the caller's decode step + verification, then commit() (length
  update len += n_acc + 1 with rollback of the rejected rows, the emitted
  tokens y*_0 .. y*_{n_acc}, fork detection, done detection, reference-
  counted release, and the interleaved output of a page once its parent is
  done and none of its children is live).
* Emitted tokens.  EOS ends a request and is not recorded; a request is also
  done when it has recorded max_new tokens.  A page's output is its parent's
  tokens with each child's tokens placed right after the fork token that
  spawned it.
"""

WAITING, ACTIVE, DONE = "waiting", "active", "done"


def ceil_div(a, b):
    return -(-a // b)


class Req:
    def __init__(self, rid, is_child, parent, prompt_len, max_new, window, fork_len=0):
        self.id = rid
        self.arrival = rid
        self.is_child = is_child
        self.parent = parent            # child: the parent's id; parent: its own id
        self.max_new = max_new
        self.len = prompt_len           # rows of its own sequence (parent: the page's)
        self.kept = 0                   # rows whose K/V is held and valid
        self.fork_len = fork_len        # child: parent rows it sees
        self.window = list(window)      # tokens to feed next
        self.out = []
        self.forks = []                 # (index of the fork token in out, child id)
        self.blocks = []                # own block ids (parent: the page's blocks)
        self.shared = []                # child: the parent's blocks it references
        self.status = WAITING


class Scheduler:
    def __init__(self, num_blocks, block_rows, tau, window, max_active, fork_token, child_token, eos_token):
        self.B = block_rows
        self.num_blocks = num_blocks
        self.ref = [0] * num_blocks
        self.free = list(range(num_blocks))   # which ids are free; counts are what tests compare
        self.tau, self.K, self.n_max = tau, window, max_active
        self.fork_token, self.child_token, self.eos = fork_token, child_token, eos_token
        self.reqs = []
        self.P, self.Q = [], []
        self.fork_rel = {}
        self.queue_dirty = False
        self.finished = []                    # (parent id, interleaved tokens)
        self.batch = None

    # ------------------------------------------------------------ blocks
    def used_blocks(self):
        return self.num_blocks - len(self.free)

    def _take(self):
        b = self.free.pop(0)
        self.ref[b] = 1
        return b

    def _drop(self, b):
        self.ref[b] -= 1
        if self.ref[b] == 0:
            self.free.append(b)

    def _alloc(self, r):
        """AllocKV: blocks for len + k rows, all or nothing."""
        need = ceil_div(r.len + len(r.window), self.B) - len(r.blocks)
        if need > len(self.free):
            return False
        r.blocks += [self._take() for _ in range(max(need, 0))]
        return True

    def _shrink(self, r, rows):
        """Drop r's own blocks past `rows` rows."""
        keep = ceil_div(rows, self.B)
        while len(r.blocks) > keep:
            self._drop(r.blocks.pop())

    def _live_children(self, pid):
        return [self.reqs[c] for c in self.fork_rel.get(pid, [])]

    def _partial_free(self, v):
        if v.is_child:
            keep = 0
        else:   # the rows its live children see stay referenced and valid
            keep = max([c.fork_len for c in self._live_children(v.id)], default=0)
        self._shrink(v, keep)
        v.kept = min(v.kept, keep)

    # ------------------------------------------------------------ requests
    def submit(self, prompt_len, first_token, max_new):
        r = Req(len(self.reqs), False, None, prompt_len, max_new, [first_token])
        r.parent = r.id
        self.reqs.append(r)
        self.Q.append(r)
        self.fork_rel[r.id] = []
        return r.id

    def _spawn(self, p, fork_len):
        c = Req(len(self.reqs), True, p.id, 0, p.max_new, [self.child_token], fork_len)
        self.reqs.append(c)
        c.shared = p.blocks[:ceil_div(fork_len, self.B)]   # fork_ptr: references, no copy
        for b in c.shared:
            self.ref[b] += 1
        self.Q.append(c)
        self.fork_rel[p.id].append(c.id)
        self.queue_dirty = True
        return c

    # ------------------------------------------------------------ one iteration
    def schedule(self):
        # FCFS order of the waiting queue
        if self.queue_dirty:
            def key(r):
                if r.is_child:
                    return (0, self.reqs[r.parent].arrival, -len(self.fork_rel[r.parent]), r.arrival)
                return (1, r.arrival)
            self.Q.sort(key=key)
            self.queue_dirty = False
        # KV for every active request; preempt the youngest while it fails
        preempted = []
        for r in list(self.P):
            if r not in self.P:
                continue
            while not self._alloc(r):
                v = max(self.P, key=lambda x: x.arrival)
                self._partial_free(v)
                self.P.remove(v)
                v.status = WAITING
                self.Q.insert(0, v)
                preempted.append(v.id)
                if v is r:
                    break
        # admission: parents gated, children bypass
        admitted = []
        while self.Q:
            r = self.Q[0]
            if not r.is_child and (self.used_blocks() > self.tau * self.num_blocks or len(self.P) >= self.n_max):
                break
            if not self._alloc(r):
                break
            self.Q.pop(0)
            self.P.append(r)
            r.status = ACTIVE
            admitted.append(r.id)
        # the step's batch: pages by their parent's arrival, the parent first
        pages = sorted({r.parent for r in self.P}, key=lambda p: self.reqs[p].arrival)
        order = []
        for p in pages:
            members = [r for r in self.P if r.parent == p]
            members.sort(key=lambda r: (r.is_child, r.arrival))
            order += members
        batch = dict(pages=pages, requests=[r.id for r in order],
                     branch_page=[pages.index(r.parent) for r in order],
                     num_new=[len(r.window) for r in order],
                     past_len=[r.len for r in order],
                     fork_len=[r.fork_len if r.is_child else 0 for r in order],
                     prefix_len=[max([r.fork_len for r in order if r.is_child and r.parent == p], default=0)
                                 for p in pages],
                     tokens_in=[t for r in order for t in r.window],
                     prefill=[(r.kept, r.len) for r in order],
                     preempted=preempted, admitted=admitted)
        for r in order:
            r.kept = r.len   # the caller computes the prefill rows before the step
        self.batch = order
        return batch

    def commit(self, verified, n_acc, draft_out):
        """verified [T], n_acc [nb], draft_out [nb][>= K] of the step."""
        q = 0
        for b, r in enumerate(self.batch):
            k = len(r.window)
            n = int(n_acc[b])
            ys = [int(t) for t in verified[q:q + n + 1]]
            base = r.len
            r.len = base + n + 1          # s_0 .. s_n are kept
            r.kept = r.len
            self._shrink(r, r.len)        # rejected rows roll back
            r.window = [int(t) for t in draft_out[b][:self.K]]
            for i, t in enumerate(ys):
                if t == self.eos:
                    r.status = DONE
                    break
                r.out.append(t)
                if t == self.fork_token and not r.is_child:
                    c = self._spawn(r, base + i + 1)
                    r.forks.append((len(r.out) - 1, c.id))
                if len(r.out) >= r.max_new:
                    r.status = DONE
                    break
            q += k
        # reference-counted release
        for r in list(self.P):
            if r.status != DONE:
                continue
            self.P.remove(r)
            for blk in r.blocks + r.shared:
                self._drop(blk)
            r.blocks, r.shared = [], []
            if r.is_child:
                self.fork_rel[r.parent].remove(r.id)
            p = self.reqs[r.parent]
            if p.status == DONE and not self.fork_rel[p.id] and p.id in self.fork_rel:
                self.finished.append((p.id, self.interleave(p)))
                del self.fork_rel[p.id]
        self.batch = None

    def interleave(self, p):
        out = []
        spawned = dict(p.forks)
        for i, t in enumerate(p.out):
            out.append(t)
            if i in spawned:
                out += self.reqs[spawned[i]].out
        return out

    def info(self):
        return dict(waiting=[r.id for r in self.Q], active=[r.id for r in self.P],
                    free_blocks=len(self.free), lens={r.id: r.len for r in self.reqs})
