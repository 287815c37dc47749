// Host scheduler of the inference workflow (C ABI in include/hpd.h; section
// "Inference Workflow", Algorithm 1: FCFS scheduling with hierarchical
// parallel decoding).  Plain C++; the K/V blocks are an hpd_kv_pool owned by
// the scheduler (a page is a root sequence, a child a branch of it).
#include <algorithm>
#include <cstdint>
#include <deque>
#include <new>
#include <string>
#include <tuple>
#include <vector>

#include "hpd.h"

namespace hpd {
void set_last_error(const std::string &msg);
}

namespace {

enum { kWaiting = 0, kActive = 1, kDone = 2 };

struct Request {
  int32_t id = 0;
  bool child = false;
  int32_t page = 0;         // the parent's id (a parent: its own)
  int32_t max_new = 0;
  int32_t len = 0;          // rows of its own sequence (a parent: the page's)
  int32_t kept = 0;         // rows of them whose K/V is held
  int32_t fork_len = 0;     // child: page rows it sees
  int32_t seq = -1;         // hpd_kv_pool sequence
  int state = kWaiting;
  std::vector<int32_t> window, out;
  std::vector<std::pair<int32_t, int32_t>> forks;   // (index of the fork token in out, child)
  std::vector<int32_t> live_children;                // parent: children not finished
  bool emitted = false;                              // parent: page output produced
};

}  // namespace

struct hpd_sched {
  hpd_sched_config cfg{};
  hpd_kv_pool *pool = nullptr;
  std::vector<Request> reqs;
  std::vector<int32_t> active;     // P, in admission order
  std::deque<int32_t> queue;       // Q
  bool queue_dirty = false;
  bool pending = false;            // a batch awaits its commit
  std::deque<std::pair<int32_t, std::vector<int32_t>>> finished;
  // the scheduled batch
  std::vector<int32_t> pages, prefix_len, branch_page, num_new, past_len, fork_len, request, tokens_in,
      prefill_from, prefill_to, preempted, admitted, page_seq, branch_seq, blocks, page_block0, branch_block0;

  ~hpd_sched() { hpd_kv_pool_destroy(pool); }
};

namespace {

hpd_status fail(hpd_status st, const std::string &msg) {
  hpd::set_last_error(msg);
  return st;
}

// AllocKV: room for the request's next step, len + k rows, all or nothing.
hpd_status alloc_kv(hpd_sched *s, Request &r) {
  return hpd_kv_seq_reserve(s->pool, r.seq, r.len + (int32_t)r.window.size());
}

// PartialFree: a child gives back its own rows (it keeps seeing the page); a
// parent keeps the page rows its live children see.  Dropped rows are
// recomputed when the request resumes.
hpd_status partial_free(hpd_sched *s, Request &v) {
  int32_t keep = 0;
  if (!v.child)
    for (int32_t c : v.live_children) keep = std::max(keep, s->reqs[c].fork_len);
  v.kept = std::min(v.kept, keep);
  return hpd_kv_seq_truncate(s->pool, v.seq, keep);
}

void sort_queue(hpd_sched *s) {
  auto key = [s](int32_t id) {
    const Request &r = s->reqs[id];
    if (r.child) {
      const Request &p = s->reqs[r.page];
      return std::make_tuple(0, p.id, -(int32_t)p.live_children.size(), r.id);
    }
    return std::make_tuple(1, r.id, 0, 0);
  };
  std::stable_sort(s->queue.begin(), s->queue.end(), [&](int32_t a, int32_t b) { return key(a) < key(b); });
}

hpd_status build_batch(hpd_sched *s) {
  // pages in order of their parent's arrival (= id); the parent first, then
  // its children by arrival
  std::vector<int32_t> order(s->active);
  std::sort(order.begin(), order.end(), [s](int32_t a, int32_t b) {
    const Request &x = s->reqs[a], &y = s->reqs[b];
    return std::make_tuple(x.page, x.child, x.id) < std::make_tuple(y.page, y.child, y.id);
  });
  s->pages.clear();
  s->prefix_len.clear();
  s->branch_page.clear();
  s->num_new.clear();
  s->past_len.clear();
  s->fork_len.clear();
  s->request.clear();
  s->tokens_in.clear();
  s->prefill_from.clear();
  s->prefill_to.clear();
  s->page_seq.clear();
  s->branch_seq.clear();
  for (int32_t id : order) {
    Request &r = s->reqs[id];
    if (s->pages.empty() || s->pages.back() != r.page) {
      s->pages.push_back(r.page);
      s->prefix_len.push_back(0);
      s->page_seq.push_back(s->reqs[r.page].seq);
    }
    if (r.child) s->prefix_len.back() = std::max(s->prefix_len.back(), r.fork_len);
    s->branch_page.push_back((int32_t)s->pages.size() - 1);
    s->num_new.push_back((int32_t)r.window.size());
    s->past_len.push_back(r.len);
    s->fork_len.push_back(r.child ? r.fork_len : 0);
    s->request.push_back(id);
    s->tokens_in.insert(s->tokens_in.end(), r.window.begin(), r.window.end());
    s->prefill_from.push_back(r.kept);
    s->prefill_to.push_back(r.len);
    s->branch_seq.push_back(r.seq);
  }
  s->page_block0.assign(s->pages.size(), 0);
  s->branch_block0.assign(order.size(), 0);
  int32_t n = 0;
  hpd_status st = hpd_kv_batch_tables(s->pool, (int32_t)s->pages.size(), s->page_seq.data(),
                                      (int32_t)order.size(), s->branch_seq.data(), nullptr, 0,
                                      s->page_block0.data(), s->branch_block0.data(), &n);
  if (st != HPD_OK && n == 0) return st;
  s->blocks.assign((size_t)std::max(n, 1), 0);
  st = hpd_kv_batch_tables(s->pool, (int32_t)s->pages.size(), s->page_seq.data(), (int32_t)order.size(),
                           s->branch_seq.data(), s->blocks.data(), n, s->page_block0.data(), s->branch_block0.data(),
                           &n);
  if (st != HPD_OK) return st;
  s->blocks.resize((size_t)n);
  for (int32_t id : order) s->reqs[id].kept = s->reqs[id].len;   // the caller computes the prefill rows first
  return HPD_OK;
}

void fill_out(const hpd_sched *s, hpd_sched_batch *out) {
  *out = hpd_sched_batch{};
  const bool any = !s->request.empty();
  out->num_pages = (int32_t)s->pages.size();
  out->num_branches = (int32_t)s->request.size();
  out->num_tokens = (int32_t)s->tokens_in.size();
  if (any) {
    out->prefix_len = s->prefix_len.data();
    out->branch_page = s->branch_page.data();
    out->num_new = s->num_new.data();
    out->past_len = s->past_len.data();
    out->fork_len = s->fork_len.data();
    out->request = s->request.data();
    out->tokens_in = s->tokens_in.data();
    out->prefill_from = s->prefill_from.data();
    out->prefill_to = s->prefill_to.data();
    out->paged.block_rows = s->cfg.block_rows;
    out->paged.num_blocks = s->cfg.num_blocks;
    out->paged.num_entries = (int32_t)s->blocks.size();
    out->paged.blocks = s->blocks.data();
    out->paged.page_block0 = s->page_block0.data();
    out->paged.branch_block0 = s->branch_block0.data();
  }
  out->num_preempted = (int32_t)s->preempted.size();
  out->preempted = s->preempted.empty() ? nullptr : s->preempted.data();
  out->num_admitted = (int32_t)s->admitted.size();
  out->admitted = s->admitted.empty() ? nullptr : s->admitted.data();
}

std::vector<int32_t> interleave(const hpd_sched *s, const Request &p) {
  std::vector<int32_t> o;
  size_t f = 0;
  for (size_t i = 0; i < p.out.size(); ++i) {
    o.push_back(p.out[i]);
    for (; f < p.forks.size() && p.forks[f].first == (int32_t)i; ++f) {
      const std::vector<int32_t> &c = s->reqs[p.forks[f].second].out;
      o.insert(o.end(), c.begin(), c.end());
    }
  }
  return o;
}

}  // namespace

extern "C" {

hpd_status hpd_sched_create(const hpd_sched_config *config, hpd_sched **out) {
  if (!config || !out) return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_create: NULL argument");
  *out = nullptr;
  const hpd_sched_config &c = *config;
  if (!(c.kv_threshold >= 0.0 && c.kv_threshold <= 1.0) || c.window < 1 || c.window > HPD_MAX_K ||
      c.max_active < 1)
    return fail(HPD_ERR_INVALID_ARGUMENT,
                "hpd_sched_create: need kv_threshold in [0, 1], window in 1..HPD_MAX_K and max_active >= 1");
  hpd_sched *s = nullptr;
  try {
    s = new hpd_sched;
  } catch (const std::bad_alloc &) {
    return fail(HPD_ERR_HOST_ALLOC, "hpd_sched_create: out of host memory");
  }
  s->cfg = c;
  const hpd_status st = hpd_kv_pool_create(c.num_blocks, c.block_rows, &s->pool);
  if (st != HPD_OK) {
    delete s;
    return st;
  }
  *out = s;
  return HPD_OK;
}

void hpd_sched_destroy(hpd_sched *sched) { delete sched; }

hpd_status hpd_sched_submit(hpd_sched *s, int32_t prompt_len, int32_t first_token, int32_t max_new,
                            int32_t *request) {
  if (!s || !request) return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_submit: NULL argument");
  if (prompt_len < 1 || max_new < 1)
    return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_submit: need prompt_len >= 1 and max_new >= 1");
  if (s->pending) return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_submit: a scheduled batch awaits its commit");
  int32_t seq = -1;
  hpd_status st = hpd_kv_seq_new(s->pool, -1, 0, &seq);
  if (st != HPD_OK) return st;
  try {
    Request r;
    r.id = (int32_t)s->reqs.size();
    r.page = r.id;
    r.max_new = max_new;
    r.len = prompt_len;
    r.seq = seq;
    r.window.assign(1, first_token);
    s->reqs.push_back(std::move(r));
    s->queue.push_back(s->reqs.back().id);
  } catch (const std::bad_alloc &) {
    hpd_kv_seq_release(s->pool, seq);
    return fail(HPD_ERR_HOST_ALLOC, "hpd_sched_submit: out of host memory");
  }
  *request = s->reqs.back().id;
  return HPD_OK;
}

hpd_status hpd_sched_schedule(hpd_sched *s, hpd_sched_batch *out) {
  if (!s || !out) return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_schedule: NULL argument");
  if (s->pending) return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_schedule: the last batch was not committed");
  try {
    s->preempted.clear();
    s->admitted.clear();
    if (s->queue_dirty) {   // FCFS order
      sort_queue(s);
      s->queue_dirty = false;
    }
    // K/V for every active request; preempt the youngest while it fails
    const std::vector<int32_t> snapshot(s->active);
    for (int32_t id : snapshot) {
      if (std::find(s->active.begin(), s->active.end(), id) == s->active.end()) continue;   // preempted
      for (;;) {
        hpd_status st = alloc_kv(s, s->reqs[id]);
        if (st == HPD_OK) break;
        if (st != HPD_ERR_OUT_OF_BLOCKS) return st;
        const int32_t v = *std::max_element(s->active.begin(), s->active.end());   // youngest: largest id
        if ((st = partial_free(s, s->reqs[v])) != HPD_OK) return st;
        s->active.erase(std::find(s->active.begin(), s->active.end(), v));
        s->reqs[v].state = kWaiting;
        s->queue.push_front(v);
        s->preempted.push_back(v);
        if (v == id) break;
      }
    }
    // admission: parents gated by K/V usage and concurrency, children bypass
    while (!s->queue.empty()) {
      Request &r = s->reqs[s->queue.front()];
      const int32_t used = s->cfg.num_blocks - hpd_kv_pool_free_blocks(s->pool);
      if (!r.child && ((double)used > s->cfg.kv_threshold * (double)s->cfg.num_blocks ||
                       (int32_t)s->active.size() >= s->cfg.max_active))
        break;
      const hpd_status st = alloc_kv(s, r);
      if (st == HPD_ERR_OUT_OF_BLOCKS) break;
      if (st != HPD_OK) return st;
      s->queue.pop_front();
      s->active.push_back(r.id);
      r.state = kActive;
      s->admitted.push_back(r.id);
    }
    const hpd_status st = build_batch(s);
    if (st != HPD_OK) return st;
  } catch (const std::bad_alloc &) {
    return fail(HPD_ERR_HOST_ALLOC, "hpd_sched_schedule: out of host memory");
  }
  s->pending = true;
  fill_out(s, out);
  return HPD_OK;
}

hpd_status hpd_sched_commit(hpd_sched *s, const int32_t *verified, const int32_t *n_acc,
                            const int32_t *draft_out) {
  if (!s) return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_commit: NULL scheduler");
  if (!s->pending) return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_commit: no scheduled batch");
  const size_t nb = s->request.size();
  if (nb && (!verified || !n_acc || !draft_out))
    return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_commit: NULL array");
  for (size_t b = 0; b < nb; ++b)
    if (n_acc[b] < 0 || n_acc[b] >= s->num_new[b])
      return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_commit: n_acc out of 0..num_new - 1");
  try {
    int32_t q = 0;
    for (size_t b = 0; b < nb; ++b) {
      const int32_t rid = s->request[b];   // by id: spawning a child may move the requests
      const int32_t n = n_acc[b], base = s->reqs[rid].len;
      {
        Request &r = s->reqs[rid];
        r.len = base + n + 1;   // the fed tokens s_0 .. s_n stay; the rest rolls back
        r.kept = r.len;
        const hpd_status st = hpd_kv_seq_truncate(s->pool, r.seq, r.len);
        if (st != HPD_OK) return st;
        r.window.assign(draft_out + (size_t)b * HPD_MAX_K, draft_out + (size_t)b * HPD_MAX_K + s->cfg.window);
      }
      for (int32_t i = 0; i <= n; ++i) {
        const int32_t t = verified[q + i];
        if (t == s->cfg.eos_token) {
          s->reqs[rid].state = kDone;
          break;
        }
        s->reqs[rid].out.push_back(t);
        if (t == s->cfg.fork_token && !s->reqs[rid].child) {   // the child sees the rows before the fork token
          const int32_t fork = base + i + 1;
          int32_t seq = -1;
          const hpd_status st = hpd_kv_seq_new(s->pool, s->reqs[rid].seq, fork, &seq);
          if (st != HPD_OK) return st;
          Request c;
          c.id = (int32_t)s->reqs.size();
          c.child = true;
          c.page = rid;
          c.max_new = s->reqs[rid].max_new;
          c.fork_len = fork;
          c.seq = seq;
          c.window.assign(1, s->cfg.child_token);
          const int32_t cid = c.id, at = (int32_t)s->reqs[rid].out.size() - 1;
          s->reqs.push_back(std::move(c));
          s->reqs[rid].forks.emplace_back(at, cid);
          s->reqs[rid].live_children.push_back(cid);
          s->queue.push_back(cid);
          s->queue_dirty = true;
        }
        if ((int32_t)s->reqs[rid].out.size() >= s->reqs[rid].max_new) {
          s->reqs[rid].state = kDone;
          break;
        }
      }
      q += s->num_new[b];
    }
    // reference-counted release; a page is output when its parent and all
    // of its children have finished
    const std::vector<int32_t> snapshot(s->active);
    for (int32_t id : snapshot) {
      Request &r = s->reqs[id];
      if (r.state != kDone) continue;
      s->active.erase(std::find(s->active.begin(), s->active.end(), id));
      hpd_status st = hpd_kv_seq_release(s->pool, r.seq);
      if (st != HPD_OK) return st;
      Request &p = s->reqs[r.page];
      if (r.child) p.live_children.erase(std::find(p.live_children.begin(), p.live_children.end(), id));
      if (p.state == kDone && p.live_children.empty() && !p.emitted) {
        p.emitted = true;
        s->finished.emplace_back(p.id, interleave(s, p));
      }
    }
  } catch (const std::bad_alloc &) {
    return fail(HPD_ERR_HOST_ALLOC, "hpd_sched_commit: out of host memory");
  }
  s->pending = false;
  return HPD_OK;
}

hpd_status hpd_sched_next_output(hpd_sched *s, int32_t *page, int32_t *tokens, int32_t capacity, int32_t *len) {
  if (!s || !page || !len) return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_next_output: NULL argument");
  if (s->finished.empty()) {
    *page = -1;
    *len = 0;
    return HPD_OK;
  }
  const auto &f = s->finished.front();
  *page = f.first;
  *len = (int32_t)f.second.size();
  if (capacity >= *len && (tokens || *len == 0)) {
    std::copy(f.second.begin(), f.second.end(), tokens);
    s->finished.pop_front();
  }
  return HPD_OK;
}

hpd_status hpd_sched_counts(const hpd_sched *s, int32_t *waiting, int32_t *active, int32_t *free_blocks) {
  if (!s) return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_counts: NULL scheduler");
  if (waiting) *waiting = (int32_t)s->queue.size();
  if (active) *active = (int32_t)s->active.size();
  if (free_blocks) *free_blocks = hpd_kv_pool_free_blocks(s->pool);
  return HPD_OK;
}

hpd_status hpd_sched_request(const hpd_sched *s, int32_t request, int32_t *state, int32_t *len, int32_t *kept,
                             int32_t *recorded) {
  if (!s || request < 0 || request >= (int32_t)s->reqs.size())
    return fail(HPD_ERR_INVALID_ARGUMENT, "hpd_sched_request: unknown request");
  const Request &r = s->reqs[request];
  if (state) *state = r.state;
  if (len) *len = r.len;
  if (kept) *kept = r.kept;
  if (recorded) *recorded = (int32_t)r.out.size();
  return HPD_OK;
}

}  // extern "C"
