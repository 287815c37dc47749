// Randomised stress of the host-side C++ (the planner, the paged K/V pool and
// the Algorithm 1 scheduler) for runs under AddressSanitizer and UBSan:
// tests/test_host_sanitize.py builds this file with the three sources.
// Inputs are random, valid and invalid; every result is checked against
// invariants that hold for any correct implementation:
//   planner    T = sum k_b, q_row and visible counts by their definitions,
//              each token's slot range inside the partial slots;
//   K/V pool   no block held by two live sequences, the free count equal to
//              the blocks not held, the whole pool back after releasing all;
//   scheduler  every batch it returns is a valid planner input (block ids in
//              range, tables long enough) and a rejected commit changes
//              nothing.
// Usage: host_stress SEED ITERATIONS.  Exit 0 = every check held.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <set>
#include <string>
#include <vector>

#include "hpd.h"
#include "plan.h"

// The library's error sink lives with the HIP entry points (not built here):
// this stand-in keeps the last message so rejected calls can be checked for one.
namespace hpd {
std::string g_stress_last_error;
void set_last_error(const std::string &msg) { g_stress_last_error = msg; }
}  // namespace hpd

namespace {

uint64_t g_seed = 0;
int g_iter = 0;
// what the run exercised (printed at the end, so a run that tests nothing shows)
long g_plans_ok = 0, g_plans_rejected = 0, g_batches = 0, g_branches = 0, g_pages = 0, g_pool_ops = 0;

#define CHECK(c)                                                                                     \
  do {                                                                                               \
    if (!(c)) {                                                                                      \
      std::fprintf(stderr, "check failed at line %d: %s (seed %llu, iteration %d)\n", __LINE__, #c, \
                   (unsigned long long)g_seed, g_iter);                                              \
      std::exit(1);                                                                                  \
    }                                                                                                \
  } while (0)

struct Rng {   // splitmix64
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
  }
  int range(int lo, int hi) { return lo + (int)(next() % (uint64_t)(hi - lo + 1)); }   // inclusive
  bool pct(int p) { return range(0, 99) < p; }
};

int ceil_div(int a, int b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------- planner

void stress_plan(Rng &r) {
  // A valid batch; a quarter of them then get exactly one defect that makes
  // them invalid, which the planner must reject (and accept all others).
  enum { NONE, NO_PAGES, HEAD_DIM, NUM_NEW_0, NUM_NEW_BIG, PAST_NEG, FORK_BIG, PAGE_ORDER, BLOCK_ID, TABLE_SHORT,
         ROW_NEG, NUM_DEFECTS };
  const int defect = r.pct(75) ? NONE : r.range(1, NUM_DEFECTS - 1);
  hpd_attn_desc a{};
  const int G = 1 << r.range(0, 3);
  a.num_kv_heads = r.range(1, 4);
  a.num_q_heads = a.num_kv_heads * G;
  a.head_dim = defect == HEAD_DIM ? 32 : 64;
  a.softmax_scale = 0.f;
  a.dtype = a.out_dtype = r.range(0, 1);

  const int np = defect == NO_PAGES ? 0 : r.range(1, 4);
  std::vector<int32_t> prefix(np), page, num_new, past, fork;
  for (int p = 0; p < np; ++p) {
    prefix[p] = r.pct(10) ? 0 : r.range(1, 5000);
    const int n = r.range(p == 0 ? 1 : 0, 12);
    for (int i = 0; i < n; ++i) {
      page.push_back(p);
      num_new.push_back(r.range(1, HPD_MAX_K));
      past.push_back(r.range(0, 1500));
      fork.push_back(r.range(0, prefix[p]));
    }
  }
  const int nb = (int)page.size();
  const bool use_fork = defect == FORK_BIG || r.pct(50);
  bool invalid = defect == NO_PAGES || defect == HEAD_DIM;
  if (nb > 0) {
    const int i = r.range(0, nb - 1);
    if (defect == NUM_NEW_0) num_new[i] = 0, invalid = true;
    if (defect == NUM_NEW_BIG) num_new[i] = HPD_MAX_K + 1, invalid = true;
    if (defect == PAST_NEG) past[i] = -1, invalid = true;
    if (defect == FORK_BIG) fork[i] = prefix[page[i]] + 1, invalid = true;
    if (defect == PAGE_ORDER && page.front() != page.back()) std::swap(page.front(), page.back()), invalid = true;
  }

  hpd_batch_desc b{};
  b.num_pages = np;
  b.prefix_len = prefix.data();
  b.num_branches = nb;
  b.branch_page = page.data();
  b.num_new = num_new.data();
  b.past_len = past.data();
  b.fork_len = use_fork ? fork.data() : nullptr;

  std::vector<int32_t> blocks, page0(np), branch0(nb);
  std::vector<int64_t> prefix_row(np), priv_row(nb);
  hpd_paged_kv pg{};
  const bool paged = defect == BLOCK_ID || defect == TABLE_SHORT || (defect != ROW_NEG && r.pct(40));
  if (paged) {   // random block ids, each sequence's entries in order
    pg.block_rows = 64 << r.range(0, 2);
    pg.num_blocks = r.range(1, 4096);
    auto add = [&](int rows) {
      const int first = (int)blocks.size();
      for (int e = 0; e < ceil_div(std::max(rows, 0), pg.block_rows); ++e) blocks.push_back(r.range(0, pg.num_blocks - 1));
      return first;
    };
    for (int p = 0; p < np; ++p) page0[p] = add(prefix[p]);
    for (int i = 0; i < nb; ++i) branch0[i] = add(past[i] + num_new[i]);
    if (!blocks.empty() && !invalid) {
      if (defect == BLOCK_ID) blocks[r.range(0, (int)blocks.size() - 1)] = pg.num_blocks, invalid = true;
      if (defect == TABLE_SHORT) blocks.pop_back(), invalid = true;
    }
    pg.num_entries = (int)blocks.size();
    pg.blocks = blocks.data();
    pg.page_block0 = page0.data();
    pg.branch_block0 = branch0.data();
    b.paged = &pg;
  } else if (defect == ROW_NEG || r.pct(50)) {   // explicit rows with gaps
    int64_t row = 0;
    for (int p = 0; p < np; ++p) prefix_row[p] = (row += r.range(0, 100)), row += prefix[p];
    row = 0;
    for (int i = 0; i < nb; ++i) priv_row[i] = (row += r.range(0, 100)), row += past[i] + num_new[i];
    if (defect == ROW_NEG && np > 0 && !invalid) prefix_row[r.range(0, np - 1)] = -5, invalid = true;
    b.prefix_row = prefix_row.data();
    b.priv_row = priv_row.data();
  }

  hpd::Plan P;
  std::string err;
  const hpd_status st = hpd::build_plan(&a, &b, &P, &err);
  if (invalid) {
    if (st == HPD_OK) std::fprintf(stderr, "defect %d accepted\n", defect);
    CHECK(st != HPD_OK && !err.empty());
    ++g_plans_rejected;
    return;
  }
  if (st != HPD_OK) std::fprintf(stderr, "valid batch rejected: %s\n", err.c_str());
  CHECK(st == HPD_OK);
  ++g_plans_ok;
  int T = 0;
  for (int i = 0; i < nb; ++i) {
    CHECK(P.q_row[i] == T);
    const int F = use_fork ? fork[i] : prefix[page[i]];
    for (int j = 0; j < num_new[i]; ++j) CHECK(P.visible[T + j] == F + past[i] + j + 1);
    T += num_new[i];
  }
  CHECK(P.T == T && (int)P.token_slots.size() == 2 * T);
  for (int t = 0; t < T; ++t) CHECK(P.token_slots[2 * t] >= 0 && P.token_slots[2 * t + 1] >= 1);
}

// ---------------------------------------------------------------- K/V pool

void stress_pool(Rng &r) {
  const int nblk = r.range(1, 64), B = 64 << r.range(0, 1);
  hpd_kv_pool *pool = nullptr;
  CHECK(hpd_kv_pool_create(nblk, B, &pool) == HPD_OK && pool);
  struct Seq { int id, parent; };
  std::vector<Seq> live;
  std::set<int> zombie_roots;   // released roots whose branches still live
  for (int op = 0; op < 300; ++op) {
    ++g_pool_ops;
    const int kind = r.range(0, 6);
    if (kind == 0 || live.empty()) {   // a new root, or a branch of a live root
      std::vector<int> roots;
      for (auto &s : live) if (s.parent < 0) roots.push_back(s.id);
      int32_t id = -1;
      if (roots.empty() || r.pct(40)) {
        CHECK(hpd_kv_seq_new(pool, -1, 0, &id) == HPD_OK);
        live.push_back({id, -1});
      } else {
        const int root = roots[r.range(0, (int)roots.size() - 1)];
        int32_t len, nb, par, fl;
        CHECK(hpd_kv_seq_info(pool, root, &len, &nb, &par, &fl) == HPD_OK && par == -1);
        const int f = r.pct(5) ? len + 1 : r.range(0, len);
        const hpd_status st = hpd_kv_seq_new(pool, root, f, &id);
        CHECK((st == HPD_OK) == (f <= len));
        if (st == HPD_OK) live.push_back({id, root});
      }
    } else {
      const int k = r.range(0, (int)live.size() - 1);
      const int id = live[k].id;
      int32_t len, nb, par, fl;
      CHECK(hpd_kv_seq_info(pool, id, &len, &nb, &par, &fl) == HPD_OK && nb == ceil_div(len, B));
      if (kind <= 2) {
        const int before = hpd_kv_pool_free_blocks(pool);
        const int want = len + r.range(0, 3 * B);
        const hpd_status st = hpd_kv_seq_reserve(pool, id, want);
        CHECK(st == HPD_OK || st == HPD_ERR_OUT_OF_BLOCKS);
        if (st != HPD_OK) CHECK(hpd_kv_pool_free_blocks(pool) == before);
      } else if (kind <= 4) {
        const hpd_status st = hpd_kv_seq_truncate(pool, id, r.range(0, len));
        CHECK(st == HPD_OK || (par == -1 && st == HPD_ERR_INVALID_ARGUMENT));   // below a branch's fork
      } else {
        bool has_kids = false;
        for (auto &s : live) has_kids |= s.parent == id;
        CHECK(hpd_kv_seq_release(pool, id) == HPD_OK);
        hpd::g_stress_last_error.clear();
        CHECK(hpd_kv_seq_release(pool, id) != HPD_OK);   // no longer live
        CHECK(!hpd::g_stress_last_error.empty());
        if (has_kids) zombie_roots.insert(id);
        live.erase(live.begin() + k);
        for (auto it = zombie_roots.begin(); it != zombie_roots.end();) {
          bool kids = false;
          for (auto &s : live) kids |= s.parent == *it;
          it = kids ? std::next(it) : zombie_roots.erase(it);
        }
      }
    }
    // blocks are never shared between live sequences; the free count adds up
    std::set<int> held;
    size_t total = 0;
    for (auto &s : live) {
      int32_t len, nb, par, fl;
      CHECK(hpd_kv_seq_info(pool, s.id, &len, &nb, &par, &fl) == HPD_OK);
      std::vector<int32_t> ids(nb + 1, -1);
      CHECK(hpd_kv_seq_blocks(pool, s.id, ids.data(), nb) == HPD_OK);
      for (int e = 0; e < nb; ++e) {
        CHECK(ids[e] >= 0 && ids[e] < nblk);
        held.insert(ids[e]);
      }
      CHECK(ids[nb] == -1);   // capacity respected
      total += nb;
    }
    CHECK(held.size() == total);
    const int free_now = hpd_kv_pool_free_blocks(pool);
    CHECK(free_now >= 0 && free_now + (int)held.size() <= nblk);
    if (zombie_roots.empty()) CHECK(free_now + (int)held.size() == nblk);
  }
  // release branches first, then roots: everything returns
  std::stable_sort(live.begin(), live.end(), [](const Seq &x, const Seq &y) { return x.parent > y.parent; });
  for (auto &s : live) CHECK(hpd_kv_seq_release(pool, s.id) == HPD_OK);
  CHECK(hpd_kv_pool_free_blocks(pool) == nblk);
  hpd_kv_pool_destroy(pool);
}

// ---------------------------------------------------------------- scheduler

void stress_sched(Rng &r) {
  constexpr int FORK = 5, CHILD = 6, EOS = 7;
  hpd_sched_config c{};
  c.num_blocks = r.range(4, 256);
  c.block_rows = 64;
  c.kv_threshold = r.range(50, 100) / 100.0;
  c.window = r.range(1, 4);
  c.max_active = r.range(1, 16);
  c.fork_token = FORK;
  c.child_token = CHILD;
  c.eos_token = EOS;
  hpd_sched *s = nullptr;
  CHECK(hpd_sched_create(&c, &s) == HPD_OK && s);
  int submitted = 0;
  auto submit = [&]() {
    int32_t id = -1;
    if (hpd_sched_submit(s, r.range(1, 500), r.range(8, 100), r.range(1, 40), &id) == HPD_OK) {
      CHECK(id >= 0);
      ++submitted;
    }
  };
  for (int i = r.range(1, 6); i > 0; --i) submit();
  hpd_attn_desc a{16, 2, 64, 0.f, HPD_BF16, HPD_BF16};
  int idle = 0;
  for (int it = 0; it < 400 && idle < 3; ++it) {
    if (r.pct(3)) submit();
    hpd_sched_batch bt{};
    CHECK(hpd_sched_schedule(s, &bt) == HPD_OK);
    const int nb = bt.num_branches, T = bt.num_tokens;
    if (nb == 0) {
      CHECK(hpd_sched_commit(s, nullptr, nullptr, nullptr) == HPD_OK);
      ++idle;
    } else {
      idle = 0;
      ++g_batches;
      g_branches += nb;
      // the batch is a valid planner input over the scheduler's own pool
      for (int e = 0; e < bt.paged.num_entries; ++e) CHECK(bt.paged.blocks[e] >= 0 && bt.paged.blocks[e] < c.num_blocks);
      hpd_batch_desc b{};
      b.num_pages = bt.num_pages;
      b.prefix_len = bt.prefix_len;
      b.num_branches = nb;
      b.branch_page = bt.branch_page;
      b.num_new = bt.num_new;
      b.past_len = bt.past_len;
      b.fork_len = bt.fork_len;
      b.paged = &bt.paged;
      hpd::Plan P;
      std::string err;
      const hpd_status pst = hpd::build_plan(&a, &b, &P, &err);
      if (pst != HPD_OK) std::fprintf(stderr, "plan of a scheduled batch: %s\n", err.c_str());
      CHECK(pst == HPD_OK && P.T == T);
      for (int i = 0; i < nb; ++i) CHECK(bt.prefill_from[i] <= bt.prefill_to[i]);
      std::vector<int32_t> verified(T), n_acc(nb), drafts((size_t)nb * HPD_MAX_K);
      for (auto &v : verified) v = r.pct(8) ? FORK : r.pct(3) ? EOS : r.range(8, 100);
      for (auto &d : drafts) d = r.pct(5) ? FORK : r.range(8, 100);
      for (int i = 0; i < nb; ++i) n_acc[i] = r.range(0, bt.num_new[i] - 1);
      if (r.pct(5)) {   // a rejected commit leaves everything as it was
        int32_t w0, a0, f0, w1, a1, f1;
        CHECK(hpd_sched_counts(s, &w0, &a0, &f0) == HPD_OK);
        std::vector<int32_t> bad = n_acc;
        bad[r.range(0, nb - 1)] = r.pct(50) ? -1 : HPD_MAX_K + 1;
        hpd::g_stress_last_error.clear();
        CHECK(hpd_sched_commit(s, verified.data(), bad.data(), drafts.data()) == HPD_ERR_INVALID_ARGUMENT);
        CHECK(!hpd::g_stress_last_error.empty());
        CHECK(hpd_sched_counts(s, &w1, &a1, &f1) == HPD_OK && w0 == w1 && a0 == a1 && f0 == f1);
      }
      CHECK(hpd_sched_commit(s, verified.data(), n_acc.data(), drafts.data()) == HPD_OK);
    }
    for (;;) {   // take every finished page
      int32_t page = -1, len = 0;
      CHECK(hpd_sched_next_output(s, &page, nullptr, 0, &len) == HPD_OK);
      if (page < 0) break;
      ++g_pages;
      if (len == 0) continue;   // an empty page is taken by the length query itself
      std::vector<int32_t> toks(len + 1, -1);
      CHECK(hpd_sched_next_output(s, &page, toks.data(), len, &len) == HPD_OK);
      CHECK(toks[len] == -1);
      for (int i = 0; i < len; ++i) CHECK(toks[i] != EOS);
    }
    int32_t w, act, fr;
    CHECK(hpd_sched_counts(s, &w, &act, &fr) == HPD_OK && fr >= 0 && fr <= c.num_blocks);
    if (w == 0 && act == 0) CHECK(fr == c.num_blocks);
  }
  (void)submitted;
  hpd_sched_destroy(s);
}

}  // namespace

int main(int argc, char **argv) {
  if (argc != 3) {
    std::fprintf(stderr, "usage: host_stress SEED ITERATIONS\n");
    return 2;
  }
  g_seed = std::strtoull(argv[1], nullptr, 10);
  const int iters = std::atoi(argv[2]);
  Rng r{g_seed * 0x2545f4914f6cdd1dull + 1};
  for (g_iter = 0; g_iter < iters; ++g_iter) {
    stress_plan(r);
    if (g_iter % 8 == 0) stress_pool(r);
    if (g_iter % 16 == 0) stress_sched(r);
  }
  std::printf("host_stress seed %llu: %d iterations ok; plans %ld accepted, %ld rejected; pool ops %ld; "
              "scheduled batches %ld (%ld branches), pages output %ld\n",
              (unsigned long long)g_seed, iters, g_plans_ok, g_plans_rejected, g_pool_ops, g_batches, g_branches,
              g_pages);
  return 0;
}
