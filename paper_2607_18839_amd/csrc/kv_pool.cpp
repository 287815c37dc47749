// Host manager of paged K/V blocks (C ABI in include/hpd.h): block ids of a
// pool, root sequences (a page's prefix) and branches forked from a root that
// see its first fork_len rows by reference (section "Inference Workflow",
// Algorithm 1: per-request KV shared by forked branches, rollback of
// rejected drafts).  Plain C++; no device memory is touched.
#include <algorithm>
#include <cstdint>
#include <new>
#include <string>
#include <vector>

#include "hpd.h"

namespace hpd {
void set_last_error(const std::string &msg);
}

struct hpd_kv_pool {
  struct Seq {
    bool live = false;       // not released
    bool holds = false;      // still owns its blocks (a released root with branches keeps them)
    int32_t parent = -1;     // root: -1
    int32_t fork_len = 0;    // branch: rows of the root it sees
    int32_t len = 0;
    int32_t branches = 0;    // root: live branches
    std::vector<int32_t> blocks;
  };
  int32_t num_blocks = 0, block_rows = 0;
  std::vector<int32_t> free_list;   // stack: last freed is reused first
  std::vector<Seq> seqs;
  std::vector<int32_t> free_ids;

  int64_t blocks_for(int64_t rows) const { return (rows + block_rows - 1) / block_rows; }
  // Returns the blocks of a released root that no live branch sees any more
  // (a block is freed when its last reference goes, as with per-block
  // reference counts).
  void trim_released_root(int32_t id) {
    int32_t need = 0;
    for (const Seq &c : seqs)
      if (c.live && c.parent == id) need = std::max(need, c.fork_len);
    Seq &r = seqs[id];
    const size_t keep = (size_t)blocks_for(need);
    while (r.blocks.size() > keep) {
      free_list.push_back(r.blocks.back());
      r.blocks.pop_back();
    }
    r.len = std::min(r.len, need);
  }
  void give_back(Seq &s) {
    for (auto it = s.blocks.rbegin(); it != s.blocks.rend(); ++it) free_list.push_back(*it);
    s.blocks.clear();
    s.holds = false;
  }
};

namespace {

hpd_status err(hpd_status st, const std::string &msg) {
  hpd::set_last_error(msg);
  return st;
}

bool live_seq(const hpd_kv_pool *p, int32_t s) {
  return p && s >= 0 && s < (int32_t)p->seqs.size() && p->seqs[s].live;
}

// Live, or a released root still holding blocks for its live branches.
bool holding_seq(const hpd_kv_pool *p, int32_t s) {
  return p && s >= 0 && s < (int32_t)p->seqs.size() && (p->seqs[s].live || p->seqs[s].holds);
}

}  // namespace

extern "C" {

hpd_status hpd_kv_pool_create(int32_t num_blocks, int32_t block_rows, hpd_kv_pool **out) {
  if (!out) return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_pool_create: out is NULL");
  *out = nullptr;
  if (num_blocks <= 0 || block_rows <= 0 || block_rows % 64 != 0 ||
      (int64_t)num_blocks * block_rows > INT32_MAX)
    return err(HPD_ERR_INVALID_ARGUMENT,
               "hpd_kv_pool_create: need num_blocks > 0, block_rows a positive multiple of 64 and "
               "num_blocks * block_rows < 2^31");
  try {
    hpd_kv_pool *p = new hpd_kv_pool;
    p->num_blocks = num_blocks;
    p->block_rows = block_rows;
    p->free_list.reserve(num_blocks);
    for (int32_t b = num_blocks - 1; b >= 0; --b) p->free_list.push_back(b);   // block 0 is handed out first
    *out = p;
  } catch (const std::bad_alloc &) {
    return err(HPD_ERR_HOST_ALLOC, "hpd_kv_pool_create: out of host memory");
  }
  return HPD_OK;
}

void hpd_kv_pool_destroy(hpd_kv_pool *pool) { delete pool; }

int32_t hpd_kv_pool_free_blocks(const hpd_kv_pool *pool) {
  return pool ? (int32_t)pool->free_list.size() : 0;
}

hpd_status hpd_kv_seq_new(hpd_kv_pool *pool, int32_t parent, int32_t fork_len, int32_t *seq) {
  if (!pool || !seq) return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_new: NULL argument");
  if (parent != -1) {
    if (!live_seq(pool, parent) || pool->seqs[parent].parent != -1)
      return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_new: parent must be a live root sequence");
    if (fork_len < 0 || fork_len > pool->seqs[parent].len)
      return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_new: fork_len must be in 0..parent length");
  } else if (fork_len != 0) {
    return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_new: a root has fork_len 0");
  }
  try {
    int32_t id;
    if (!pool->free_ids.empty()) {
      id = pool->free_ids.back();
      pool->free_ids.pop_back();
    } else {
      id = (int32_t)pool->seqs.size();
      pool->seqs.emplace_back();
    }
    hpd_kv_pool::Seq &s = pool->seqs[id];
    s = hpd_kv_pool::Seq{};
    s.live = s.holds = true;
    s.parent = parent;
    s.fork_len = fork_len;
    if (parent != -1) ++pool->seqs[parent].branches;
    *seq = id;
  } catch (const std::bad_alloc &) {
    return err(HPD_ERR_HOST_ALLOC, "hpd_kv_seq_new: out of host memory");
  }
  return HPD_OK;
}

hpd_status hpd_kv_seq_reserve(hpd_kv_pool *pool, int32_t seq, int32_t new_len) {
  if (!live_seq(pool, seq)) return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_reserve: not a live sequence");
  hpd_kv_pool::Seq &s = pool->seqs[seq];
  if (new_len < s.len) return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_reserve: new_len below the length");
  const int64_t need = pool->blocks_for(new_len) - (int64_t)s.blocks.size();
  if (need > (int64_t)pool->free_list.size())
    return err(HPD_ERR_OUT_OF_BLOCKS, "hpd_kv_seq_reserve: needs " + std::to_string(need) + " blocks, " +
                                          std::to_string(pool->free_list.size()) + " free");
  try {
    s.blocks.reserve(s.blocks.size() + (size_t)std::max<int64_t>(need, 0));
  } catch (const std::bad_alloc &) {
    return err(HPD_ERR_HOST_ALLOC, "hpd_kv_seq_reserve: out of host memory");
  }
  for (int64_t i = 0; i < need; ++i) {
    s.blocks.push_back(pool->free_list.back());
    pool->free_list.pop_back();
  }
  s.len = new_len;
  return HPD_OK;
}

hpd_status hpd_kv_seq_truncate(hpd_kv_pool *pool, int32_t seq, int32_t new_len) {
  if (!live_seq(pool, seq)) return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_truncate: not a live sequence");
  hpd_kv_pool::Seq &s = pool->seqs[seq];
  if (new_len < 0 || new_len > s.len)
    return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_truncate: new_len must be in 0..length");
  if (s.parent == -1)
    for (const hpd_kv_pool::Seq &c : pool->seqs)
      if (c.live && c.parent == seq && c.fork_len > new_len)
        return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_truncate: a live branch sees rows past new_len");
  const size_t keep = (size_t)pool->blocks_for(new_len);
  while (s.blocks.size() > keep) {
    pool->free_list.push_back(s.blocks.back());
    s.blocks.pop_back();
  }
  s.len = new_len;
  return HPD_OK;
}

hpd_status hpd_kv_seq_release(hpd_kv_pool *pool, int32_t seq) {
  if (!live_seq(pool, seq)) return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_release: not a live sequence");
  hpd_kv_pool::Seq &s = pool->seqs[seq];
  s.live = false;
  auto retire = [&](int32_t id) {   // a released sequence that no branch needs any more
    pool->give_back(pool->seqs[id]);
    pool->free_ids.push_back(id);
  };
  if (s.parent != -1) {
    hpd_kv_pool::Seq &root = pool->seqs[s.parent];
    const int32_t parent = s.parent;
    retire(seq);
    if (--root.branches == 0 && !root.live) retire(parent);
    else if (!root.live) pool->trim_released_root(parent);
  } else if (s.branches == 0) {
    retire(seq);
  } else {
    pool->trim_released_root(seq);
  }
  return HPD_OK;
}

hpd_status hpd_kv_seq_info(const hpd_kv_pool *pool, int32_t seq, int32_t *len, int32_t *num_blocks,
                           int32_t *parent, int32_t *fork_len) {
  if (!live_seq(pool, seq)) return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_info: not a live sequence");
  const hpd_kv_pool::Seq &s = pool->seqs[seq];
  if (len) *len = s.len;
  if (num_blocks) *num_blocks = (int32_t)s.blocks.size();
  if (parent) *parent = s.parent;
  if (fork_len) *fork_len = s.fork_len;
  return HPD_OK;
}

hpd_status hpd_kv_seq_blocks(const hpd_kv_pool *pool, int32_t seq, int32_t *blocks_out, int32_t capacity) {
  if (!live_seq(pool, seq)) return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_blocks: not a live sequence");
  const hpd_kv_pool::Seq &s = pool->seqs[seq];
  if (capacity < (int32_t)s.blocks.size() || (!blocks_out && !s.blocks.empty()))
    return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_seq_blocks: capacity below the block count");
  std::copy(s.blocks.begin(), s.blocks.end(), blocks_out);
  return HPD_OK;
}

hpd_status hpd_kv_batch_tables(const hpd_kv_pool *pool, int32_t num_pages, const int32_t *page_seq,
                               int32_t num_branches, const int32_t *branch_seq, int32_t *blocks_out,
                               int32_t capacity, int32_t *page_block0_out, int32_t *branch_block0_out,
                               int32_t *entries) {
  if (!pool || !entries || num_pages < 0 || num_branches < 0 || (num_pages && (!page_seq || !page_block0_out)) ||
      (num_branches && (!branch_seq || !branch_block0_out)))
    return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_batch_tables: NULL argument or negative count");
  int64_t n = 0;
  for (int32_t i = 0; i < num_pages + num_branches; ++i) {
    const int32_t id = i < num_pages ? page_seq[i] : branch_seq[i - num_pages];
    if (i < num_pages ? !holding_seq(pool, id) : !live_seq(pool, id))
      return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_batch_tables: not a live sequence");
    n += (int64_t)pool->seqs[id].blocks.size();
  }
  if (n > INT32_MAX) return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_batch_tables: too many entries");
  *entries = (int32_t)n;
  if (n > capacity || (n > 0 && !blocks_out))
    return err(HPD_ERR_INVALID_ARGUMENT, "hpd_kv_batch_tables: capacity below the entries needed");
  int32_t at = 0;
  for (int32_t i = 0; i < num_pages + num_branches; ++i) {
    const int32_t id = i < num_pages ? page_seq[i] : branch_seq[i - num_pages];
    if (i < num_pages) page_block0_out[i] = at;
    else branch_block0_out[i - num_pages] = at;
    for (int32_t b : pool->seqs[id].blocks) blocks_out[at++] = b;
  }
  return HPD_OK;
}

}  // extern "C"
