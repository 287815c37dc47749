// Host planner of the branch-parallel decode step (plain C++17, no HIP).
//
// Turns a ragged batch description into the canonical bookkeeping of one step
// and the work lists of the attention kernels.  The method batches every
// active branch of every page into one forward (Algorithm 1, the parallel
// draft over the active pool); each branch sees its page's shared prefix and
// its own rows only (section "Layout-Coordinated Parallel Decoding",
// paragraph "Dynamic Branch Forking and Efficient Context Isolation"), and its
// k drafts are causal among themselves (section "Integration with P-MTP").
//
// Partial softmax slots: every (token, query head) output row receives one
// partial (O, lse) per shared key split of its page and one per private key
// chunk of its branch.  token_slots[t] = (first slot, slot count); partial row
// index = (first + i) * Hq + h.  The merge kernel reduces them.
#include "plan.h"

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>

namespace hpd {
namespace {

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

hpd_status fail(std::string *err, hpd_status st, const std::string &msg) {
  if (err) *err = msg;
  return st;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

hpd_status build_plan(const hpd_attn_desc *attn, const hpd_batch_desc *batch, Plan *out,
                      std::string *err) {
  if (!attn || !batch || !out) return fail(err, HPD_ERR_INVALID_ARGUMENT, "NULL descriptor");
  const hpd_attn_desc &a = *attn;
  if (a.head_dim != HPD_HEAD_DIM)
    return fail(err, HPD_ERR_UNSUPPORTED, "head_dim must be 64, got " + std::to_string(a.head_dim));
  if (a.num_q_heads < 1 || a.num_q_heads > HPD_MAX_Q_HEADS)
    return fail(err, HPD_ERR_INVALID_ARGUMENT, "num_q_heads out of range");
  if (a.num_kv_heads < 1 || a.num_q_heads % a.num_kv_heads != 0)
    return fail(err, HPD_ERR_INVALID_ARGUMENT, "num_q_heads must be a positive multiple of num_kv_heads");
  if (a.num_q_heads / a.num_kv_heads > HPD_MAX_GROUP)
    return fail(err, HPD_ERR_UNSUPPORTED, "num_q_heads / num_kv_heads exceeds HPD_MAX_GROUP");
  if ((a.dtype != HPD_F32 && a.dtype != HPD_BF16) || (a.out_dtype != HPD_F32 && a.out_dtype != HPD_BF16))
    return fail(err, HPD_ERR_INVALID_ARGUMENT, "dtype / out_dtype must be HPD_F32 or HPD_BF16");
  if (std::isnan(a.softmax_scale) || std::isinf(a.softmax_scale))
    return fail(err, HPD_ERR_INVALID_ARGUMENT, "softmax_scale is not finite");

  const hpd_batch_desc &b = *batch;
  if (b.num_pages < 1) return fail(err, HPD_ERR_INVALID_ARGUMENT, "num_pages must be >= 1");
  if (b.num_branches < 1) return fail(err, HPD_ERR_INVALID_ARGUMENT, "num_branches must be >= 1");
  if (!b.prefix_len || !b.branch_page || !b.num_new || !b.past_len)
    return fail(err, HPD_ERR_INVALID_ARGUMENT, "NULL required batch array");

  Plan P;
  P.attn = a;
  P.G = a.num_q_heads / a.num_kv_heads;
  P.scale = a.softmax_scale > 0.f ? a.softmax_scale : 1.0f / std::sqrt((float)a.head_dim);
  P.num_pages = b.num_pages;
  P.num_branches = b.num_branches;
  const int np = b.num_pages, nb = b.num_branches, Hq = a.num_q_heads, Hkv = a.num_kv_heads,
            G = P.G;

  P.prefix_len.assign(b.prefix_len, b.prefix_len + np);
  P.branch_page.assign(b.branch_page, b.branch_page + nb);
  P.num_new.assign(b.num_new, b.num_new + nb);
  P.past_len.assign(b.past_len, b.past_len + nb);

  // ---- validation of the ragged structure
  for (int p = 0; p < np; ++p)
    if (P.prefix_len[p] < 0)
      return fail(err, HPD_ERR_INVALID_ARGUMENT, "prefix_len[" + std::to_string(p) + "] < 0");
  for (int i = 0; i < nb; ++i) {
    const std::string at = "[" + std::to_string(i) + "]";
    if (P.branch_page[i] < 0 || P.branch_page[i] >= np)
      return fail(err, HPD_ERR_INVALID_ARGUMENT, "branch_page" + at + " out of range");
    if (i > 0 && P.branch_page[i] < P.branch_page[i - 1])
      return fail(err, HPD_ERR_INVALID_ARGUMENT, "branch_page must be non-decreasing");
    if (P.num_new[i] < 1 || P.num_new[i] > HPD_MAX_K)
      return fail(err, HPD_ERR_INVALID_ARGUMENT, "num_new" + at + " must be in 1..HPD_MAX_K");
    if (P.past_len[i] < 0) return fail(err, HPD_ERR_INVALID_ARGUMENT, "past_len" + at + " < 0");
  }
  P.fork.resize(nb);
  P.has_fork = b.fork_len != nullptr;
  for (int i = 0; i < nb; ++i) {
    const int Pp = P.prefix_len[P.branch_page[i]];
    int F = Pp;
    if (b.fork_len) {
      F = b.fork_len[i];
      if (F < 0 || F > Pp)
        return fail(err, HPD_ERR_INVALID_ARGUMENT,
                    "fork_len[" + std::to_string(i) + "] must be in 0..prefix_len of its page");
    }
    P.fork[i] = F;
  }

  // ---- paged K/V: validation
  const hpd_paged_kv *pg = b.paged;
  if (pg) {
    if (b.prefix_row || b.priv_row)
      return fail(err, HPD_ERR_INVALID_ARGUMENT, "paged K/V: prefix_row and priv_row must be NULL");
    if (pg->block_rows <= 0 || pg->block_rows % 64 != 0)
      return fail(err, HPD_ERR_INVALID_ARGUMENT, "paged K/V: block_rows must be a positive multiple of 64");
    if (pg->num_blocks <= 0 || (int64_t)pg->num_blocks * pg->block_rows > INT32_MAX)
      return fail(err, HPD_ERR_INVALID_ARGUMENT, "paged K/V: num_blocks * block_rows must be in 1..2^31 - 1");
    if (pg->num_entries < 0 || (pg->num_entries > 0 && !pg->blocks) || !pg->page_block0 || !pg->branch_block0)
      return fail(err, HPD_ERR_INVALID_ARGUMENT, "paged K/V: NULL table");
    for (int32_t e = 0; e < pg->num_entries; ++e)
      if (pg->blocks[e] < 0 || pg->blocks[e] >= pg->num_blocks)
        return fail(err, HPD_ERR_INVALID_ARGUMENT, "paged K/V: block id out of range");
    auto span_ok = [&](int32_t first, int64_t rows) {
      const int64_t n = (rows + pg->block_rows - 1) / pg->block_rows;
      return first >= 0 && first + n <= pg->num_entries;
    };
    for (int p = 0; p < np; ++p)
      if (!span_ok(pg->page_block0[p], P.prefix_len[p]))
        return fail(err, HPD_ERR_INVALID_ARGUMENT, "paged K/V: page_block0[" + std::to_string(p) + "] out of range");
    for (int i = 0; i < nb; ++i)
      if (!span_ok(pg->branch_block0[i], (int64_t)P.past_len[i] + P.num_new[i]))
        return fail(err, HPD_ERR_INVALID_ARGUMENT, "paged K/V: branch_block0[" + std::to_string(i) + "] out of range");
  }

  // ---- canonical bookkeeping
  P.prefix_row.resize(np);
  int64_t acc = 0;
  for (int p = 0; p < np; ++p) {
    P.prefix_row[p] = b.prefix_row ? b.prefix_row[p] : acc;
    if (P.prefix_row[p] < 0) return fail(err, HPD_ERR_INVALID_ARGUMENT, "prefix_row < 0");
    acc += P.prefix_len[p];
    P.shared_rows = std::max<int64_t>(P.shared_rows, P.prefix_row[p] + P.prefix_len[p]);
  }
  P.priv_row.resize(nb);
  P.q_row.resize(nb);
  acc = 0;
  int64_t tacc = 0;
  for (int i = 0; i < nb; ++i) {
    const int64_t rows = (int64_t)P.past_len[i] + P.num_new[i];
    P.priv_row[i] = b.priv_row ? b.priv_row[i] : acc;
    if (P.priv_row[i] < 0) return fail(err, HPD_ERR_INVALID_ARGUMENT, "priv_row < 0");
    acc += rows;
    P.priv_rows = std::max<int64_t>(P.priv_rows, P.priv_row[i] + rows);
    P.q_row[i] = (int32_t)tacc;
    tacc += P.num_new[i];
    if (tacc > INT32_MAX / HPD_MAX_Q_HEADS)
      return fail(err, HPD_ERR_INVALID_ARGUMENT, "too many query tokens");
  }
  if (P.shared_rows > INT32_MAX || P.priv_rows > INT32_MAX)
    return fail(err, HPD_ERR_INVALID_ARGUMENT, "K/V row index exceeds 2^31 - 1");
  // pool row of row i of a paged sequence whose blocks start at entry first
  auto pool_row = [&](int32_t first, int64_t i) -> int32_t {
    return (int32_t)((int64_t)pg->blocks[first + i / pg->block_rows] * pg->block_rows + i % pg->block_rows);
  };
  if (pg) {
    P.paged = true;
    P.shared_rows = P.priv_rows = (int64_t)pg->num_blocks * pg->block_rows;
    P.page_tile0.resize(np);
    for (int p = 0; p < np; ++p) {
      P.page_tile0[p] = (int32_t)P.shared_tiles.size();
      for (int64_t i = 0; i < P.prefix_len[p]; i += 64) P.shared_tiles.push_back(pool_row(pg->page_block0[p], i));
    }
    P.branch_tile0.resize(nb);
    for (int i = 0; i < nb; ++i) {
      P.branch_tile0[i] = (int32_t)P.priv_tiles.size();
      for (int64_t r = 0; r < (int64_t)P.past_len[i] + P.num_new[i]; r += 64)
        P.priv_tiles.push_back(pool_row(pg->branch_block0[i], r));
    }
  }
  P.T = (int)tacc;
  P.page_T.assign(np, 0);
  for (int i = 0; i < nb; ++i) P.page_T[P.branch_page[i]] += P.num_new[i];
  P.page_q_row.resize(np);
  int32_t qacc = 0;
  for (int p = 0; p < np; ++p) {
    P.page_q_row[p] = qacc;
    qacc += P.page_T[p];
  }
  P.visible.resize(P.T);
  P.token_fork.resize(P.T);
  P.token_dest.resize(P.T);
  for (int i = 0; i < nb; ++i)
    for (int j = 0; j < P.num_new[i]; ++j) {
      P.visible[P.q_row[i] + j] = P.fork[i] + P.past_len[i] + j + 1;
      P.token_fork[P.q_row[i] + j] = P.fork[i];
      P.token_dest[P.q_row[i] + j] = pg ? pool_row(pg->branch_block0[i], (int64_t)P.past_len[i] + j)
                                        : (int32_t)(P.priv_row[i] + P.past_len[i] + j);
    }

  // ---- stacked positions.  Position i of page p (its rows i * G .. i * G +
  // G - 1 per kv head) holds token pos_token[page_q_row + i].  With fork
  // offsets the page's tokens are stacked in descending order of their fork
  // point (ties keep token order), so that a work item, and each wave of it,
  // holds rows whose visible prefixes are close: items end at the largest
  // fork point of their rows and waves skip the key tiles none of their rows
  // sees.
  P.pos_token.resize(2 * (size_t)P.T);
  std::vector<char> page_sorted(np, 0);
  for (int p = 0; p < np; ++p) {
    const int q0 = P.page_q_row[p], n = P.page_T[p];
    std::vector<int32_t> order(n);
    for (int i = 0; i < n; ++i) order[i] = q0 + i;
    if (P.has_fork)
      std::stable_sort(order.begin(), order.end(),
                       [&](int32_t x, int32_t y) { return P.token_fork[x] > P.token_fork[y]; });
    for (int i = 0; i < n; ++i) {
      P.pos_token[2 * (size_t)(q0 + i)] = order[i];
      P.pos_token[2 * (size_t)(q0 + i) + 1] = P.token_fork[order[i]];
      if (order[i] != q0 + i) page_sorted[p] = 1;
    }
  }
  // Largest visible prefix among the rows of each (page, row group).
  const int group_rows = kSharedWaves * kTileRows;
  std::vector<std::vector<int32_t>> group_fork(np);
  for (int p = 0; p < np; ++p) {
    const int R = P.page_T[p] * G;
    group_fork[p].reserve(ceil_div(R, group_rows));
    for (int r0 = 0; r0 < R; r0 += group_rows) {
      // the stacked positions of rows r0 .. r1 - 1
      int f = 0;
      const int i1 = (std::min(R, r0 + group_rows) - 1) / G;
      for (int i = r0 / G; i <= i1; ++i) f = std::max(f, P.pos_token[2 * (size_t)(P.page_q_row[p] + i) + 1]);
      group_fork[p].push_back(f);
    }
  }

  // ---- partial slots per token
  // Prefix keys per shared work item: a multiple of kSharedSplitUnit, sized so
  // that the shared-prefix work is about one workgroup per CU
  // (kSharedTargetItems); longer items amortise each workgroup's fixed
  // start-up and write-out, and fewer splits mean fewer partials to merge.
  // Each page's prefix is cut into equal ranges of at most `split` keys
  // (rounded up to kSharedSplitUnit), so one page's items are balanced.
  auto split_shape = [&](int p, int64_t split, int32_t &ns, int32_t &sk) {
    ns = (int32_t)ceil_div(P.prefix_len[p], split);
    sk = ns > 0 ? (int32_t)(kSharedSplitUnit * ceil_div(ceil_div(P.prefix_len[p], ns), kSharedSplitUnit)) : 0;
    if (sk > 0) ns = (int32_t)ceil_div(P.prefix_len[p], sk);
  };
  // Items for a split length.  With fork offsets, a row group's items stop
  // at its largest fork point.
  auto shared_items_for = [&](int64_t split) {
    int64_t n = 0;
    for (int p = 0; p < np; ++p) {
      if (!P.has_fork) {
        n += (int64_t)Hkv * (int64_t)group_fork[p].size() * ceil_div(P.prefix_len[p], split);
        continue;
      }
      int32_t ns, sk;
      split_shape(p, split, ns, sk);
      if (sk == 0) continue;
      for (int32_t f : group_fork[p]) n += (int64_t)Hkv * std::min<int64_t>(ns, ceil_div(f, sk));
    }
    return n;
  };
  // Grow the split until the items fit the target or one split covers every
  // page's whole prefix: with many pages, kv heads and row groups even one
  // split per page can exceed the target, and longer splits then change
  // nothing.
  int64_t max_prefix = 0;
  for (int p = 0; p < np; ++p) max_prefix = std::max<int64_t>(max_prefix, P.prefix_len[p]);
  const int64_t mult_cap = std::max<int64_t>(1, ceil_div(max_prefix, kSharedSplitUnit));
  int64_t units = shared_items_for(kSharedSplitUnit);
  int64_t mult = std::min(mult_cap, std::max<int64_t>(1, ceil_div(units, kSharedTargetItems)));
  while (mult < mult_cap && shared_items_for(kSharedSplitUnit * mult) > kSharedTargetItems) ++mult;   // ceilings per page
  // (paged K/V: at most 64 tiles per item, each item's tile rows fit a wave)
  P.split_keys = (int32_t)std::min<int64_t>(kSharedSplitUnit * mult, b.paged ? 4096 : INT32_MAX / 2);
  std::vector<int32_t> page_splits(np), page_split_keys(np);
  for (int p = 0; p < np; ++p) split_shape(p, P.split_keys, page_splits[p], page_split_keys[p]);
  // Shared splits a branch sees: those starting below its visible prefix
  // (all of its page's splits without fork offsets).  Its tokens' partial
  // slots are those splits, then its private chunks.
  std::vector<int32_t> vis_splits(nb);
  for (int i = 0; i < nb; ++i) {
    const int p = P.branch_page[i];
    vis_splits[i] = page_split_keys[p] > 0 ? (int32_t)ceil_div((int64_t)P.fork[i], page_split_keys[p]) : 0;
  }
  P.token_slots.resize(2 * (size_t)P.T);
  int64_t slot = 0;
  for (int i = 0; i < nb; ++i) {
    const int chunks = (int)ceil_div((int64_t)P.past_len[i] + P.num_new[i], kPrivateChunkKeys);
    const int cnt = vis_splits[i] + chunks;
    for (int j = 0; j < P.num_new[i]; ++j) {
      P.token_slots[2 * (size_t)(P.q_row[i] + j)] = (int32_t)slot;
      P.token_slots[2 * (size_t)(P.q_row[i] + j) + 1] = cnt;
      slot += cnt;
    }
  }
  P.num_slots = slot;
  if (P.num_slots * Hq > INT32_MAX)
    return fail(err, HPD_ERR_INVALID_ARGUMENT, "too many partial rows");

  // ---- shared-prefix work items: (page, kv head, key split, row group);
  // items that read the same key range are adjacent.  With fork offsets an
  // item's key range ends at the largest visible prefix among its rows, an
  // item no row of which sees its first key is not emitted, and a row writes
  // its partial of the split only if it sees the split's first key (the
  // kernels apply the same rule).
  {
    size_t n = 0;   // an upper bound: items trimmed by fork offsets are not emitted
    for (int p = 0; p < np; ++p) n += (size_t)Hkv * page_splits[p] * group_fork[p].size();
    P.shared_items.reserve(n * SI_NFIELDS);
  }
  for (int p = 0; p < np; ++p) {
    const int Pp = P.prefix_len[p];
    const int R = P.page_T[p] * G;
    if (Pp == 0 || R == 0) continue;
    for (int g = 0; g < Hkv; ++g)
      for (int s = 0; s < page_splits[p]; ++s)
        for (int r0 = 0; r0 < R; r0 += group_rows) {
          const int nr = std::min(group_rows, R - r0);
          const int k0 = s * page_split_keys[p];
          int k1 = std::min(Pp, k0 + page_split_keys[p]);
          int flags = 0;
          if (P.has_fork) {
            const int max_fork = group_fork[p][r0 / group_rows];
            if (max_fork <= k0) continue;
            k1 = std::min(k1, max_fork);
            for (int r = r0; r < r0 + nr; ++r)
              if (P.pos_token[2 * (size_t)(P.page_q_row[p] + r / G) + 1] < k1) flags |= SI_FLAG_FORK;
            if (page_sorted[p]) flags |= SI_FLAG_SORTED;
          }
          int32_t it[SI_NFIELDS] = {};
          it[SI_PAGE] = p; it[SI_KVH] = g; it[SI_ROW0] = r0; it[SI_NROWS] = nr;
          it[SI_KEY0] = k0; it[SI_KEY1] = k1; it[SI_SLOT] = s; it[SI_FLAGS] = flags;
          it[SI_PREFIX_ROW] = pg ? P.page_tile0[p] : (int32_t)P.prefix_row[p];
          it[SI_PAGE_Q_ROW] = P.page_q_row[p];
          it[SI_PAGE_ROWS] = R;
          P.shared_items.insert(P.shared_items.end(), it, it + SI_NFIELDS);
        }
  }

  if (np == 1 && !P.has_fork && !pg && P.prefix_len[0] > 0 && P.page_T[0] > 0 && P.prefix_row[0] <= INT32_MAX) {
    P.regular.on = 1;
    P.regular.groups = (int32_t)ceil_div((int64_t)P.page_T[0] * G, group_rows);
    P.regular.splits = page_splits[0];
    P.regular.split_keys = page_split_keys[0];
    P.regular.rows = P.page_T[0] * G;
    P.regular.prefix_len = P.prefix_len[0];
    P.regular.prefix_row = (int32_t)P.prefix_row[0];
    P.regular.page_q_row = P.page_q_row[0];
  }

  // ---- private work items: (branch, kv head, row tile, key chunk)
  {
    size_t n = 0;
    for (int i = 0; i < nb; ++i)
      n += (size_t)Hkv * ceil_div(P.num_new[i] * G, kTileRows) *
           ceil_div((int64_t)P.past_len[i] + P.num_new[i], kPrivateChunkKeys);
    P.private_items.reserve(n * PI_NFIELDS);
  }
  for (int i = 0; i < nb; ++i) {
    const int keys = P.past_len[i] + P.num_new[i];
    const int R = P.num_new[i] * G;
    const int splits = vis_splits[i];
    for (int g = 0; g < Hkv; ++g)
      for (int r0 = 0; r0 < R; r0 += kTileRows)
        for (int c = 0; c * kPrivateChunkKeys < keys; ++c) {
          int32_t it[PI_NFIELDS] = {};
          it[PI_BRANCH] = i; it[PI_KVH] = g; it[PI_ROW0] = r0;
          it[PI_NROWS] = std::min(kTileRows, R - r0);
          it[PI_KEY0] = c * kPrivateChunkKeys;
          it[PI_KEY1] = std::min(keys, (c + 1) * kPrivateChunkKeys);
          it[PI_SLOT] = splits + c; it[PI_PAST] = P.past_len[i];
          it[PI_PRIV_ROW] = pg ? P.branch_tile0[i] : (int32_t)P.priv_row[i];
          it[PI_Q_ROW] = P.q_row[i];
          it[PI_NUM_NEW] = P.num_new[i];
          P.private_items.insert(P.private_items.end(), it, it + PI_NFIELDS);
        }
  }

  // ---- workspace layout: tables (uploaded once) then partials
  size_t off = 0;
  P.off_shared_tiles = off;
  off = align256(off + P.shared_tiles.size() * sizeof(int32_t));
  P.off_priv_tiles = off;
  off = align256(off + P.priv_tiles.size() * sizeof(int32_t));
  P.off_branch_q_row = off;
  off = align256(off + P.q_row.size() * sizeof(int32_t));
  P.off_branch_new = off;
  off = align256(off + P.num_new.size() * sizeof(int32_t));
  P.off_shared_items = off;
  off = align256(off + P.shared_items.size() * sizeof(int32_t));
  P.off_private_items = off;
  off = align256(off + P.private_items.size() * sizeof(int32_t));
  P.off_token_slots = off;
  off = align256(off + P.token_slots.size() * sizeof(int32_t));
  P.off_token_fork = off;
  off = align256(off + P.token_fork.size() * sizeof(int32_t));
  P.off_token_dest = off;
  off = align256(off + P.token_dest.size() * sizeof(int32_t));
  P.off_token_vis = off;
  off = align256(off + P.visible.size() * sizeof(int32_t));
  P.off_pos_token = off;
  off = align256(off + P.pos_token.size() * sizeof(int32_t));
  P.off_counters = off;   // zeroed by the upload; every user resets what it uses
  off = align256(off + kNumCounters * sizeof(int32_t));
  P.table_bytes = off;
  P.off_part_o = off;
  off = align256(off + (size_t)P.num_slots * Hq * HPD_HEAD_DIM * sizeof(float));
  P.off_part_lse = off;
  off = align256(off + (size_t)P.num_slots * Hq * sizeof(float));
  P.workspace_bytes = off;

  // sorted items find their page's stacked positions from the token_fork table
  for (size_t i = 0; i < P.shared_items.size(); i += SI_NFIELDS)
    if (P.shared_items[i + SI_FLAGS] & SI_FLAG_SORTED)
      P.shared_items[i + SI_POS] =
          (int32_t)((P.off_pos_token - P.off_token_fork) / sizeof(int32_t) + 2 * (size_t)P.shared_items[i + SI_PAGE_Q_ROW]);
  P.table_image.assign(P.table_bytes, 0);
  auto put = [&](size_t at, const std::vector<int32_t> &v) {
    if (!v.empty()) std::memcpy(P.table_image.data() + at, v.data(), v.size() * sizeof(int32_t));
  };
  put(P.off_shared_tiles, P.shared_tiles);
  put(P.off_priv_tiles, P.priv_tiles);
  put(P.off_branch_q_row, P.q_row);
  put(P.off_branch_new, P.num_new);
  put(P.off_shared_items, P.shared_items);
  put(P.off_private_items, P.private_items);
  put(P.off_token_slots, P.token_slots);
  put(P.off_token_fork, P.token_fork);
  put(P.off_token_dest, P.token_dest);
  put(P.off_token_vis, P.visible);
  put(P.off_pos_token, P.pos_token);

  *out = std::move(P);
  return HPD_OK;
}

}  // namespace hpd
