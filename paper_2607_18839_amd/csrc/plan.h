// Internal plan structure shared by the planner (host C++) and the launchers.
// Not part of the public ABI: callers see only the opaque hpd_plan.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "hpd.h"

namespace hpd {

// Work item of the shared-prefix kernel: one workgroup of kSharedWaves waves,
// each wave one 32-row tile of the stacked query rows of (page, kv head), all
// of them over the same prefix key range [key_begin, key_end).
// Stacked row r of (page p, kv head g) is query head g * G + r % G of token
// page_q_row[p] + r / G.
// SI_PREFIX_ROW / PI_PRIV_ROW: the first K/V row of the page's prefix /
// branch's private rows, or with paged K/V its first entry in the shared /
// private tile table.
enum SharedItemField {
  SI_PAGE = 0, SI_KVH, SI_ROW0, SI_NROWS, SI_KEY0, SI_KEY1, SI_SLOT, SI_FLAGS,
  SI_PREFIX_ROW, SI_PAGE_Q_ROW, SI_PAGE_ROWS, SI_POS, SI_NFIELDS
};
// SI_POS (items with SI_FLAG_SORTED): the page's first pos_token entry, in
// int32 elements from the start of the token_fork table.
// Work item of the private kernel: one wave, one 32-row tile of the stacked
// rows of (branch, kv head), private keys [key_begin, key_end) of the branch.
// Stacked row r of (branch b, kv head g) is query head g * G + r % G of the
// branch's new token j = r / G, which sees private keys 0 .. L_b + j.
enum PrivateItemField {
  PI_BRANCH = 0, PI_KVH, PI_ROW0, PI_NROWS, PI_KEY0, PI_KEY1, PI_SLOT, PI_PAST,
  PI_PRIV_ROW, PI_Q_ROW, PI_NUM_NEW, PI_RESERVED, PI_NFIELDS
};

constexpr int kSharedWaves = 4;      // waves per shared-prefix workgroup
constexpr int kTileRows = 32;        // stacked query rows per wave (MFMA 32x32)
constexpr int kKeyTile = 64;         // keys per LDS tile
constexpr int kSharedSplitUnit = 128;   // shared work items cover multiples of this many prefix keys
constexpr int kSharedTargetItems = 256; // aim: about one shared-prefix workgroup per CU
constexpr int kPrivateChunkKeys = 128;  // private keys per private work item
constexpr int SI_FLAG_FORK = 1;      // rows have their own fork limits
constexpr int SI_FLAG_SORTED = 2;    // stacked positions map to tokens through pos_token
constexpr int kNumCounters = 8192;   // self-resetting arrival counters (split-K / merges)

struct Plan {
  hpd_attn_desc attn{};
  int G = 0;                // query heads per kv head
  float scale = 0.f;        // softmax scale actually used
  int T = 0, num_pages = 0, num_branches = 0;
  bool has_fork = false;

  std::vector<int32_t> prefix_len, branch_page, num_new, past_len, fork;
  std::vector<int64_t> prefix_row, priv_row;
  std::vector<int32_t> q_row, page_q_row, page_T, visible;
  int64_t shared_rows = 0, priv_rows = 0;

  // Paged K/V: physical row of the first key of every 64-key tile, per page
  // prefix (page_tile0[p] + i) and per branch (branch_tile0[b] + i).  Shared
  // and private work items then carry a tile-table offset where contiguous
  // plans carry a first row.
  bool paged = false;
  std::vector<int32_t> shared_tiles, priv_tiles, page_tile0, branch_tile0;

  std::vector<int32_t> shared_items, private_items;   // [n][SI_NFIELDS / PI_NFIELDS]
  std::vector<int32_t> token_slots;                   // [T][2]: first slot, count
  std::vector<int32_t> token_fork;                    // [T] visible prefix per token
  std::vector<int32_t> token_dest;                    // [T] private row of token t: priv_row + L + j
  // [T][2] (token, visible prefix) of each stacked position.  With fork
  // offsets a page's tokens are stacked in descending order of their fork
  // point, so that each work item (and each wave of it) holds rows whose
  // visible prefixes are close; without them position = token.
  std::vector<int32_t> pos_token;
  // (visible[t] - 1 is token t's position in its branch's sequence)
  int64_t num_slots = 0;                              // partial rows = num_slots * Hq
  int32_t split_keys = 0;                             // prefix keys per shared work item
  // One page without fork offsets: its shared items are (kv head, split, row
  // group) in that nesting order and the kernels compute an item's fields
  // from its index instead of reading the table.
  struct RegularShared {
    int32_t on = 0, groups = 0, splits = 0, split_keys = 0, rows = 0, prefix_len = 0, prefix_row = 0,
            page_q_row = 0;
  } regular;

  // device workspace layout (byte offsets, 256-aligned)
  size_t off_shared_tiles = 0, off_priv_tiles = 0, off_branch_q_row = 0, off_branch_new = 0;
  size_t off_shared_items = 0, off_private_items = 0, off_token_slots = 0,
         off_token_fork = 0, off_token_dest = 0, off_pos_token = 0, off_token_vis = 0, off_counters = 0, off_part_o = 0, off_part_lse = 0, table_bytes = 0,
         workspace_bytes = 0;
  std::vector<unsigned char> table_image;             // host copy of [0, table_bytes)

  int num_shared_items() const { return (int)(shared_items.size() / SI_NFIELDS); }
  int num_private_items() const { return (int)(private_items.size() / PI_NFIELDS); }
};

// Builds the plan; on failure returns a status and sets *err.
hpd_status build_plan(const hpd_attn_desc *attn, const hpd_batch_desc *batch, Plan *out,
                      std::string *err);

}  // namespace hpd

struct hpd_plan {
  hpd::Plan p;
};
