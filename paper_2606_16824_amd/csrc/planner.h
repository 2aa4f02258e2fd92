// Host planner: turns host-side lengths into the extend work list.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "cw_internal.h"
#include "plan_expand.h"

namespace cw {

struct Tuning {
  int32_t kv_chunk_tiles = 0;  // 0 = automatic
  int32_t target_wgs = 0;      // 0 = automatic
  int32_t extend_kernel = 0;   // 0 = automatic, 1 = eight waves of 32 rows, 2 = four waves of 64 rows
  int32_t deal_rounds = 1;     // 1 = deal bundles of whole GPU rounds across XCDs, 0 = keep them on one
  int32_t plan_direct = 0;     // 1 = kernels read the plan from the pinned staging slot, 0 = copy it first
  int32_t suffix_weight = 125; // split-K cost of a key tile past the prefix, in percent of a prefix tile
  int32_t compact_decode = 1;  // 1 = decode plans are uploaded in compact form
  int32_t arg_plans = 1;       // 1 = extend plans of up to 16 KB travel in the kernel arguments
};

struct ExtendPlan {
  std::vector<SeqInfo> seqs;
  std::vector<WorkItem> items;  // launch order
  std::vector<CombineGroup> groups;
  int64_t n_parts = 0;
  // Workspace layout (byte offsets, 256-byte aligned).
  size_t off_seqs = 0, off_items = 0, off_groups = 0, off_part_o = 0, off_part_ml = 0;
  size_t meta_bytes = 0;  // seqs + items + groups: the part uploaded per call
  size_t total_bytes = 0;
  int32_t part_rows = 0;  // rows per partial slot
  // decode plans: the same items and groups in compact form (see plan_expand.h)
  bool compact = false;
  std::vector<DecodeRec> recs;
  std::vector<int32_t> tails;
  ExpandDesc desc{};  // offsets relative to the plan's own meta
};

// Builds the plan for a kernel whose workgroups own `block_m` rows and of
// which `wgs_per_cu` are resident per CU.  `num_cus` and `num_xcds` describe
// the device.  Lengths must already be validated.  Sequence b's first packed
// row is cu_rows[b] and its block-table row bt_rows[b] when given (a sub-batch
// of a larger step), else the prefix sum of the suffix lengths and b.
ExtendPlan build_extend_plan(const int32_t* prefix_lens, const int32_t* suffix_lens,
                             int32_t num_seqs, int32_t num_kv_heads, int32_t gqa_group,
                             int32_t head_dim, int32_t block_m, int32_t wgs_per_cu,
                             int32_t num_cus, int32_t num_xcds, const Tuning& tuning,
                             const int32_t* cu_rows = nullptr, const int32_t* bt_rows = nullptr);

// Decode plan (every suffix length 1): one item per (sequence, kv head, key
// chunk) with `gqa_group` rows; `keys_per_tile` is the decode kernel's tile.
ExtendPlan build_decode_plan(const int32_t* prefix_lens, int32_t num_seqs, int32_t num_kv_heads,
                             int32_t gqa_group, int32_t head_dim, int32_t page_size,
                             int32_t keys_per_tile, int32_t waves_per_cu, int32_t num_cus,
                             const Tuning& tuning, const int32_t* cu_rows = nullptr,
                             const int32_t* bt_rows = nullptr);

// Serialises seqs, items and groups into `dst` (meta_bytes long) at their offsets.
void pack_plan_meta(const ExtendPlan& plan, uint8_t* dst);
// Only the meta's first off_items bytes (the sequences).
void pack_plan_head(const ExtendPlan& plan, uint8_t* dst);

}  // namespace cw
