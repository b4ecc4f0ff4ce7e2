// Host-side planning for the four entry points: argument validation, workspace layout
// and the per-call work lists.  Plain C++ (no HIP); the entry points in tide_api.hip
// upload the blob it builds with one host-to-device copy.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "tide.h"
#include "tide_common.h"

namespace tide {

// Where each region lives inside the caller's workspace (byte offsets).
struct Plan {
  int op = 0;
  int32_t num_tasks = 0;
  // upload region [0, upload_bytes): header, task table, items
  size_t tasks_off = 0;
  size_t items_off = 0;
  size_t upload_bytes = 0;
  // extend split-KV plan: per-row merge descriptors (uploaded after the items)
  bool split = false;
  size_t merge_rows_off = 0;
  // decode: per-(task, kv head) arrival counters, zeros in the uploaded blob, used when
  // the split kernel merges (fold_merge: few splits per task) instead of a merge kernel
  size_t tickets_off = 0;
  bool fold_merge = false;
  int64_t row_slots = 0;  // partial row slots (each holds every query head)
  // the planner's run-time estimates (microseconds) of the plain and chosen extend plans;
  // 0 when the call was too large to consider splitting
  double est_plain_us = 0.0;
  double est_us = 0.0;
  // decode and split-extend partials (not uploaded)
  size_t part_o_off = 0;
  size_t part_ml_off = 0;
  size_t total_bytes = 0;
  int32_t num_items = 0;
  // extend: tokens per work item and waves per workgroup
  int32_t tokens_per_item = 0;
  int32_t waves = 0;
  // decode
  int32_t chunk = 0;
  int32_t max_splits = 0;
  int32_t total_rows = 0;
  std::vector<uint8_t> blob;  // bytes to upload (header + tasks + items)
};

// Shape validation shared by every entry point.
int check_dims(const tide_dims* dims);

// Validates lengths and builds the plan.  When `build_blob` is false only the sizes are
// computed (tide_workspace_size).  `bt_stride` < 0 skips the block-table capacity check.
int make_plan(int op, int32_t num_tasks, const int32_t* lens_a, const int32_t* lens_b,
              const tide_dims& dims, int32_t num_splits, int32_t bt_stride, bool build_blob,
              Plan* plan);

// Shared-prefix decode: groups are consecutive task ranges [group_start[g],
// group_start[g+1]); the first shared_lens[g] keys (a multiple of the page size, below
// every member's kv_len) live in pages every member's block table shares.
constexpr int kOpDecodeShared = 100;  // internal op code of the plan
int make_plan_shared(int32_t num_tasks, const int32_t* kv_lens, int32_t num_groups,
                     const int32_t* group_start, const int32_t* shared_lens,
                     const tide_dims& dims, int32_t num_splits, int32_t bt_stride,
                     bool build_blob, Plan* plan);

// Waves per workgroup of the extend kernel for a head size and GQA group.
int32_t extend_waves(int32_t head_dim, int32_t group);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace tide
