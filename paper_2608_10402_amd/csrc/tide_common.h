// Definitions shared by the host planner and the gfx950 kernels: the work-item records
// uploaded into the caller's workspace, and the kernel argument blocks.
#pragma once

#include <stdint.h>

namespace tide {

constexpr int kPage = 16;         // tokens per page
constexpr int kMaxGroup = 16;     // largest supported Hq / Hkv
// Largest supported Hkv: a pool page (Hkv blocks of kPage rows of head_dim bf16) then
// spans at most 2^28 bytes, which the extend kernel's 32-bit page stride holds.
constexpr int kMaxKvHeads = 65536;
constexpr int kExtendKeyTile = 64;  // keys per extend-kernel iteration (4 pages)
constexpr int kDecodeStep = 32;   // keys per decode-kernel iteration (2 pages)
constexpr int kWsAlign = 256;
constexpr int kXcds = 8;          // MI355X: 8 accelerator dies, one L2 each

// One task as the kernels see it.  `row_start` indexes the packed token rows of Q/O
// (extend, prefill) or the task itself (decode); tokens at positions
// [prefix, prefix + extend) are the ones this call processes.
struct TaskDesc {
  int32_t row_start;
  int32_t prefix;
  int32_t extend;
  int32_t aux;  // decode: number of splits of this task; append: first new-row index
};

// Extend / prefill work item: tokens [tok0, tok0 + ntok) of `task` (relative to its
// prefix) for every query head that reads kv head `kv_head`.
struct ExtendItem {
  int32_t task;
  int32_t kv_head;
  int32_t tok0;
  int32_t ntok;
};

// Extend / prefill work item of the split-KV plan, used when a call has too few items
// to fill the chip: key tiles [t_begin, t_end) of the item (64 keys each, counted from
// key 0).  split >= 0: one of the item's chunks; its unnormalised partial for row slot
// s = pbase + split * ntok + tk (tk = token inside the item) and query head h goes to
// part_o[(s * Hq + h) * d] and part_ml[(s * Hq + h) * 4], and a merge combines the
// chunks.  split == -1: the item is not split and writes its output directly.
struct ExtendChunkItem {
  int32_t task;
  int32_t kv_head;
  int32_t tok0;
  int32_t ntok;
  int32_t t_begin;
  int32_t t_end;
  int32_t split;
  int32_t pbase;
};

// Merge descriptor of one packed extend row: its partials sit in row slots base,
// base + stride, ..., base + (nsplit - 1) * stride; nsplit == 0 means the row was
// written directly and has nothing to merge.
struct MergeRow {
  int32_t base;
  int32_t stride;
  int32_t nsplit;
  int32_t pad;
};

// Decode split-K item: keys [k_begin, min(kv_len, k_begin + chunk)) of one (task, kv head).
struct DecodeItem {
  int32_t task;
  int32_t kv_head;
  int32_t split;
  int32_t k_begin;
};

// Shared-prefix decode item: keys [k_begin, k_end) for tasks first_task ..
// first_task + ntasks - 1 and one kv head.  With ntasks > 1 the keys lie in the prefix
// the tasks share (the same physical pages, read through first_task's block table), and
// the item writes one split partial per task; ntasks * group <= 16.
struct SharedDecodeItem {
  int32_t first_task;
  int32_t ntasks;
  int32_t kv_head;
  int32_t split;
  int32_t k_begin;
  int32_t k_end;
  int32_t pad[2];
};

// Append item: positions [pos_begin, pos_end) of `task`, all inside logical page `lpage`.
struct AppendItem {
  int32_t task;
  int32_t lpage;
  int32_t pos_begin;
  int32_t pos_end;
};

// Layout of the per-call header at the start of the workspace.
struct WsHeader {
  int32_t error_flags;  // bit 0: a block-table page id was outside [0, num_pages)
  int32_t pad[63];
};

struct AppendArgs {
  const uint16_t* k_new;
  const uint16_t* v_new;
  uint16_t* k_pool;
  uint16_t* v_pool;
  const int32_t* block_table;
  int64_t num_pages;
  int32_t bt_stride;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t num_items;
  const TaskDesc* tasks;
  const AppendItem* items;
  int32_t* error_flags;
};

struct ExtendArgs {
  const uint16_t* q;
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* block_table;
  int64_t num_pages;
  int32_t bt_stride;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;
  float scale_log2;  // sm_scale * log2(e): scores are kept in base-2 units
  int32_t num_items;
  const TaskDesc* tasks;
  const ExtendItem* items;
  uint16_t* out;
  float* lse;
  int32_t* error_flags;
  // split-KV plan (chunk_items non-null): items, per-row merge descriptors and the
  // partial buffers [row slots][Hq][d] and [row slots][Hq][4] (max in base-2 units, sum of
  // the bf16-rounded weights, exact fp32 sum, unused)
  const ExtendChunkItem* chunk_items;
  const MergeRow* merge_rows;
  float* part_o;
  float* part_ml;
  int32_t total_rows;
  // fused append (non-null k_new): the new tokens' K/V rows, packed like q by extend_lens,
  // [rows][Hkv][d].  Keys at or past a task's prefix are read from them instead of the
  // pool, and each item writes its own tokens' rows into the pool.
  const uint16_t* k_new;
  const uint16_t* v_new;
};

struct DecodeArgs {
  const uint16_t* q;
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* block_table;
  int64_t num_pages;
  int32_t bt_stride;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;
  float scale_log2;
  int32_t num_tasks;
  int32_t num_items;
  int32_t chunk;       // keys per split (multiple of kDecodeStep)
  int32_t max_splits;  // split slots per (task, q head) in the partial buffers
  const TaskDesc* tasks;  // prefix + extend == kv_len, aux == number of splits
  const void* items;      // DecodeItem, or SharedDecodeItem for the shared-prefix variant
  float* part_o;   // [num_tasks][Hq][max_splits][d] unnormalised partial outputs
  float* part_ml;  // [num_tasks][Hq][max_splits][4]: max (base-2 units), sum of the
                   // bf16-rounded weights, exact fp32 sum, unused
  uint16_t* out;
  float* lse;
  int32_t* error_flags;
  // fused append: the K/V rows of each task's newest token (position kv_len - 1),
  // [num_tasks][Hkv][d]; the split that holds that position writes them into the pool
  // and uses them directly.  Null for a plain decode.
  const uint16_t* k_new;
  const uint16_t* v_new;
  // plain decode: one arrival counter per (task, kv head), zero at launch (uploaded with
  // the work list); the split that brings it to the task's split count merges that kv
  // head's rows.  Null for the shared-prefix variant, which merges in a second kernel.
  int32_t* tickets;
};

}  // namespace tide
