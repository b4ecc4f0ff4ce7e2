// Host-side checker of the work lists built by the planner (plan.cpp), compiled with g++
// by test_plan.py; no GPU involved.
//
// Each stdin line is one call: "op hq hkv d ntasks p_0 e_0 p_1 e_1 ..." (op 2 = extend,
// 4 = full prefill, which reads e_i as the sequence length and ignores p_i), or
// "3 hq hkv d ntasks num_splits kv_0 .. kv_{n-1}" (decode), or
// "100 hq hkv d ntasks num_splits ngroups gs_0 .. gs_ngroups sh_0 .. kv_0 .." (decode with
// shared group prefixes; gs = group starts, sh = shared prefix lengths).  Decode calls are
// checked by check_decode / check_shared below.  For every extend / prefill call the
// checker builds the plan, reads the uploaded blob back and verifies what the kernels
// assume:
//   * every (task, kv head, token) row block is covered by exactly one item, and every
//     item's tokens lie inside its task;
//   * split plan: the chunks of each (block, kv head) partition the key tiles the block
//     sees, their partial row slots lie inside the partial buffers and no (slot, head) is
//     written twice, and each packed row's merge descriptor names exactly its chunks;
//   * the workspace regions lie in order inside total_bytes without overlap.
// It prints "ok <split> <items> <row_slots> <total_bytes> <est_plain_us> <est_us>" per call, or "FAIL <reason>"
// and exits non-zero.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <iostream>
#include <map>
#include <set>
#include <sstream>
#include <string>
#include <tuple>
#include <vector>

#include "plan.h"

using namespace tide;

static int fail(const char* what, long a = 0, long b = 0) {
  printf("FAIL %s %ld %ld\n", what, a, b);
  return 1;
}

static int check(int op, const tide_dims& dims, const std::vector<int32_t>& pa,
                 const std::vector<int32_t>& pb) {
  const int32_t n = (int32_t)pa.size();
  Plan plan;
  int rc = make_plan(op, n, pa.data(), op == TIDE_OP_EXTEND ? pb.data() : nullptr, dims, 0, -1,
                     true, &plan);
  if (rc != TIDE_OK) return fail("make_plan", rc);
  Plan sized;
  rc = make_plan(op, n, pa.data(), op == TIDE_OP_EXTEND ? pb.data() : nullptr, dims, 0, -1,
                 false, &sized);
  if (rc != TIDE_OK || sized.total_bytes != plan.total_bytes || sized.split != plan.split)
    return fail("size-only plan differs");
  const int32_t G = dims.num_q_heads / dims.num_kv_heads;
  const int32_t Hkv = dims.num_kv_heads;
  const int32_t tb = plan.tokens_per_item;
  if (tb * G > 256 || tb <= 0) return fail("tokens per item", tb);
  const TaskDesc* tasks = reinterpret_cast<const TaskDesc*>(plan.blob.data() + plan.tasks_off);
  if (plan.blob.size() != plan.upload_bytes) return fail("blob size");
  if (plan.upload_bytes > plan.total_bytes) return fail("upload beyond total");
  // region order
  if (plan.items_off < plan.tasks_off + n * sizeof(TaskDesc)) return fail("items overlap tasks");
  const size_t isz = plan.split ? sizeof(ExtendChunkItem) : sizeof(ExtendItem);
  const size_t items_end = plan.items_off + (size_t)plan.num_items * isz;
  if (items_end > plan.upload_bytes) return fail("items beyond upload");
  if (plan.split) {
    if (plan.merge_rows_off < items_end) return fail("merge rows overlap items");
    if (plan.merge_rows_off + (size_t)plan.total_rows * sizeof(MergeRow) > plan.upload_bytes)
      return fail("merge rows beyond upload");
    const size_t slots = (size_t)plan.row_slots * dims.num_q_heads;
    if (plan.part_o_off < plan.upload_bytes) return fail("partials overlap upload");
    if (plan.part_ml_off < plan.part_o_off + slots * dims.head_dim * 4) return fail("part_o size");
    if (plan.total_bytes < plan.part_ml_off + slots * 16) return fail("part_ml size");
    if (plan.part_o_off % 16 || plan.part_ml_off % 16) return fail("partial alignment");
  }

  // rows of each task, per kv head: which item covered them
  std::map<std::tuple<int, int, int>, int> covered;  // (task, kv head, token) -> count
  // split: per (task, kv head, tok0) the chunk tile ranges and split ids
  std::map<std::tuple<int, int, int>, std::vector<std::tuple<int, int, int, int, int>>> chunks;
  std::set<std::pair<int64_t, int>> slot_heads;  // (row slot, kv head)
  for (int32_t i = 0; i < plan.num_items; ++i) {
    int task, kvh, tok0, ntok, tbeg = 0, tend = 0, split = -1, pbase = 0;
    if (plan.split) {
      const ExtendChunkItem it =
          reinterpret_cast<const ExtendChunkItem*>(plan.blob.data() + plan.items_off)[i];
      task = it.task, kvh = it.kv_head, tok0 = it.tok0, ntok = it.ntok;
      tbeg = it.t_begin, tend = it.t_end, split = it.split, pbase = it.pbase;
    } else {
      const ExtendItem it = reinterpret_cast<const ExtendItem*>(plan.blob.data() + plan.items_off)[i];
      task = it.task, kvh = it.kv_head, tok0 = it.tok0, ntok = it.ntok;
    }
    if (ntok == 0) continue;  // padding slot
    if (task < 0 || task >= n || kvh < 0 || kvh >= Hkv) return fail("item ids", task, kvh);
    const TaskDesc td = tasks[task];
    if (tok0 < 0 || ntok < 0 || ntok > tb || tok0 + ntok > td.extend) return fail("item tokens", tok0, ntok);
    if (!plan.split || split <= 0)
      for (int t = 0; t < ntok; ++t) covered[{task, kvh, tok0 + t}]++;
    if (plan.split) {
      const int ntiles = (td.prefix + tok0 + ntok + 63) / 64;
      if (tbeg < 0 || tend <= tbeg || tend > ntiles) return fail("chunk tiles", tbeg, tend);
      chunks[{task, kvh, tok0}].push_back({tbeg, tend, split, pbase, ntok});
      if (split >= 0)
        for (int t = 0; t < ntok; ++t) {
          const int64_t slot = (int64_t)pbase + (int64_t)split * ntok + t;
          if (slot < 0 || slot >= plan.row_slots) return fail("slot range", slot, plan.row_slots);
          if (!slot_heads.insert({slot, kvh}).second) return fail("slot written twice", slot, kvh);
        }
    }
  }
  int64_t rows = 0;
  for (int32_t b = 0; b < n; ++b) {
    if (tasks[b].row_start != rows) return fail("row_start", b);
    for (int32_t g = 0; g < Hkv; ++g)
      for (int t = 0; t < tasks[b].extend; ++t)
        if (covered[{b, g, t}] != 1) return fail("row coverage", b, t);
    rows += tasks[b].extend;
  }
  if (rows != plan.total_rows) return fail("total rows");
  if (plan.split) {
    const MergeRow* mr = reinterpret_cast<const MergeRow*>(plan.blob.data() + plan.merge_rows_off);
    std::vector<int> seen((size_t)plan.total_rows, 0);
    for (const auto& kv : chunks) {
      const int task = std::get<0>(kv.first), tok0 = std::get<2>(kv.first);
      std::vector<std::tuple<int, int, int, int, int>> c = kv.second;
      std::sort(c.begin(), c.end());
      const int ntok = std::get<4>(c[0]);
      const int ntiles = (tasks[task].prefix + tok0 + ntok + 63) / 64;
      int at = 0;
      for (size_t k = 0; k < c.size(); ++k) {
        if (std::get<0>(c[k]) != at) return fail("chunk gap", task, tok0);
        at = std::get<1>(c[k]);
        const int want = c.size() == 1 ? -1 : (int)k;
        if (std::get<2>(c[k]) != want) return fail("split id", std::get<2>(c[k]), want);
        if (std::get<3>(c[k]) != std::get<3>(c[0])) return fail("pbase differs");
      }
      if (at != ntiles) return fail("chunks end", at, ntiles);
      for (int t = 0; t < ntok; ++t) {
        const int r = tasks[task].row_start + tok0 + t;
        const MergeRow m = mr[r];
        seen[r]++;
        if (c.size() == 1) {
          if (m.nsplit != 0) return fail("unsplit row has merge", r);
        } else if (m.nsplit != (int)c.size() || m.stride != ntok || m.base != std::get<3>(c[0]) + t) {
          return fail("merge row", r, m.nsplit);
        }
      }
    }
    for (int64_t r = 0; r < plan.total_rows; ++r)
      if (seen[r] != Hkv) return fail("merge row seen", r, seen[r]);
  }
  printf("ok %d %d %lld %zu %.1f %.1f\n", plan.split ? 1 : 0, plan.num_items,
         (long long)plan.row_slots, plan.total_bytes, plan.est_plain_us, plan.est_us);
  return 0;
}

// Regions of a decode workspace: tasks, items, then (plain decode) the arrival counters,
// all inside the upload; the partial buffers after it, large enough for every
// (task, query head, split) slot.
static int check_decode_layout(const Plan& plan, const tide_dims& dims, int32_t n,
                               size_t item_size, bool counters) {
  if (plan.blob.size() != plan.upload_bytes) return fail("blob size");
  if (plan.items_off < plan.tasks_off + (size_t)n * sizeof(TaskDesc)) return fail("items overlap tasks");
  const size_t items_end = plan.items_off + (size_t)plan.num_items * item_size;
  if (items_end > plan.upload_bytes) return fail("items beyond upload");
  if (counters) {
    if (plan.tickets_off < items_end) return fail("counters overlap items");
    const size_t end = plan.tickets_off + (size_t)n * dims.num_kv_heads * sizeof(int32_t);
    if (end > plan.upload_bytes) return fail("counters beyond upload");
    for (size_t i = plan.tickets_off; i < end; ++i)
      if (plan.blob[i] != 0) return fail("counter not zero", (long)i);
  }
  const size_t slots = (size_t)n * dims.num_q_heads * (size_t)plan.max_splits;
  if (plan.part_o_off < plan.upload_bytes) return fail("partials overlap upload");
  if (plan.part_ml_off < plan.part_o_off + slots * dims.head_dim * 4) return fail("part_o size");
  if (plan.total_bytes < plan.part_ml_off + slots * 16) return fail("part_ml size");
  if (plan.part_o_off % 16 || plan.part_ml_off % 16) return fail("partial alignment");
  return 0;
}

// Plain decode: every (task, kv head) is cut into chunks of plan.chunk keys, split s
// covering keys [s * chunk, min(kv, (s + 1) * chunk)); each (task, kv head, split) is one
// item; the task table holds kv - 1 + 1 and the split count; full chunks come first, then
// the shorter last chunks, longest first; the in-kernel merge is chosen at <= 4 splits
// per task on average.
static int check_decode(const tide_dims& dims, int32_t num_splits, const std::vector<int32_t>& kv) {
  const int32_t n = (int32_t)kv.size();
  Plan plan, sized;
  int rc = make_plan(TIDE_OP_DECODE, n, kv.data(), nullptr, dims, num_splits, -1, true, &plan);
  if (rc != TIDE_OK) return fail("make_plan", rc);
  rc = make_plan(TIDE_OP_DECODE, n, kv.data(), nullptr, dims, num_splits, -1, false, &sized);
  if (rc != TIDE_OK || sized.total_bytes != plan.total_bytes || sized.fold_merge != plan.fold_merge)
    return fail("size-only plan differs");
  if (check_decode_layout(plan, dims, n, sizeof(DecodeItem), true)) return 1;
  const int64_t chunk = plan.chunk;
  if (chunk < kDecodeStep || chunk % kDecodeStep) return fail("chunk", (long)chunk);
  const int32_t Hkv = dims.num_kv_heads;
  const TaskDesc* tasks = reinterpret_cast<const TaskDesc*>(plan.blob.data() + plan.tasks_off);
  int32_t max_splits = 0;
  for (int32_t b = 0; b < n; ++b) {
    const int32_t want = (int32_t)((kv[b] + chunk - 1) / chunk);
    if (tasks[b].row_start != b || tasks[b].prefix + tasks[b].extend != kv[b] ||
        tasks[b].extend != 1 || tasks[b].aux != want)
      return fail("task row", b, tasks[b].aux);
    max_splits = std::max(max_splits, want);
  }
  if (plan.max_splits != max_splits) return fail("max splits", plan.max_splits, max_splits);
  std::set<std::tuple<int, int, int>> seen;
  const DecodeItem* items = reinterpret_cast<const DecodeItem*>(plan.blob.data() + plan.items_off);
  int64_t prev_len = chunk;
  bool in_tail = false;
  for (int32_t i = 0; i < plan.num_items; ++i) {
    const DecodeItem it = items[i];
    if (it.task < 0 || it.task >= n || it.kv_head < 0 || it.kv_head >= Hkv) return fail("item ids", i);
    if (it.split < 0 || it.split >= tasks[it.task].aux) return fail("split id", i, it.split);
    if ((int64_t)it.k_begin != it.split * chunk) return fail("k_begin", i, it.k_begin);
    if (!seen.insert({it.task, it.kv_head, it.split}).second) return fail("item twice", i);
    const int64_t len = std::min<int64_t>(chunk, kv[it.task] - it.k_begin);
    if (len <= 0) return fail("empty item", i);
    if (len < chunk) in_tail = true;
    else if (in_tail) return fail("full chunk after a tail chunk", i);
    if (in_tail && len > prev_len) return fail("tail not longest first", i);
    prev_len = len;
  }
  int64_t want_items = 0;
  for (int32_t b = 0; b < n; ++b) want_items += (int64_t)tasks[b].aux * Hkv;
  if ((int64_t)plan.num_items != want_items || (int64_t)seen.size() != want_items)
    return fail("item count", plan.num_items, (long)want_items);
  if (plan.fold_merge != (plan.num_items <= 4 * (int64_t)n * Hkv)) return fail("fold choice");
  printf("ok %d %lld %d %d %zu\n", plan.num_items, (long long)chunk, plan.max_splits,
         plan.fold_merge ? 1 : 0, plan.total_bytes);
  return 0;
}

// Shared-prefix decode: for every task and kv head, the items that cover it (prompt
// chunks of its group, read once for up to 16 / G trajectories, then its own chunks)
// give split ids 0 .. aux-1 exactly once and key ranges that tile [0, kv) in split
// order; a prompt item stays inside the prompt and its group, an own item after the
// prompt; every item fits the 16 MFMA columns; items are ordered longest first.
static int check_shared(const tide_dims& dims, int32_t num_splits, const std::vector<int32_t>& kv,
                        const std::vector<int32_t>& gs, const std::vector<int32_t>& sh) {
  const int32_t n = (int32_t)kv.size(), ng = (int32_t)sh.size();
  Plan plan, sized;
  int rc = make_plan_shared(n, kv.data(), ng, gs.data(), sh.data(), dims, num_splits, -1, true, &plan);
  if (rc != TIDE_OK) return fail("make_plan_shared", rc);
  rc = make_plan_shared(n, kv.data(), ng, gs.data(), sh.data(), dims, num_splits, -1, false, &sized);
  if (rc != TIDE_OK || sized.total_bytes != plan.total_bytes) return fail("size-only plan differs");
  if (check_decode_layout(plan, dims, n, sizeof(SharedDecodeItem), false)) return 1;
  const int32_t Hkv = dims.num_kv_heads, G = dims.num_q_heads / dims.num_kv_heads;
  const TaskDesc* tasks = reinterpret_cast<const TaskDesc*>(plan.blob.data() + plan.tasks_off);
  std::vector<int32_t> group_of(n), shared_of(n);
  for (int32_t g = 0; g < ng; ++g)
    for (int32_t b = gs[g]; b < gs[g + 1]; ++b) group_of[b] = g, shared_of[b] = sh[g];
  // (task, kv head) -> split -> key range
  std::map<std::pair<int, int>, std::map<int, std::pair<int, int>>> cover;
  const SharedDecodeItem* items =
      reinterpret_cast<const SharedDecodeItem*>(plan.blob.data() + plan.items_off);
  int prev_len = INT32_MAX;
  for (int32_t i = 0; i < plan.num_items; ++i) {
    const SharedDecodeItem it = items[i];
    if (it.first_task < 0 || it.ntasks < 1 || it.first_task + it.ntasks > n) return fail("item tasks", i);
    if (it.ntasks * G > 16) return fail("item columns", i, it.ntasks);
    if (it.kv_head < 0 || it.kv_head >= Hkv) return fail("item head", i);
    if (it.k_begin < 0 || it.k_end <= it.k_begin) return fail("item keys", i);
    const int g = group_of[it.first_task];
    if (group_of[it.first_task + it.ntasks - 1] != g) return fail("item spans groups", i);
    const bool prompt = it.k_end <= sh[g] && it.split < (sh[g] + plan.chunk - 1) / plan.chunk;
    if (!prompt && (it.ntasks != 1 || it.k_begin < sh[g])) return fail("own item", i);
    const int len = it.k_end - it.k_begin;
    if (len > prev_len) return fail("not longest first", i);
    prev_len = len;
    for (int t = it.first_task; t < it.first_task + it.ntasks; ++t) {
      if (it.k_end > kv[t]) return fail("item past context", i, t);
      auto& m = cover[{t, it.kv_head}];
      if (!m.insert({it.split, {it.k_begin, it.k_end}}).second) return fail("split twice", t, it.split);
    }
  }
  int32_t max_splits = 0;
  for (int32_t b = 0; b < n; ++b) {
    if (tasks[b].row_start != b) return fail("row_start", b);
    max_splits = std::max(max_splits, tasks[b].aux);
    for (int32_t h = 0; h < Hkv; ++h) {
      const auto& m = cover[{b, h}];
      if ((int)m.size() != tasks[b].aux) return fail("split count", b, (long)m.size());
      int at = 0, s = 0;
      for (const auto& kvp : m) {
        if (kvp.first != s++) return fail("split ids", b, kvp.first);
        if (kvp.second.first != at) return fail("key gap", b, at);
        at = kvp.second.second;
      }
      if (at != kv[b]) return fail("keys end", b, at);
    }
  }
  if (plan.max_splits < max_splits) return fail("max splits", plan.max_splits, max_splits);
  printf("ok %d %d %d %zu\n", plan.num_items, plan.chunk, plan.max_splits, plan.total_bytes);
  return 0;
}

int main() {
  std::string line;
  int bad = 0;
  while (std::getline(std::cin, line)) {
    std::istringstream in(line);
    int op, hq, hkv, d, n;
    if (!(in >> op >> hq >> hkv >> d >> n)) continue;
    tide_dims dims = {};
    dims.num_q_heads = hq;
    dims.num_kv_heads = hkv;
    dims.head_dim = d;
    dims.page_size = 16;
    dims.sm_scale = 0.088f;
    if (op == TIDE_OP_DECODE || op == kOpDecodeShared) {
      int splits = 0, ng = 0;
      in >> splits;
      std::vector<int32_t> gs, sh;
      if (op == kOpDecodeShared) {
        in >> ng;
        gs.resize(ng + 1);
        sh.resize(ng);
        for (auto& x : gs) in >> x;
        for (auto& x : sh) in >> x;
      }
      std::vector<int32_t> kv(n);
      for (auto& x : kv) in >> x;
      bad |= op == TIDE_OP_DECODE ? check_decode(dims, splits, kv) : check_shared(dims, splits, kv, gs, sh);
    } else {
      std::vector<int32_t> pa(n), pb(n);
      for (int i = 0; i < n; ++i) in >> pa[i] >> pb[i];
      if (op == TIDE_OP_FULL_PREFILL) pa = pb;
      bad |= check(op, dims, pa, pb);
    }
    fflush(stdout);
  }
  return bad;
}
