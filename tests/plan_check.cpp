// Host-side checker of the extend / prefill work lists built by the planner (plan.cpp),
// compiled with g++ by test_plan.py; no GPU involved.
//
// Each stdin line is one call: "op hq hkv d ntasks p_0 e_0 p_1 e_1 ..." (op 2 = extend,
// 4 = full prefill, which reads e_i as the sequence length and ignores p_i).  For every
// call the checker builds the plan, reads the uploaded blob back and verifies what the
// kernels assume:
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

int main() {
  std::string line;
  int bad = 0;
  while (std::getline(std::cin, line)) {
    std::istringstream in(line);
    int op, hq, hkv, d, n;
    if (!(in >> op >> hq >> hkv >> d >> n)) continue;
    std::vector<int32_t> pa(n), pb(n);
    for (int i = 0; i < n; ++i) in >> pa[i] >> pb[i];
    tide_dims dims = {};
    dims.num_q_heads = hq;
    dims.num_kv_heads = hkv;
    dims.head_dim = d;
    dims.page_size = 16;
    dims.sm_scale = 0.088f;
    if (op == TIDE_OP_FULL_PREFILL) pa = pb;
    bad |= check(op, dims, pa, pb);
    fflush(stdout);
  }
  return bad;
}
