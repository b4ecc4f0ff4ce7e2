// Host-side planning: validation, workspace layout and work lists (see plan.h).
#include "plan.h"

#include <math.h>
#include <string.h>

#include <algorithm>
#include <numeric>

namespace tide {

int check_dims(const tide_dims* dims) {
  if (!dims) return TIDE_ERR_INVALID_ARG;
  if (dims->num_q_heads <= 0 || dims->num_kv_heads <= 0 || dims->head_dim <= 0 ||
      dims->page_size <= 0)
    return TIDE_ERR_INVALID_ARG;
  if (!(dims->sm_scale > 0.0f) || !isfinite(dims->sm_scale)) return TIDE_ERR_INVALID_ARG;
  if (dims->head_dim != 64 && dims->head_dim != 128) return TIDE_ERR_UNSUPPORTED;
  if (dims->page_size != kPage) return TIDE_ERR_UNSUPPORTED;
  if (dims->num_q_heads % dims->num_kv_heads != 0) return TIDE_ERR_UNSUPPORTED;
  if (dims->num_q_heads / dims->num_kv_heads > kMaxGroup) return TIDE_ERR_UNSUPPORTED;
  return TIDE_OK;
}

int32_t extend_waves(int32_t head_dim, int32_t group) {
  (void)head_dim;
  (void)group;
  return 8;
}

namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Per-task (prefix, extend) of the positions this call touches or attends.
int task_lengths(int op, int32_t b, const int32_t* lens_a, const int32_t* lens_b, int32_t* prefix,
                 int32_t* extend) {
  switch (op) {
    case TIDE_OP_KV_APPEND:
    case TIDE_OP_EXTEND:
      *prefix = lens_a[b];
      *extend = lens_b[b];
      if (*prefix < 0 || *extend < 0) return TIDE_ERR_INVALID_ARG;
      break;
    case TIDE_OP_FULL_PREFILL:
      *prefix = 0;
      *extend = lens_a[b];
      if (*extend < 0) return TIDE_ERR_INVALID_ARG;
      break;
    case TIDE_OP_DECODE:
      if (lens_a[b] <= 0) return TIDE_ERR_INVALID_ARG;
      *prefix = lens_a[b] - 1;
      *extend = 1;
      break;
    default:
      return TIDE_ERR_INVALID_ARG;
  }
  if ((int64_t)*prefix + *extend > INT32_MAX) return TIDE_ERR_INVALID_ARG;
  return TIDE_OK;
}

}  // namespace

int make_plan(int op, int32_t num_tasks, const int32_t* lens_a, const int32_t* lens_b,
              const tide_dims& dims, int32_t num_splits, int32_t bt_stride, bool build_blob,
              Plan* plan) {
  if (!plan) return TIDE_ERR_INVALID_ARG;
  if (op != TIDE_OP_KV_APPEND && op != TIDE_OP_EXTEND && op != TIDE_OP_DECODE &&
      op != TIDE_OP_FULL_PREFILL)
    return TIDE_ERR_INVALID_ARG;
  if (num_tasks < 0) return TIDE_ERR_INVALID_ARG;
  if (num_tasks > 0 && !lens_a) return TIDE_ERR_INVALID_ARG;
  if (num_tasks > 0 && (op == TIDE_OP_KV_APPEND || op == TIDE_OP_EXTEND) && !lens_b)
    return TIDE_ERR_INVALID_ARG;
  if (op == TIDE_OP_DECODE && num_splits < 0) return TIDE_ERR_INVALID_ARG;
  int rc = check_dims(&dims);
  if (rc != TIDE_OK) return rc;

  const int32_t group = dims.num_q_heads / dims.num_kv_heads;
  *plan = Plan();
  plan->op = op;
  plan->num_tasks = num_tasks;

  std::vector<TaskDesc> tasks((size_t)num_tasks);
  int64_t rows = 0;
  int64_t max_len = 0;
  for (int32_t b = 0; b < num_tasks; ++b) {
    int32_t p = 0, e = 0;
    rc = task_lengths(op, b, lens_a, lens_b, &p, &e);
    if (rc != TIDE_OK) return rc;
    tasks[b].row_start = (int32_t)(op == TIDE_OP_DECODE ? b : rows);
    tasks[b].prefix = p;
    tasks[b].extend = e;
    tasks[b].aux = 0;
    rows += (op == TIDE_OP_DECODE) ? 1 : e;
    if (rows > INT32_MAX) return TIDE_ERR_INVALID_ARG;
    max_len = std::max<int64_t>(max_len, (int64_t)p + e);
    if (bt_stride >= 0 && ceil_div((int64_t)p + e, kPage) > bt_stride) return TIDE_ERR_CAPACITY;
  }
  plan->total_rows = (int32_t)rows;

  // ---- work items -------------------------------------------------------------------
  std::vector<uint8_t> items_bytes;
  int64_t n_items = 0;
  if (op == TIDE_OP_KV_APPEND) {
    std::vector<AppendItem> items;
    for (int32_t b = 0; b < num_tasks; ++b) {
      const int32_t p = tasks[b].prefix, e = tasks[b].extend;
      if (e == 0) continue;
      for (int64_t lp = p / kPage; lp <= (int64_t)(p + e - 1) / kPage; ++lp) {
        AppendItem it;
        it.task = b;
        it.lpage = (int32_t)lp;
        it.pos_begin = (int32_t)std::max<int64_t>(p, lp * kPage);
        it.pos_end = (int32_t)std::min<int64_t>((int64_t)p + e, (lp + 1) * kPage);
        items.push_back(it);
      }
    }
    n_items = (int64_t)items.size();
    if (build_blob) {
      items_bytes.resize(items.size() * sizeof(AppendItem));
      if (!items.empty()) memcpy(items_bytes.data(), items.data(), items_bytes.size());
    }
  } else if (op == TIDE_OP_EXTEND || op == TIDE_OP_FULL_PREFILL) {
    const int32_t waves = extend_waves(dims.head_dim, group);
    const int32_t tb = waves * 32 / group;  // tokens per item: waves*32 rows of (token, head)
    plan->waves = waves;
    plan->tokens_per_item = tb;
    // Work units are (task, kv head): all query blocks of a unit read the same K/V.
    // Workgroups are dispatched round-robin over the XCDs (item i runs on XCD i % 8),
    // each with its own L2.  Every unit is placed on one XCD, its blocks consecutive in
    // that XCD's order, so the blocks that walk the same K/V run side by side and share
    // it through L2 instead of re-reading HBM.  Units go longest first to the least
    // loaded XCD; inside a unit the longest blocks go first.
    struct Unit {
      int64_t cost;
      int32_t task, kv_head;
    };
    std::vector<Unit> units;
    for (int32_t b = 0; b < num_tasks; ++b) {
      const int32_t p = tasks[b].prefix, e = tasks[b].extend;
      if (e == 0) continue;
      int64_t cost = 0;
      for (int32_t t0 = 0; t0 < e; t0 += tb) {
        const int32_t n = std::min(tb, e - t0);
        cost += (int64_t)n * ((int64_t)p + t0 + n);
      }
      for (int32_t g = 0; g < dims.num_kv_heads; ++g) units.push_back({cost, b, g});
    }
    std::stable_sort(units.begin(), units.end(),
                     [](const Unit& x, const Unit& y) { return x.cost > y.cost; });
    std::vector<std::vector<ExtendItem>> queues(kXcds);
    std::vector<int64_t> load(kXcds, 0);
    for (const Unit& u : units) {
      const int x = (int)(std::min_element(load.begin(), load.end()) - load.begin());
      load[x] += u.cost;
      const int32_t p = tasks[u.task].prefix, e = tasks[u.task].extend;
      const int32_t nblk = (e + tb - 1) / tb;
      for (int32_t k = nblk - 1; k >= 0; --k) {  // later blocks see more keys
        ExtendItem it;
        it.task = u.task;
        it.kv_head = u.kv_head;
        it.tok0 = k * tb;
        it.ntok = std::min(tb, e - k * tb);
        queues[x].push_back(it);
      }
      (void)p;
    }
    size_t depth = 0;
    for (const auto& qx : queues) depth = std::max(depth, qx.size());
    std::vector<ExtendItem> items(depth * kXcds);
    for (size_t i = 0; i < depth; ++i)
      for (int x = 0; x < kXcds; ++x) {
        ExtendItem it = {0, 0, 0, 0};  // ntok == 0: an empty slot the kernel skips
        if (i < queues[x].size()) it = queues[x][i];
        items[i * kXcds + x] = it;
      }
    while (!items.empty() && items.back().ntok == 0) items.pop_back();
    n_items = (int64_t)items.size();
    if (build_blob) {
      items_bytes.resize(items.size() * sizeof(ExtendItem));
      if (!items.empty()) memcpy(items_bytes.data(), items.data(), items_bytes.size());
    }
  } else {  // decode
    int64_t chunk = 0;
    if (num_splits > 0) {
      for (int32_t b = 0; b < num_tasks; ++b)
        chunk = std::max<int64_t>(chunk, ceil_div(tasks[b].prefix + 1, num_splits));
      chunk = std::max<int64_t>(kDecodeStep, ceil_div(chunk, kDecodeStep) * kDecodeStep);
    } else {
      int64_t total = 0;
      for (int32_t b = 0; b < num_tasks; ++b) total += (int64_t)tasks[b].prefix + 1;
      total *= dims.num_kv_heads;
      chunk = ceil_div(total, 8192);
      chunk = ceil_div(chunk, kDecodeStep) * kDecodeStep;
      chunk = std::min<int64_t>(std::max<int64_t>(chunk, 256), 16384);
    }
    int32_t max_splits = 0;
    std::vector<DecodeItem> items;
    for (int32_t b = 0; b < num_tasks; ++b) {
      const int64_t kv = (int64_t)tasks[b].prefix + 1;
      const int32_t s = (int32_t)ceil_div(kv, chunk);
      tasks[b].aux = s;
      max_splits = std::max(max_splits, s);
      for (int32_t sp = 0; sp < s; ++sp)
        for (int32_t g = 0; g < dims.num_kv_heads; ++g) {
          DecodeItem it;
          it.task = b;
          it.kv_head = g;
          it.split = sp;
          it.k_begin = (int32_t)(sp * chunk);
          items.push_back(it);
        }
    }
    plan->chunk = (int32_t)chunk;
    plan->max_splits = max_splits;
    n_items = (int64_t)items.size();
    if (build_blob) {
      items_bytes.resize(items.size() * sizeof(DecodeItem));
      if (!items.empty()) memcpy(items_bytes.data(), items.data(), items_bytes.size());
    }
  }
  if (n_items > INT32_MAX / 4) return TIDE_ERR_INVALID_ARG;
  plan->num_items = (int32_t)n_items;

  // ---- layout -------------------------------------------------------------------------
  size_t off = sizeof(WsHeader);
  plan->tasks_off = off;
  off = align_up(off + tasks.size() * sizeof(TaskDesc), kWsAlign);
  plan->items_off = off;
  off = align_up(off + (size_t)n_items * 16, kWsAlign);
  plan->upload_bytes = off;
  if (op == TIDE_OP_DECODE) {
    const size_t slots = (size_t)num_tasks * dims.num_q_heads * (size_t)plan->max_splits;
    plan->part_o_off = off;
    off = align_up(off + slots * dims.head_dim * sizeof(float), kWsAlign);
    plan->part_ml_off = off;
    off = align_up(off + slots * 4 * sizeof(float), kWsAlign);
  }
  plan->total_bytes = off;

  if (build_blob) {
    plan->blob.assign(plan->upload_bytes, 0);
    if (!tasks.empty())
      memcpy(plan->blob.data() + plan->tasks_off, tasks.data(), tasks.size() * sizeof(TaskDesc));
    if (!items_bytes.empty())
      memcpy(plan->blob.data() + plan->items_off, items_bytes.data(), items_bytes.size());
  }
  return TIDE_OK;
}

int make_plan_shared(int32_t num_tasks, const int32_t* kv_lens, int32_t num_groups,
                     const int32_t* group_start, const int32_t* shared_lens,
                     const tide_dims& dims, int32_t num_splits, int32_t bt_stride,
                     bool build_blob, Plan* plan) {
  if (!plan) return TIDE_ERR_INVALID_ARG;
  int rc = check_dims(&dims);
  if (rc != TIDE_OK) return rc;
  if (num_tasks < 0 || num_splits < 0 || num_groups < 0) return TIDE_ERR_INVALID_ARG;
  *plan = Plan();
  plan->op = kOpDecodeShared;
  plan->num_tasks = num_tasks;
  if (num_tasks > 0) {
    if (!kv_lens || !group_start || !shared_lens || num_groups < 1) return TIDE_ERR_INVALID_ARG;
    if (group_start[0] != 0 || group_start[num_groups] != num_tasks) return TIDE_ERR_INVALID_ARG;
  }
  const int32_t group = dims.num_q_heads / dims.num_kv_heads;
  const int32_t per_item = std::max<int32_t>(1, 16 / group);  // trajectories per prefix item

  std::vector<TaskDesc> tasks((size_t)num_tasks);
  std::vector<int32_t> shared_of((size_t)num_tasks, 0);
  for (int32_t g = 0; g < (num_tasks > 0 ? num_groups : 0); ++g) {
    const int32_t s0 = group_start[g], s1 = group_start[g + 1];
    const int32_t sh = shared_lens[g];
    if (s1 <= s0 || s1 > num_tasks) return TIDE_ERR_INVALID_ARG;
    if (sh < 0 || sh % kPage != 0) return TIDE_ERR_INVALID_ARG;
    for (int32_t b = s0; b < s1; ++b) {
      if (kv_lens[b] <= 0 || sh > kv_lens[b] - 1) return TIDE_ERR_INVALID_ARG;
      if (bt_stride >= 0 && ceil_div(kv_lens[b], kPage) > bt_stride) return TIDE_ERR_CAPACITY;
      tasks[b] = TaskDesc{b, kv_lens[b] - 1, 1, 0};
      shared_of[b] = sh;
    }
  }
  plan->total_rows = num_tasks;

  // Chunk length: the same rule as decode, counting a shared prefix once per item group.
  int64_t chunk = 0;
  if (num_splits > 0) {
    for (int32_t b = 0; b < num_tasks; ++b)
      chunk = std::max<int64_t>(chunk, ceil_div(kv_lens[b], num_splits));
    chunk = std::max<int64_t>(kDecodeStep, ceil_div(chunk, kDecodeStep) * kDecodeStep);
  } else {
    int64_t total = 0;
    for (int32_t g = 0; g < (num_tasks > 0 ? num_groups : 0); ++g) {
      const int32_t n = group_start[g + 1] - group_start[g];
      total += ceil_div(n, per_item) * (int64_t)shared_lens[g];
    }
    for (int32_t b = 0; b < num_tasks; ++b) total += (int64_t)kv_lens[b] - shared_of[b];
    total *= dims.num_kv_heads;
    chunk = ceil_div(total, 8192);
    chunk = ceil_div(chunk, kDecodeStep) * kDecodeStep;
    chunk = std::min<int64_t>(std::max<int64_t>(chunk, 256), 16384);
  }

  std::vector<SharedDecodeItem> items;
  int32_t max_splits = 0;
  for (int32_t g = 0; g < (num_tasks > 0 ? num_groups : 0); ++g) {
    const int32_t s0 = group_start[g], s1 = group_start[g + 1], sh = shared_lens[g];
    const int32_t np = (int32_t)ceil_div(sh, chunk);
    for (int32_t f = s0; f < s1; f += per_item)
      for (int32_t h = 0; h < dims.num_kv_heads; ++h)
        for (int32_t j = 0; j < np; ++j) {
          SharedDecodeItem it = {};
          it.first_task = f;
          it.ntasks = std::min(per_item, s1 - f);
          it.kv_head = h;
          it.split = j;
          it.k_begin = (int32_t)(j * chunk);
          it.k_end = (int32_t)std::min<int64_t>(sh, (j + 1) * chunk);
          items.push_back(it);
        }
    for (int32_t b = s0; b < s1; ++b) {
      const int32_t ns = (int32_t)ceil_div((int64_t)kv_lens[b] - sh, chunk);
      tasks[b].aux = np + ns;
      max_splits = std::max(max_splits, np + ns);
      for (int32_t h = 0; h < dims.num_kv_heads; ++h)
        for (int32_t i = 0; i < ns; ++i) {
          SharedDecodeItem it = {};
          it.first_task = b;
          it.ntasks = 1;
          it.kv_head = h;
          it.split = np + i;
          it.k_begin = (int32_t)(sh + i * chunk);
          it.k_end = (int32_t)std::min<int64_t>(kv_lens[b], sh + (i + 1) * chunk);
          items.push_back(it);
        }
    }
  }
  if ((int64_t)items.size() > INT32_MAX / 4) return TIDE_ERR_INVALID_ARG;
  plan->chunk = (int32_t)chunk;
  plan->max_splits = max_splits;
  plan->num_items = (int32_t)items.size();

  size_t off = sizeof(WsHeader);
  plan->tasks_off = off;
  off = align_up(off + tasks.size() * sizeof(TaskDesc), kWsAlign);
  plan->items_off = off;
  off = align_up(off + items.size() * sizeof(SharedDecodeItem), kWsAlign);
  plan->upload_bytes = off;
  const size_t slots = (size_t)num_tasks * dims.num_q_heads * (size_t)max_splits;
  plan->part_o_off = off;
  off = align_up(off + slots * dims.head_dim * sizeof(float), kWsAlign);
  plan->part_ml_off = off;
  off = align_up(off + slots * 4 * sizeof(float), kWsAlign);
  plan->total_bytes = off;
  if (build_blob) {
    plan->blob.assign(plan->upload_bytes, 0);
    if (!tasks.empty())
      memcpy(plan->blob.data() + plan->tasks_off, tasks.data(), tasks.size() * sizeof(TaskDesc));
    if (!items.empty())
      memcpy(plan->blob.data() + plan->items_off, items.data(), items.size() * sizeof(SharedDecodeItem));
  }
  return TIDE_OK;
}

}  // namespace tide
