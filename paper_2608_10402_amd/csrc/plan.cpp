// Host-side planning: validation, workspace layout and work lists (see plan.h).
#include "plan.h"

#include <math.h>
#include <stdlib.h>
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
  if (dims->num_kv_heads > kMaxKvHeads) return TIDE_ERR_UNSUPPORTED;
  return TIDE_OK;
}

int32_t extend_waves(int32_t head_dim, int32_t group) {
  (void)head_dim;
  (void)group;
  return 8;
}

namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Automatic decode chunk.  The device holds 2048 decode waves at once (8 per CU).  When
// most (task, kv head) units are cut into several chunks, the items are nearly all full
// chunks and a launch of n items runs in about ceil(n / 2048) rounds, each about as long
// as a chunk plus a fixed cost (first loads, partial stores, a wave's start and end); a
// launch just above a multiple of 2048 items then leaves a mostly empty last round.  So
// for every round count R the planner takes the shortest chunk whose items fit in R
// rounds and keeps the R with the least R * (kDecodeRoundCost + chunk).  When that gives
// fewer than 4 chunks per unit, most items are units' shorter last chunks of scattered
// lengths; many items then balance the launch better, and the chunk is
// sum(kv) * Hkv / 4096 keys.  Chunks are multiples of the kernel step within [512, 16384].
// Measured on MI355X over 15 shapes (8-1024 tasks, 0.6k-60k keys, 2-8 kv heads, GQA
// 4:1 to 8:1): the round rule is 8-11% faster on agent_resume_7b, multimodal_resume,
// long_horizon and the prune resume than about 4096 items, and 5% slower on
// resumed_decode (2 chunks per unit), where the item count rule stays.
constexpr int64_t kDecodeWaveSlots = 2048;
constexpr int64_t kDecodeRoundCost = 1200;  // keys
constexpr int64_t kDecodeMinUnitChunks = 4;
constexpr int64_t kDecodeMaxRoundsTried = 8;
constexpr int64_t kDecodeMinChunk = 512;
constexpr int64_t kDecodeMaxChunk = 16384;
constexpr int64_t kDecodeTargetItems = 4096;
constexpr int64_t kFoldMeanSplits = 4;  // merge inside the split kernel up to this mean

// The automatic decode chunk (see kDecodeRoundCost).  Round rule: for R rounds from the
// fewest that can hold the items, the shortest chunk (a multiple of the kernel step) whose
// items fit in R * 2048 waves, scored R * (kDecodeRoundCost + chunk); items fall as the
// chunk grows, so each R is a binary search.  R stops growing once the shortest allowed
// chunk fits, once R rounds of it already score worse than the best found, or after
// kDecodeMaxRoundsTried values (a few dozen passes over the tasks per call).  Item rule,
// when the round rule would leave fewer than 4 chunks per unit (or cannot reach 4 at
// all): sum(kv) * Hkv / 4096 keys.
int64_t decode_auto_chunk(const std::vector<TaskDesc>& tasks, int32_t hkv) {
  const int64_t units = (int64_t)tasks.size() * hkv;
  // Items for a chunk of m kernel steps: Hkv * sum over tasks of ceil(kv / (32 m)), from
  // each task's length in steps (32-bit divisions: this runs a few dozen times per call).
  std::vector<uint32_t> steps(tasks.size());
  for (size_t b = 0; b < tasks.size(); ++b)
    steps[b] = (uint32_t)ceil_div((int64_t)tasks[b].prefix + 1, kDecodeStep);
  auto items_at = [&](int64_t m) {
    int64_t n = 0;
    for (uint32_t k : steps) n += (k + (uint32_t)m - 1) / (uint32_t)m;
    return n * hkv;
  };
  auto item_rule = [&]() {
    int64_t total = 0;
    for (const TaskDesc& t : tasks) total += (int64_t)t.prefix + 1;
    int64_t c = ceil_div(total * hkv, kDecodeTargetItems);
    c = ceil_div(c, kDecodeStep) * kDecodeStep;
    return std::min<int64_t>(std::max<int64_t>(c, kDecodeMinChunk), kDecodeMaxChunk);
  };
  if (items_at(kDecodeMinChunk / kDecodeStep) < kDecodeMinUnitChunks * units) return item_rule();
  const int64_t lo_step = kDecodeMinChunk / kDecodeStep, hi_step = kDecodeMaxChunk / kDecodeStep;
  const int64_t r0 = std::max<int64_t>(1, ceil_div(items_at(kDecodeMaxChunk / kDecodeStep),
                                                   kDecodeWaveSlots));
  int64_t best = kDecodeMaxChunk, best_score = INT64_MAX;
  int64_t hi_prev = hi_step;  // R rounds' chunk also fits R + 1 rounds: the next search's top
  for (int64_t r = r0; r < r0 + kDecodeMaxRoundsTried; ++r) {
    if (r * (kDecodeRoundCost + kDecodeMinChunk) >= best_score) break;  // cannot win
    const int64_t cap = r * kDecodeWaveSlots;
    int64_t lo = lo_step, hi = hi_prev;  // in kernel steps; items_at(hi) <= cap
    if (items_at(lo) <= cap) hi = lo;
    while (hi - lo > 1) {
      const int64_t mid = (lo + hi) / 2;
      if (items_at(mid) <= cap) hi = mid;
      else lo = mid;
    }
    hi_prev = hi;
    const int64_t c = hi * kDecodeStep;
    const int64_t score = r * (kDecodeRoundCost + c);
    if (score < best_score) {
      best_score = score;
      best = c;
    }
    if (hi == lo_step) break;  // more rounds can only add cost
  }
  if (items_at(best / kDecodeStep) < kDecodeMinUnitChunks * units) return item_rule();
  return best;
}

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

// ---- extend / prefill work lists ------------------------------------------------------
//
// A work item is one block of tb = 256 / G tokens of one (task, kv head): its 256 query
// rows are the block's (token, head) pairs, and one 8-wave workgroup, which fills a CU,
// walks the key tiles (64 keys) the block sees.  Two plans are considered:
//   plain  every item walks all its tiles and writes its rows;
//   split  a block that spans many tiles is cut into chunks of about T tiles that run on
//          different CUs and write unnormalised fp32 partials, which a second kernel
//          merges (the split-K scheme of flash decoding, applied to extend blocks).
// Splitting pays when a call has too few items to keep 256 CUs busy to the end.  The
// choice compares closed-form run-time estimates: the makespan of n workgroups costing
// c_i tiles each on 256 CUs is max c when n <= 256 (all start at once), and is taken as
// max(max c, sum c / 256 + max c / 2) otherwise; a tile costs less while few CUs are
// busy (the clock is higher), and a split plan adds the merge's HBM traffic and launch.
// The planner runs on every call, so everything here is linear in the number of blocks,
// and only the chosen plan is materialised.
namespace {

constexpr int kCus = 256;  // MI355X compute units, 32 per XCD
// Cost model, in units of one key tile of one workgroup at full occupancy; the overheads
// and rates were fitted to measured one- to 64-task calls (GQA 28/4, d = 128).
constexpr double kItemOverhead = 0.5;     // first-tile latency and epilogue
constexpr double kChunkOverhead = 2.5;    // the same plus the fp32 partial write
constexpr double kCuFlopsPerUs = 3.9e6;   // sustained MFMA rate of one CU, all CUs busy
constexpr double kIdleClockGain = 0.25;   // a tile is up to this much cheaper with idle CUs
constexpr double kHbmBytesPerUs = 5.0e6;  // sustained HBM rate of the merge
constexpr double kMergeLaunchUs = 4.0;    // second kernel launch
constexpr double kSplitGain = 1.0;        // split whenever estimated faster
constexpr int kMinChunkTiles = 8;
constexpr int kMaxChunks = 512;
constexpr int64_t kSplitMaxItems = 2048;  // larger calls fill the chip with the plain plan

struct Block {
  int32_t task, tok0, ntok, ntiles;
};

// Chunks of a block for chunk length T: about ntiles / T (at most kMaxChunks), on a
// fixed grid [c*T, (c+1)*T) whose last chunk takes the rest (up to 1.5 T below the cap),
// so the same chunk of a unit's blocks covers the same keys.  T == 0: the plain plan
// (one chunk).
inline int32_t num_chunks(int32_t ntiles, int32_t T) {
  if (T <= 0) return 1;
  return (int32_t)std::min<int64_t>(kMaxChunks, std::max<int64_t>(1, (ntiles + T / 2) / T));
}

inline int32_t chunk_tiles(int32_t ntiles, int32_t T, int32_t n, int32_t c) {
  return c == n - 1 ? ntiles - c * T : T;
}

inline double chunk_cost(int32_t ntiles, int32_t T, int32_t n, int32_t c) {
  return chunk_tiles(ntiles, T, n, c) + (n > 1 ? kChunkOverhead : kItemOverhead);
}

// Estimated run time (us) of the plan with chunk length T (0: plain).
double estimate(const std::vector<Block>& blocks, int32_t num_kv_heads, int32_t num_q_heads,
                int32_t head_dim, int32_t T, double tile_us, int64_t* row_slots) {
  double total = 0.0, biggest = 0.0;
  int64_t items = 0, slots = 0;
  for (const Block& b : blocks) {
    const int32_t n = num_chunks(b.ntiles, T);
    items += n;
    if (n > 1) slots += (int64_t)b.ntok * n;
    total += (n - 1) * chunk_cost(b.ntiles, T, n, 0) + chunk_cost(b.ntiles, T, n, n - 1);
    for (int32_t c : {0, n - 1}) biggest = std::max(biggest, chunk_cost(b.ntiles, T, n, c));
  }
  items *= num_kv_heads;
  total *= num_kv_heads;
  const double busy = std::min(1.0, (double)items / kCus);
  const double t_eff = tile_us * (1.0 - kIdleClockGain * (1.0 - busy));
  // up to one workgroup per CU, all start at once and the longest one ends the call
  const double span = items <= kCus ? biggest : std::max(biggest, total / kCus + 0.5 * biggest);
  double us = span * t_eff;
  if (slots > 0)
    us += (double)slots * num_q_heads * (head_dim * 4.0 + 16.0) * 2.0 / kHbmBytesPerUs +
          kMergeLaunchUs;
  *row_slots = slots;
  return us;
}

// Consecutive blocks [k0, k1) of one task (longest first), chunk c (-1: whole blocks)
// of kv head g.  Workgroups of a piece read the same K/V.
struct Piece {
  double cost;
  int32_t k0, k1, g, c;
};

// Item order.  Workgroups are dispatched round-robin over the XCDs (slot i runs on XCD
// i % 8), each with its own L2.  A column -- one (task, kv head, chunk) -- is kept on one
// XCD, its items consecutive, so workgroups that walk the same K/V run side by side and
// share it through L2 instead of re-reading HBM.  A column longer than a quarter of an
// XCD's share is cut into consecutive pieces first, so that a call with fewer units than
// XCDs still reaches every XCD; pieces then go longest first to the least loaded XCD.
// Returns, per XCD, its pieces in order.
std::vector<std::vector<Piece>> place(const std::vector<Block>& blocks,
                                      const std::vector<int32_t>& task_first,
                                      const std::vector<int32_t>& nchunks, int32_t num_kv_heads,
                                      int32_t T) {
  const int32_t ntasks = (int32_t)task_first.size() - 1;
  std::vector<Piece> cols;
  double total = 0.0, biggest = 0.0;
  for (int32_t b = 0; b < ntasks; ++b) {
    const int32_t k0 = task_first[b], k1 = task_first[b + 1];
    if (k0 == k1) continue;
    const int32_t nmax = nchunks[k0];  // chunk counts do not grow along a task's blocks
    for (int32_t c = 0; c < nmax; ++c) {
      int32_t end = k0;
      double cost = 0.0;
      while (end < k1 && nchunks[end] > c) {
        const double ci = chunk_cost(blocks[end].ntiles, T, nchunks[end], c);
        cost += ci;
        biggest = std::max(biggest, ci);
        ++end;
      }
      for (int32_t g = 0; g < num_kv_heads; ++g)
        cols.push_back(Piece{cost, k0, end, g, T > 0 ? c : -1});
      total += cost * num_kv_heads;
    }
  }
  const double cap = std::max(biggest, total / (kXcds * 4));
  std::vector<Piece> pieces;
  pieces.reserve(cols.size());
  for (const Piece& col : cols) {
    const int32_t c = std::max(col.c, 0);
    Piece cur{0.0, col.k0, col.k0, col.g, col.c};
    for (int32_t k = col.k0; k < col.k1; ++k) {
      const double ci = chunk_cost(blocks[k].ntiles, T, nchunks[k], c);
      if (cur.k1 > cur.k0 && cur.cost + ci > cap) {
        pieces.push_back(cur);
        cur = Piece{0.0, k, k, col.g, col.c};
      }
      cur.k1 = k + 1;
      cur.cost += ci;
    }
    if (cur.k1 > cur.k0) pieces.push_back(cur);
  }
  std::stable_sort(pieces.begin(), pieces.end(),
                   [](const Piece& x, const Piece& y) { return x.cost > y.cost; });
  std::vector<std::vector<Piece>> queues(kXcds);
  double load[kXcds] = {};
  for (const Piece& p : pieces) {
    const int x = (int)(std::min_element(load, load + kXcds) - load);
    load[x] += p.cost;
    queues[x].push_back(p);
  }
  return queues;
}

// Item slots in dispatch order: slot i * 8 + x is the i-th item of XCD x's queue, and an
// XCD whose queue ran out gets empty slots (ntok == 0) that return at once.
template <class Item, class Make>
std::vector<Item> interleave(const std::vector<std::vector<Piece>>& queues, Make make) {
  std::vector<std::vector<Item>> per(kXcds);
  size_t depth = 0;
  for (int x = 0; x < kXcds; ++x) {
    for (const Piece& p : queues[x])
      for (int32_t k = p.k0; k < p.k1; ++k) per[x].push_back(make(k, p.g, std::max(p.c, 0)));
    depth = std::max(depth, per[x].size());
  }
  std::vector<Item> items(depth * kXcds);  // value-initialised: ntok == 0
  for (int x = 0; x < kXcds; ++x)
    for (size_t i = 0; i < per[x].size(); ++i) items[i * kXcds + x] = per[x][i];
  while (!items.empty() && items.back().ntok == 0) items.pop_back();
  return items;
}

template <class Item>
void to_bytes(const std::vector<Item>& v, std::vector<uint8_t>* out) {
  out->resize(v.size() * sizeof(Item));
  if (!v.empty()) memcpy(out->data(), v.data(), out->size());
}

int plan_extend(const std::vector<TaskDesc>& tasks, const tide_dims& dims, bool build_blob,
                Plan* plan, std::vector<uint8_t>* items_bytes, std::vector<uint8_t>* merge_bytes,
                int64_t* n_items) {
  const int32_t group = dims.num_q_heads / dims.num_kv_heads;
  const int32_t waves = extend_waves(dims.head_dim, group);
  const int32_t tb = waves * 32 / group;  // tokens per item: waves*32 rows of (token, head)
  const int32_t hkv = dims.num_kv_heads;
  plan->waves = waves;
  plan->tokens_per_item = tb;
  // one workgroup-tile: 64 keys against 256 query rows, two products
  const double tile_us = 4.0 * kExtendKeyTile * (waves * 32) * dims.head_dim / kCuFlopsPerUs;

  // Blocks of each task, latest first (later blocks see more keys).
  const int32_t ntasks = (int32_t)tasks.size();
  std::vector<int32_t> task_first((size_t)ntasks + 1, 0);
  int64_t nblocks = 0;
  for (int32_t b = 0; b < ntasks; ++b) nblocks += (tasks[b].extend + tb - 1) / tb;
  if (nblocks * hkv > INT32_MAX / 4) return TIDE_ERR_INVALID_ARG;
  std::vector<Block> blocks;
  blocks.reserve((size_t)nblocks);
  for (int32_t b = 0; b < ntasks; ++b) {
    task_first[b] = (int32_t)blocks.size();
    const int32_t p = tasks[b].prefix, e = tasks[b].extend;
    for (int32_t k = (e + tb - 1) / tb - 1; k >= 0; --k) {
      Block bl;
      bl.task = b;
      bl.tok0 = k * tb;
      bl.ntok = std::min(tb, e - k * tb);
      bl.ntiles = (int32_t)(((int64_t)p + bl.tok0 + bl.ntok + kExtendKeyTile - 1) / kExtendKeyTile);
      blocks.push_back(bl);
    }
  }
  task_first[ntasks] = (int32_t)blocks.size();
  const int64_t plain_items = nblocks * hkv;

  // TIDE_EXTEND_SPLIT=0 keeps the plain plan, =1 takes the best split plan whenever one
  // exists (both for tests and tuning); otherwise the estimate decides.
  const char* env = getenv("TIDE_EXTEND_SPLIT");
  const int mode = (env && env[0] == '0') ? 0 : (env && env[0] == '1') ? 1 : -1;
  int32_t T = 0;
  if (mode != 0 && plain_items > 0 && plain_items <= kSplitMaxItems) {
    int64_t slots = 0;
    const double plain_us =
        estimate(blocks, hkv, dims.num_q_heads, dims.head_dim, 0, tile_us, &slots);
    plan->est_plain_us = plan->est_us = plain_us;
    double best_us = mode == 1 ? INFINITY : plain_us * kSplitGain;
    int64_t tiles = 0;
    for (const Block& b : blocks) tiles += b.ntiles;
    int64_t last = -1;
    for (int rounds = 1; rounds <= 4; ++rounds) {
      const int64_t t = std::max<int64_t>(
          kMinChunkTiles, (tiles * hkv + (int64_t)rounds * kCus - 1) / ((int64_t)rounds * kCus));
      if (t > INT32_MAX / 2 || t == last) continue;
      last = t;
      const double us =
          estimate(blocks, hkv, dims.num_q_heads, dims.head_dim, (int32_t)t, tile_us, &slots);
      if (slots > 0 && slots <= INT32_MAX / 2 && us < best_us) {
        best_us = plan->est_us = us;
        T = (int32_t)t;
      }
    }
  }

  std::vector<int32_t> nchunks(blocks.size());
  for (size_t k = 0; k < blocks.size(); ++k) nchunks[k] = num_chunks(blocks[k].ntiles, T);
  const std::vector<std::vector<Piece>> queues = place(blocks, task_first, nchunks, hkv, T);
  plan->split = T > 0;
  if (T == 0) {
    const std::vector<ExtendItem> items = interleave<ExtendItem>(
        queues, [&](int32_t k, int32_t g, int32_t) {
          return ExtendItem{blocks[k].task, g, blocks[k].tok0, blocks[k].ntok};
        });
    *n_items = (int64_t)items.size();
    if (build_blob) to_bytes(items, items_bytes);
    return TIDE_OK;
  }

  // partial row slots of the split blocks
  std::vector<int32_t> pbase(blocks.size(), 0);
  int64_t slots = 0;
  for (size_t k = 0; k < blocks.size(); ++k)
    if (nchunks[k] > 1) {
      pbase[k] = (int32_t)slots;
      slots += (int64_t)blocks[k].ntok * nchunks[k];
    }
  plan->row_slots = slots;
  const std::vector<ExtendChunkItem> items = interleave<ExtendChunkItem>(
      queues, [&](int32_t k, int32_t g, int32_t c) {
        const int32_t n = nchunks[k];
        ExtendChunkItem it;
        it.task = blocks[k].task;
        it.kv_head = g;
        it.tok0 = blocks[k].tok0;
        it.ntok = blocks[k].ntok;
        it.t_begin = c * T;
        it.t_end = it.t_begin + chunk_tiles(blocks[k].ntiles, T, n, c);
        it.split = n > 1 ? c : -1;
        it.pbase = pbase[k];
        return it;
      });
  *n_items = (int64_t)items.size();
  if (build_blob) {
    to_bytes(items, items_bytes);
    std::vector<MergeRow> rows((size_t)plan->total_rows, MergeRow{0, 0, 0, 0});
    for (size_t k = 0; k < blocks.size(); ++k) {
      if (nchunks[k] < 2) continue;
      const int32_t r0 = tasks[blocks[k].task].row_start + blocks[k].tok0;
      for (int32_t tk = 0; tk < blocks[k].ntok; ++tk)
        rows[r0 + tk] = MergeRow{pbase[k] + tk, blocks[k].ntok, nchunks[k], 0};
    }
    to_bytes(rows, merge_bytes);
  }
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
  std::vector<uint8_t> items_bytes, merge_bytes;
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
    rc = plan_extend(tasks, dims, build_blob, plan, &items_bytes, &merge_bytes, &n_items);
    if (rc != TIDE_OK) return rc;
  } else {  // decode
    int64_t chunk = 0;
    if (num_splits > 0) {
      for (int32_t b = 0; b < num_tasks; ++b)
        chunk = std::max<int64_t>(chunk, ceil_div(tasks[b].prefix + 1, num_splits));
      chunk = std::max<int64_t>(kDecodeStep, ceil_div(chunk, kDecodeStep) * kDecodeStep);
    } else {
      chunk = decode_auto_chunk(tasks, dims.num_kv_heads);
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
    // Longest first: the shorter last chunks of the tasks then run at the end of the
    // launch, while the CUs that free up early still find work (the result does not
    // depend on the order: each split writes its own partial slot).
    {
      auto keys = [&](const DecodeItem& x) {
        return std::min<int64_t>(chunk, (int64_t)tasks[x.task].prefix + 1 - x.k_begin);
      };
      std::vector<DecodeItem> tail;  // every task's last, shorter chunk
      size_t nfull = 0;
      for (const DecodeItem& it : items) {
        if (keys(it) == chunk) items[nfull++] = it;
        else tail.push_back(it);
      }
      std::stable_sort(tail.begin(), tail.end(),
                       [&](const DecodeItem& x, const DecodeItem& y) { return keys(x) > keys(y); });
      std::copy(tail.begin(), tail.end(), items.begin() + nfull);
    }
    plan->chunk = (int32_t)chunk;
    plan->max_splits = max_splits;
    n_items = (int64_t)items.size();
    // The split kernel merges a (task, kv head) in its last split when tasks have few
    // splits on average; with many, the merge tail at the end of the launch (each merge
    // one wave, latency-bound) costs more than a merge kernel (measured on MI355X: at 2.5
    // splits per task the fold saves the merge kernel's 10 us; at 16 it adds 40-57 us).
    // (and the partial rows of one (task, kv head) must fit a 32-bit buffer range)
    plan->fold_merge = n_items <= (int64_t)kFoldMeanSplits * num_tasks * dims.num_kv_heads &&
                       (int64_t)(dims.num_q_heads / dims.num_kv_heads) * max_splits *
                               dims.head_dim * 4 <= INT32_MAX;
    if (build_blob) {
      items_bytes.resize(items.size() * sizeof(DecodeItem));
      if (!items.empty()) memcpy(items_bytes.data(), items.data(), items_bytes.size());
    }
  }
  if (n_items > INT32_MAX / 4) return TIDE_ERR_INVALID_ARG;
  plan->num_items = (int32_t)n_items;
  const size_t item_size = plan->split ? sizeof(ExtendChunkItem) : 16;

  // ---- layout -------------------------------------------------------------------------
  size_t off = sizeof(WsHeader);
  plan->tasks_off = off;
  off = align_up(off + tasks.size() * sizeof(TaskDesc), kWsAlign);
  plan->items_off = off;
  off = align_up(off + (size_t)n_items * item_size, kWsAlign);
  if (plan->split) {
    plan->merge_rows_off = off;
    off = align_up(off + (size_t)plan->total_rows * sizeof(MergeRow), kWsAlign);
  }
  if (op == TIDE_OP_DECODE) {  // left zero in the blob: every call starts the counts at 0
    plan->tickets_off = off;
    off = align_up(off + (size_t)num_tasks * dims.num_kv_heads * sizeof(int32_t), kWsAlign);
  }
  plan->upload_bytes = off;
  if (plan->split) {
    const size_t slots = (size_t)plan->row_slots * dims.num_q_heads;
    plan->part_o_off = off;
    off = align_up(off + slots * dims.head_dim * sizeof(float), kWsAlign);
    plan->part_ml_off = off;
    off = align_up(off + slots * 4 * sizeof(float), kWsAlign);
  }
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
    if (plan->split && !merge_bytes.empty())
      memcpy(plan->blob.data() + plan->merge_rows_off, merge_bytes.data(), merge_bytes.size());
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
    chunk = ceil_div(total, kDecodeTargetItems);
    chunk = ceil_div(chunk, kDecodeStep) * kDecodeStep;
    chunk = std::min<int64_t>(std::max<int64_t>(chunk, kDecodeMinChunk), kDecodeMaxChunk);
  }

  std::vector<SharedDecodeItem> items;
  int32_t max_splits = 0;
  for (int32_t g = 0; g < (num_tasks > 0 ? num_groups : 0); ++g) {
    const int32_t s0 = group_start[g], s1 = group_start[g + 1], sh = shared_lens[g];
    const int32_t np = (int32_t)ceil_div(sh, chunk);
    // The items of one (kv head, chunk) -- one per run of per_item trajectories -- read the
    // same prefix keys.  They are consecutive, so they share a workgroup of the decode
    // kernel (four or eight waves by launch size, one item each, on one CU) or a
    // neighbouring one, and the later reads hit that XCD's L2.
    for (int32_t h = 0; h < dims.num_kv_heads; ++h)
      for (int32_t j = 0; j < np; ++j)
        for (int32_t f = s0; f < s1; f += per_item) {
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
  // Longest first, as for plain decode.  The sort is stable and the items of one prompt
  // chunk have equal lengths and are adjacent, so they stay adjacent.
  std::stable_sort(items.begin(), items.end(),
                   [](const SharedDecodeItem& x, const SharedDecodeItem& y) {
                     return x.k_end - x.k_begin > y.k_end - y.k_begin;
                   });
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
