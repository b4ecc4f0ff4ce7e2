// Drives the native task-batching scheduler (csrc/ctb.cpp, include/tide_ctb.h) over
// random traces under both policies until every task finishes, and over invalid
// arguments, so that a sanitizer build (test_sanitizers.py: g++ with
// -fsanitize=address,undefined) checks every access it makes.  Checks only what every
// round must satisfy (ids and page ids in range, page counts matching the op); the
// scheduling decisions are pinned against the plain oracle by test_ctb_parity.py.
// Exits 0 when every check held.
#include <stdint.h>
#include <stdio.h>

#include <vector>

#include "tide_ctb.h"

static uint64_t state = 0x243F6A8885A308D3ull;
static uint32_t next() {  // xorshift64*
  state ^= state >> 12;
  state ^= state << 25;
  state ^= state >> 27;
  return (uint32_t)((state * 0x2545F4914F6CDD1Dull) >> 32);
}
static int pick(int n) { return (int)(next() % (uint32_t)n); }

static long total_rounds = 0, total_ops = 0;

static int run_trace(int trial) {
  const int groups = 1 + pick(6);
  std::vector<int32_t> group, is_eval, group_size(groups), turn_start{0}, newt, gen, env;
  int max_ctx = 0;
  for (int g = 0; g < groups; ++g) {
    group_size[g] = 1 + pick(5);
    const int prompt = 1 + pick(200);
    const int eval = pick(4) == 0;
    for (int k = 0; k < group_size[g]; ++k) {
      group.push_back(g);
      is_eval.push_back(eval);
      const int turns = 1 + pick(5);
      int ctx = 0;
      for (int t = 0; t < turns; ++t) {
        newt.push_back(t == 0 ? prompt : 1 + pick(120));
        gen.push_back(1 + pick(200));
        env.push_back(1 + pick(4));
        ctx += newt.back() + gen.back();
      }
      turn_start.push_back((int32_t)newt.size());
      if (ctx > max_ctx) max_ctx = ctx;
    }
  }
  const int n = (int)group.size();
  tide_ctb_config cfg;
  cfg.policy = pick(2) ? TIDE_CTB_POLICY_CTB : TIDE_CTB_POLICY_REQUEST;
  cfg.num_ranks = 1 + pick(3);
  // a task needs the pages of its whole context plus one token, in whole pages
  const int need = 16 * ((max_ctx + 1 + 15) / 16);
  cfg.pages_per_rank = need / 16 + pick(200);
  cfg.budget_tokens = cfg.pages_per_rank * 16 - pick(8);
  if (cfg.budget_tokens < need) cfg.budget_tokens = need;
  cfg.max_running = 1 + pick(16);
  cfg.max_in_flight = 1 + pick(32);
  cfg.env_capacity = pick(3) ? 0 : 1 + pick(20);
  cfg.max_rounds = 200000;
  void* sim = nullptr;
  int rc = tide_ctb_create(&cfg, n, group.data(), is_eval.data(), groups, group_size.data(),
                           turn_start.data(), newt.data(), gen.data(), env.data(), &sim);
  if (rc != TIDE_OK) {
    printf("trial %d: create rc %d\n", trial, rc);
    return 1;
  }
  int bad = 0;
  for (int r = 0; r < cfg.max_rounds; ++r) {
    tide_ctb_round out;
    rc = tide_ctb_step(sim, &out);
    if (rc != TIDE_OK) {
      printf("trial %d: step rc %d\n", trial, rc);
      bad = 1;
      break;
    }
    for (int i = 0; i < out.num_ops; ++i) {
      const tide_ctb_op& op = out.ops[i];
      const bool ok = op.rank >= 0 && op.rank < cfg.num_ranks && op.task >= 0 && op.task < n &&
                      (op.kind == TIDE_CTB_OP_EXTEND || op.kind == TIDE_CTB_OP_DECODE) &&
                      op.start >= 0 && op.count >= 1 &&
                      op.num_pages == (op.start + op.count + 15) / 16 && op.page_offset >= 0 &&
                      op.page_offset + op.num_pages <= out.num_pages;
      if (!ok) {
        printf("trial %d: bad op %d in round %d\n", trial, i, r);
        bad = 1;
        continue;
      }
      for (int p = 0; p < op.num_pages; ++p) {
        const int32_t id = out.pages[op.page_offset + p];
        if (id < 0 || id >= cfg.pages_per_rank) {
          printf("trial %d: page id %d out of range\n", trial, id);
          bad = 1;
        }
      }
    }
    total_rounds += 1;
    total_ops += out.num_ops;
    for (int i = 0; i < out.num_events; ++i)
      if (out.events[i].task < 0 || out.events[i].task >= n) bad = 1;
    if (out.done) break;
  }
  tide_ctb_stats st;
  if (tide_ctb_get_stats(sim, &st) != TIDE_OK) bad = 1;
  tide_ctb_destroy(sim);
  return bad;
}

static int bad_arguments() {
  int bad = 0;
  int32_t group[2] = {0, 0}, is_eval[2] = {0, 0}, gsz[1] = {2}, ts[3] = {0, 1, 2};
  int32_t newt[2] = {10, 11}, gen[2] = {1, 1}, env[2] = {1, 1};  // prompts differ in a group
  tide_ctb_config cfg = {TIDE_CTB_POLICY_CTB, 1, 16, 256, 4, 4, 0, 1000};
  void* sim = nullptr;
  if (tide_ctb_create(&cfg, 2, group, is_eval, 1, gsz, ts, newt, gen, env, &sim) == TIDE_OK) bad = 1;
  tide_ctb_destroy(sim);
  sim = nullptr;
  newt[1] = 10;
  cfg.budget_tokens = 5;  // a task's context cannot fit
  if (tide_ctb_create(&cfg, 2, group, is_eval, 1, gsz, ts, newt, gen, env, &sim) == TIDE_OK) bad = 1;
  tide_ctb_destroy(sim);
  sim = nullptr;
  cfg.budget_tokens = 256;
  cfg.num_ranks = 0;
  if (tide_ctb_create(&cfg, 2, group, is_eval, 1, gsz, ts, newt, gen, env, &sim) == TIDE_OK) bad = 1;
  tide_ctb_destroy(sim);
  if (tide_ctb_step(nullptr, nullptr) == TIDE_OK) bad = 1;
  if (tide_ctb_destroy(nullptr) != TIDE_OK) bad = 1;
  if (bad) printf("bad arguments accepted\n");
  return bad;
}

int main() {
  int bad = bad_arguments();
  for (int t = 0; t < 300; ++t) bad |= run_trace(t);
  printf("%ld rounds, %ld ops\n", total_rounds, total_ops);
  printf(bad ? "FAIL\n" : "ok\n");
  return bad;
}
