// Host-side Continuous Task Batching scheduler (Section 4) and the request-level
// baseline it is compared with (Section 6.5), driving the paged-KV engine model described
// in include/tide_ctb.h.
//
// Data structures (all per rank unless noted):
//   free list   FIFO deque of page ids
//   LRU list    intrusive doubly linked list over page ids (prev/next arrays); the head
//               is the least recently released cached page
//   owner       (task, logical index) of every held or cached page
//   active / paused   task-id sets with O(1) removal (the priority key ends in the task
//               id, so scans over them never depend on their order)
// Token usage per rank is recomputed when a rank's scheduling starts and then updated
// as tasks are paused, resumed and admitted (footprints do not change while a rank is
// being scheduled).
#include "tide_ctb.h"

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <deque>
#include <new>
#include <unordered_map>
#include <vector>

namespace {

constexpr int32_t kPage = 16;

inline int64_t pages_for(int64_t n) { return (n + kPage - 1) / kPage; }

enum class State : uint8_t { New, Active, Paused, Done };

struct Task {
  int32_t id = 0, group = 0, is_eval = 0;
  int32_t turn0 = 0, num_turns = 0;  // turns in the trace arrays
  State state = State::New;
  int32_t rank = -1;
  int32_t turn = 0;
  int64_t ctx = 0;          // tokens in the sequence so far
  int64_t kv_valid = 0;     // leading tokens whose K/V are in the task's pages
  int64_t pending_new = 0;  // input tokens of the current turn not yet appended
  int64_t to_gen = 0;       // tokens still to generate in the current turn
  int64_t env_done = -1;    // round at which the environment answers
  std::vector<int32_t> pages;
  int32_t slot = -1;        // position in the rank's active or paused set
};

// A set of task ids with O(1) insert and erase (tasks remember their slot).
struct IdSet {
  std::vector<int32_t> ids;
  void insert(std::vector<Task>& tasks, int32_t id) {
    tasks[id].slot = static_cast<int32_t>(ids.size());
    ids.push_back(id);
  }
  void erase(std::vector<Task>& tasks, int32_t id) {
    int32_t s = tasks[id].slot;
    int32_t last = ids.back();
    ids[s] = last;
    tasks[last].slot = s;
    ids.pop_back();
    tasks[id].slot = -1;
  }
};

struct Pool {
  std::deque<int32_t> free_list;
  std::vector<int32_t> prev, next;
  std::vector<uint8_t> in_lru;
  std::vector<int32_t> owner_task, owner_idx;
  int32_t head = -1, tail = -1;
  int64_t lru_size = 0;
  // pages given up by the ops of the round being executed: a round is one batched
  // engine iteration, so they become reusable (free) or evictable (LRU) when it ends
  std::vector<int32_t> later_free, later_lru;

  explicit Pool(int32_t n)
      : prev(n, -1), next(n, -1), in_lru(n, 0), owner_task(n, -1), owner_idx(n, -1) {
    for (int32_t p = 0; p < n; ++p) free_list.push_back(p);
  }
  void lru_push_back(int32_t p) {
    prev[p] = tail;
    next[p] = -1;
    if (tail >= 0) next[tail] = p; else head = p;
    tail = p;
    in_lru[p] = 1;
    ++lru_size;
  }
  void lru_remove(int32_t p) {
    if (prev[p] >= 0) next[prev[p]] = next[p]; else head = next[p];
    if (next[p] >= 0) prev[next[p]] = prev[p]; else tail = prev[p];
    prev[p] = next[p] = -1;
    in_lru[p] = 0;
    --lru_size;
  }
  int64_t available() const { return static_cast<int64_t>(free_list.size()) + lru_size; }

  // Gives `task` its next page.  The caller guarantees one is available.
  int32_t alloc(Task& task, std::vector<Task>& tasks) {
    int32_t page;
    if (!free_list.empty()) {
      page = free_list.front();
      free_list.pop_front();
    } else {
      page = head;
      lru_remove(page);
      Task& v = tasks[owner_task[page]];
      const int32_t idx = owner_idx[page];
      // the owner keeps only the pages before idx; the later ones can no longer hit
      for (size_t j = static_cast<size_t>(idx) + 1; j < v.pages.size(); ++j) {
        const int32_t p = v.pages[j];
        lru_remove(p);
        owner_task[p] = owner_idx[p] = -1;
        free_list.push_back(p);
      }
      v.pages.resize(static_cast<size_t>(idx));
      v.kv_valid = std::min<int64_t>(v.kv_valid, static_cast<int64_t>(idx) * kPage);
    }
    owner_task[page] = task.id;
    owner_idx[page] = static_cast<int32_t>(task.pages.size());
    task.pages.push_back(page);
    return page;
  }
  // Held pages become cached, the last page first (at the end of the round if `later`).
  void release(const Task& t, bool later = false) {
    for (size_t j = t.pages.size(); j-- > 0;) {
      if (later) later_lru.push_back(t.pages[j]); else lru_push_back(t.pages[j]);
    }
  }
  // Cached pages become held again.
  void reclaim(const Task& t) {
    for (int32_t p : t.pages) lru_remove(p);
  }
  // A finished task's pages return to the free list when the round ends.
  void drop(Task& t) {
    for (int32_t p : t.pages) {
      owner_task[p] = owner_idx[p] = -1;
      later_free.push_back(p);
    }
    t.pages.clear();
    t.kv_valid = 0;
  }
  void end_round() {
    for (int32_t p : later_free) free_list.push_back(p);
    for (int32_t p : later_lru) lru_push_back(p);
    later_free.clear();
    later_lru.clear();
  }
};

struct Sim {
  tide_ctb_config cfg{};
  std::vector<Task> tasks;
  std::vector<int32_t> new_tok, gen_tok, env_rnd;
  std::vector<int32_t> group_size, group_done, group_rank, group_probe;
  std::vector<Pool> pools;
  std::vector<IdSet> active, paused;
  // arrival-order queue of tasks not yet admitted/started
  std::vector<int32_t> new_order;
  std::vector<uint8_t> new_taken;
  size_t new_head = 0;
  int64_t live = 0;  // CTB: admitted, unfinished tasks
  // request policy
  std::vector<std::deque<int32_t>> waiting;
  std::vector<std::vector<int32_t>> running;
  std::vector<int64_t> rank_tasks;  // tasks started on the rank and not finished
  int64_t in_flight = 0;
  // environment answers by round
  std::unordered_map<int64_t, std::vector<int32_t>> env_due;
  int64_t round = 0;
  int64_t remaining = 0;
  tide_ctb_stats stats{};
  // output of the last round
  std::vector<tide_ctb_op> ops;
  std::vector<int32_t> op_pages;
  std::vector<tide_ctb_event> events;

  // ------------------------------------------------------------------ helpers
  int64_t footprint(const Task& t) const {
    return kPage * pages_for(t.ctx + t.pending_new + (t.to_gen > 0 ? 1 : 0));
  }
  static int executing(const Task& t) { return (t.pending_new > 0 || t.to_gen > 0) ? 1 : 0; }

  // true if a ranks strictly below b in P(t), then arrival order (a larger key is kept)
  bool lower(const Task& a, const Task& b) const {
    if (a.is_eval != b.is_eval) return a.is_eval < b.is_eval;
    const int64_t ga = static_cast<int64_t>(group_done[a.group]) * group_size[b.group];
    const int64_t gb = static_cast<int64_t>(group_done[b.group]) * group_size[a.group];
    if (ga != gb) return ga < gb;
    const int ea = executing(a), eb = executing(b);
    if (ea != eb) return ea < eb;
    if (a.ctx != b.ctx) return a.ctx < b.ctx;
    return a.id > b.id;
  }

  void event(int32_t kind, const Task& t, int32_t rank) {
    events.push_back(tide_ctb_event{kind, t.id, rank, 0});
  }

  void load_turn(Task& t) {
    const int32_t k = t.turn0 + t.turn;
    t.pending_new = new_tok[k];
    t.to_gen = gen_tok[k];
  }

  // ------------------------------------------------------------------ round steps
  void env_completions() {
    auto it = env_due.find(round);
    if (it == env_due.end()) return;
    std::vector<int32_t> due = std::move(it->second);
    env_due.erase(it);
    std::sort(due.begin(), due.end());
    for (int32_t id : due) {
      Task& t = tasks[id];
      t.env_done = -1;
      t.turn += 1;
      load_turn(t);
      if (cfg.policy == TIDE_CTB_POLICY_REQUEST) waiting[t.rank].push_back(id);
    }
  }

  int32_t next_new(int32_t r) {
    while (new_head < new_order.size() && new_taken[new_head]) ++new_head;
    for (size_t i = new_head; i < new_order.size(); ++i) {
      if (new_taken[i]) continue;
      const Task& t = tasks[new_order[i]];
      if (group_rank[t.group] == -1 || group_rank[t.group] == r) return static_cast<int32_t>(i);
    }
    return -1;
  }

  void schedule_ctb() {
    const int64_t B = cfg.budget_tokens;
    for (int32_t r = 0; r < cfg.num_ranks; ++r) {
      Pool& pool = pools[r];
      int64_t u = 0;
      for (int32_t id : active[r].ids) u += footprint(tasks[id]);
      while (u > B) {
        int32_t victim = -1;
        for (int32_t id : active[r].ids)
          if (victim < 0 || lower(tasks[id], tasks[victim])) victim = id;
        Task& t = tasks[victim];
        active[r].erase(tasks, victim);
        paused[r].insert(tasks, victim);
        t.state = State::Paused;
        pool.release(t);
        u -= footprint(t);
        ++stats.pauses;
        event(TIDE_CTB_EV_PAUSE, t, r);
      }
      while (u < B) {
        int32_t best = -1;
        for (int32_t id : paused[r].ids) {
          const Task& t = tasks[id];
          if (u + footprint(t) > B) continue;
          if (best < 0 || lower(tasks[best], t)) best = id;
        }
        if (best >= 0) {
          Task& t = tasks[best];
          paused[r].erase(tasks, best);
          active[r].insert(tasks, best);
          t.state = State::Active;
          pool.reclaim(t);
          u += footprint(t);
          ++stats.resumes;
          event(TIDE_CTB_EV_RESUME, t, r);
          continue;
        }
        const int32_t qi = next_new(r);
        if (qi >= 0) {
          Task& t = tasks[new_order[qi]];
          const bool fits = u + group_probe[t.group] <= B;
          const bool env_ok = cfg.env_capacity <= 0 || live < cfg.env_capacity;
          if (fits && env_ok) {
            new_taken[qi] = 1;
            t.state = State::Active;
            t.rank = r;
            if (group_rank[t.group] < 0) group_rank[t.group] = r;
            load_turn(t);
            active[r].insert(tasks, t.id);
            ++live;
            u += footprint(t);
            ++stats.admits;
            event(TIDE_CTB_EV_ADMIT, t, r);
            continue;
          }
        }
        break;
      }
    }
  }

  void execute_ctb() {
    std::vector<int32_t> work;
    for (int32_t r = 0; r < cfg.num_ranks; ++r) {
      work.clear();
      for (int32_t id : active[r].ids) {
        const Task& t = tasks[id];
        if (t.pending_new > 0 || t.to_gen > 0 || t.kv_valid < t.ctx) work.push_back(id);
      }
      std::sort(work.begin(), work.end(),
                [&](int32_t a, int32_t b) { return lower(tasks[b], tasks[a]); });
      const size_t n = std::min(work.size(), static_cast<size_t>(cfg.max_running));
      for (size_t i = 0; i < n; ++i) run_op(tasks[work[i]], r);
    }
  }

  void record_op(int32_t r, int32_t kind, const Task& t, int64_t start, int64_t count) {
    tide_ctb_op op;
    op.rank = r;
    op.kind = kind;
    op.task = t.id;
    op.start = static_cast<int32_t>(start);
    op.count = static_cast<int32_t>(count);
    op.num_pages = static_cast<int32_t>(t.pages.size());
    op.page_offset = static_cast<int64_t>(op_pages.size());
    op_pages.insert(op_pages.end(), t.pages.begin(), t.pages.end());
    ops.push_back(op);
  }

  void run_op(Task& t, int32_t r) {
    Pool& pool = pools[r];
    if (t.kv_valid < t.ctx || t.pending_new > 0) {
      const int64_t P = t.kv_valid;
      const int64_t E = t.ctx + t.pending_new - P;
      while (static_cast<int64_t>(t.pages.size()) < pages_for(P + E)) pool.alloc(t, tasks);
      record_op(r, TIDE_CTB_OP_EXTEND, t, P, E);
      ++stats.extend_ops;
      stats.hit_tokens += P;
      stats.queried_tokens += P + E;
      stats.extend_tokens += E;
      t.ctx += t.pending_new;
      t.pending_new = 0;
      t.kv_valid = t.ctx;
    } else {
      const int64_t pos = t.ctx;
      while (static_cast<int64_t>(t.pages.size()) < pages_for(pos + 1)) pool.alloc(t, tasks);
      record_op(r, TIDE_CTB_OP_DECODE, t, pos, 1);
      ++stats.decode_ops;
      t.ctx += 1;
      t.kv_valid = t.ctx;
      t.to_gen -= 1;
      if (t.to_gen == 0) end_turn(t, r);
    }
  }

  void remove_running(int32_t r, int32_t id) {
    auto& run = running[r];
    run.erase(std::find(run.begin(), run.end(), id));
  }

  void end_turn(Task& t, int32_t r) {
    if (t.turn == t.num_turns - 1) {
      pools[r].drop(t);
      if (cfg.policy == TIDE_CTB_POLICY_CTB) {
        active[r].erase(tasks, t.id);
        --live;
      }
      t.state = State::Done;
      group_done[t.group] += 1;
      --remaining;
      event(TIDE_CTB_EV_FINISH, t, r);
      if (cfg.policy == TIDE_CTB_POLICY_REQUEST) {
        remove_running(r, t.id);
        --in_flight;
        --rank_tasks[r];
      }
    } else {
      t.env_done = round + env_rnd[t.turn0 + t.turn];
      env_due[t.env_done].push_back(t.id);
      if (cfg.policy == TIDE_CTB_POLICY_REQUEST) {
        remove_running(r, t.id);
        pools[r].release(t, /*later=*/true);
        t.state = State::Paused;
      }
    }
  }

  int64_t op_pages_after(const Task& t) const {
    if (t.kv_valid < t.ctx || t.pending_new > 0) return pages_for(t.ctx + t.pending_new);
    return pages_for(t.ctx + 1);
  }

  void schedule_request() {
    while (new_head < new_order.size() && in_flight < cfg.max_in_flight) {
      Task& t = tasks[new_order[new_head]];
      new_taken[new_head] = 1;
      ++new_head;
      int32_t r = 0;
      for (int32_t i = 1; i < cfg.num_ranks; ++i)
        if (rank_tasks[i] < rank_tasks[r]) r = i;
      t.rank = r;
      t.state = State::Paused;
      load_turn(t);
      ++in_flight;
      ++rank_tasks[r];
      ++stats.admits;
      event(TIDE_CTB_EV_ADMIT, t, r);
      waiting[r].push_back(t.id);
    }
    for (int32_t r = 0; r < cfg.num_ranks; ++r) {
      Pool& pool = pools[r];
      auto& run = running[r];
      int64_t avail = pool.available();
      int64_t need = 0;
      bool preempted = false;
      size_t i = 0;
      while (i < run.size()) {
        Task& t = tasks[run[i]];
        int64_t want = op_pages_after(t) - static_cast<int64_t>(t.pages.size());
        while (need + want > avail) {
          preempted = true;
          Task& v = tasks[run.back()];
          run.pop_back();
          pool.release(v);
          v.state = State::Paused;
          avail += static_cast<int64_t>(v.pages.size());
          ++stats.pauses;
          event(TIDE_CTB_EV_PAUSE, v, r);
          waiting[r].push_front(v.id);
          if (&v == &t) {
            want = 0;
            break;
          }
        }
        if (t.state == State::Active) {
          need += want;
          ++i;
        }
      }
      while (!waiting[r].empty() && !preempted &&
             static_cast<int64_t>(run.size()) < cfg.max_running) {
        Task& t = tasks[waiting[r].front()];
        const int64_t cached = static_cast<int64_t>(t.pages.size());
        const int64_t want = op_pages_after(t) - cached;
        if (need + want > avail - cached) break;
        waiting[r].pop_front();
        pool.reclaim(t);
        avail -= cached;
        need += want;
        t.state = State::Active;
        run.push_back(t.id);
        ++stats.resumes;
        event(TIDE_CTB_EV_RESUME, t, r);
      }
    }
  }

  void execute_request() {
    std::vector<int32_t> order;
    for (int32_t r = 0; r < cfg.num_ranks; ++r) {
      order = running[r];
      for (int32_t id : order) run_op(tasks[id], r);
    }
  }

  void step() {
    ops.clear();
    op_pages.clear();
    events.clear();
    env_completions();
    if (cfg.policy == TIDE_CTB_POLICY_CTB) {
      schedule_ctb();
      execute_ctb();
    } else {
      schedule_request();
      execute_request();
    }
    for (Pool& p : pools) p.end_round();
    ++round;
    stats.rounds = round;
  }
};

int validate(const tide_ctb_config* cfg, int32_t num_tasks, const int32_t* group,
             const int32_t* is_eval, int32_t num_groups, const int32_t* group_size,
             const int32_t* turn_start, const int32_t* new_tokens, const int32_t* gen_tokens,
             const int32_t* env_rounds) {
  if (!cfg || num_tasks < 0 || num_groups < 0) return TIDE_ERR_INVALID_ARG;
  if (cfg->policy != TIDE_CTB_POLICY_CTB && cfg->policy != TIDE_CTB_POLICY_REQUEST)
    return TIDE_ERR_INVALID_ARG;
  if (cfg->num_ranks < 1 || cfg->pages_per_rank < 1 || cfg->max_running < 1 ||
      cfg->max_in_flight < 1 || cfg->env_capacity < 0 || cfg->max_rounds < 1)
    return TIDE_ERR_INVALID_ARG;
  const int64_t pool_tokens = static_cast<int64_t>(cfg->pages_per_rank) * kPage;
  if (cfg->budget_tokens < 1 || cfg->budget_tokens > pool_tokens) return TIDE_ERR_INVALID_ARG;
  if (num_tasks == 0) return TIDE_OK;
  if (!group || !is_eval || !group_size || !turn_start || !new_tokens || !gen_tokens ||
      !env_rounds)
    return TIDE_ERR_INVALID_ARG;
  if (turn_start[0] != 0) return TIDE_ERR_INVALID_ARG;
  for (int32_t g = 0; g < num_groups; ++g)
    if (group_size[g] < 1) return TIDE_ERR_INVALID_ARG;
  std::vector<int32_t> prompt(static_cast<size_t>(num_groups), -1);
  for (int32_t t = 0; t < num_tasks; ++t) {
    const int32_t a = turn_start[t], b = turn_start[t + 1];
    if (b <= a || group[t] < 0 || group[t] >= num_groups) return TIDE_ERR_INVALID_ARG;
    if (new_tokens[a] < 1) return TIDE_ERR_INVALID_ARG;
    int32_t& pr = prompt[static_cast<size_t>(group[t])];
    if (pr < 0) pr = new_tokens[a];
    if (pr != new_tokens[a]) return TIDE_ERR_INVALID_ARG;
    int64_t total = 0;
    for (int32_t k = a; k < b; ++k) {
      if (new_tokens[k] < 0 || gen_tokens[k] < 1 || env_rounds[k] < 1)
        return TIDE_ERR_INVALID_ARG;
      total += static_cast<int64_t>(new_tokens[k]) + gen_tokens[k];
    }
    const int64_t need = kPage * pages_for(total + 1);
    if (need > pool_tokens) return TIDE_ERR_INVALID_ARG;
    if (cfg->policy == TIDE_CTB_POLICY_CTB && need > cfg->budget_tokens)
      return TIDE_ERR_INVALID_ARG;
    if (total + 1 > INT32_MAX) return TIDE_ERR_INVALID_ARG;
  }
  return TIDE_OK;
}

}  // namespace

extern "C" int tide_ctb_create(
    const tide_ctb_config* cfg, int32_t num_tasks, const int32_t* group, const int32_t* is_eval,
    int32_t num_groups, const int32_t* group_size, const int32_t* turn_start,
    const int32_t* new_tokens, const int32_t* gen_tokens, const int32_t* env_rounds,
    void** sim_out) {
  if (!sim_out) return TIDE_ERR_INVALID_ARG;
  *sim_out = nullptr;
  int st = validate(cfg, num_tasks, group, is_eval, num_groups, group_size, turn_start,
                    new_tokens, gen_tokens, env_rounds);
  if (st != TIDE_OK) return st;
  try {
    Sim* s = new Sim();
    s->cfg = *cfg;
    const int32_t nturns = num_tasks ? turn_start[num_tasks] : 0;
    s->new_tok.assign(new_tokens, new_tokens + nturns);
    s->gen_tok.assign(gen_tokens, gen_tokens + nturns);
    s->env_rnd.assign(env_rounds, env_rounds + nturns);
    s->group_size.assign(group_size, group_size + num_groups);
    s->group_done.assign(static_cast<size_t>(num_groups), 0);
    s->group_rank.assign(static_cast<size_t>(num_groups), -1);
    s->group_probe.assign(static_cast<size_t>(num_groups), -1);
    s->tasks.resize(static_cast<size_t>(num_tasks));
    for (int32_t t = 0; t < num_tasks; ++t) {
      Task& x = s->tasks[t];
      x.id = t;
      x.group = group[t];
      x.is_eval = is_eval[t] ? 1 : 0;
      x.turn0 = turn_start[t];
      x.num_turns = turn_start[t + 1] - turn_start[t];
      for (int32_t k = x.turn0; k < x.turn0 + x.num_turns; ++k) s->stats.input_tokens += new_tokens[k];
      // the probe: first-turn usage (prompt + first generation) of the group's first
      // trajectory in arrival order
      if (s->group_probe[x.group] < 0)
        s->group_probe[x.group] = static_cast<int32_t>(
            kPage * pages_for(static_cast<int64_t>(new_tokens[x.turn0]) + gen_tokens[x.turn0] + 1));
    }
    s->pools.reserve(static_cast<size_t>(cfg->num_ranks));
    for (int32_t r = 0; r < cfg->num_ranks; ++r) s->pools.emplace_back(cfg->pages_per_rank);
    s->active.resize(static_cast<size_t>(cfg->num_ranks));
    s->paused.resize(static_cast<size_t>(cfg->num_ranks));
    s->waiting.resize(static_cast<size_t>(cfg->num_ranks));
    s->running.resize(static_cast<size_t>(cfg->num_ranks));
    s->rank_tasks.assign(static_cast<size_t>(cfg->num_ranks), 0);
    s->new_order.resize(static_cast<size_t>(num_tasks));
    for (int32_t t = 0; t < num_tasks; ++t) s->new_order[t] = t;
    s->new_taken.assign(static_cast<size_t>(num_tasks), 0);
    s->remaining = num_tasks;
    *sim_out = s;
    return TIDE_OK;
  } catch (const std::bad_alloc&) {
    return TIDE_ERR_CAPACITY;
  }
}

extern "C" int tide_ctb_step(void* sim, tide_ctb_round* out) {
  if (!sim || !out) return TIDE_ERR_INVALID_ARG;
  Sim* s = static_cast<Sim*>(sim);
  std::memset(out, 0, sizeof(*out));
  if (s->remaining == 0) {
    s->ops.clear();
    s->op_pages.clear();
    s->events.clear();
    out->round = static_cast<int32_t>(s->round);
    out->done = 1;
    return TIDE_OK;
  }
  if (s->round >= s->cfg.max_rounds) return TIDE_ERR_CAPACITY;
  try {
    s->step();
  } catch (const std::bad_alloc&) {
    return TIDE_ERR_CAPACITY;
  }
  out->round = static_cast<int32_t>(s->round - 1);
  out->done = s->remaining == 0 ? 1 : 0;
  out->num_ops = static_cast<int32_t>(s->ops.size());
  out->num_events = static_cast<int32_t>(s->events.size());
  out->num_pages = static_cast<int64_t>(s->op_pages.size());
  out->ops = s->ops.data();
  out->pages = s->op_pages.data();
  out->events = s->events.data();
  return TIDE_OK;
}

extern "C" int tide_ctb_get_stats(const void* sim, tide_ctb_stats* out) {
  if (!sim || !out) return TIDE_ERR_INVALID_ARG;
  *out = static_cast<const Sim*>(sim)->stats;
  return TIDE_OK;
}

extern "C" int tide_ctb_destroy(void* sim) {
  delete static_cast<Sim*>(sim);
  return TIDE_OK;
}
