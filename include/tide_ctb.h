/*
 * tide_ctb.h -- C ABI of the host-side task-batching scheduler in libtide.so.
 *
 * Continuous Task Batching (TideRL, arXiv 2608.10402, Section 4) schedules whole
 * multi-turn tasks, not requests: each rollout rank is a token budget pool; a new task
 * is admitted when the rank's headroom holds its group's probed first-turn footprint
 * (Section 4.1); Algorithm 1 pauses the least-priority active task while a rank is over
 * budget and, while it is under budget, resumes the highest-priority paused task that
 * fits before admitting new ones; the priority P(t) = w1 I_eval + w2 G_completion +
 * w3 I_active + w4 L_context orders evaluation tasks, then GRPO group completion, then
 * executing tasks, then long contexts (Section 4.2 and its preemption taxonomy table;
 * the weights are read lexicographically); paused tasks resume on the rank that holds
 * their cached pages, and a group's trajectories go to one rank (worker affinity).
 *
 * The scheduler drives an engine model round by round.  A round is one engine
 * iteration: environment answers arrive, the policy schedules, then every selected
 * task runs one op on its rank's paged KV pool:
 *   extend  attention of positions [start, start + count) over the task's context,
 *           where start = the tokens whose K/V are still in its pages (a resume hit)
 *           and count = the rest of its context plus its new input (prompt or
 *           observation) -- tide_kv_append + tide_extend_attn; start = 0 is a full
 *           re-prefill;
 *   decode  one token at position start (count = 1) -- tide_kv_append +
 *           tide_decode_attn with kv_len = start + 1.
 * The scheduler chooses physical pages: a rank's pool is a FIFO free list plus an LRU
 * list of cached pages whose content is still valid (a paused task's, or with the
 * request policy a finished request's).  A cached page taken for reuse invalidates the
 * owner's later pages too, since a prefix hit needs every earlier page; a released task
 * puts its last page first in line, so its longest prefix survives longest.
 *
 * Two policies share the engine model:
 *   TIDE_CTB_POLICY_CTB      Algorithm 1 as above;
 *   TIDE_CTB_POLICY_REQUEST  request-level continuous batching with prefix caching and a
 *                            fixed task concurrency (the fixed-concurrency baseline of
 *                            Section 6.5): each turn is a request, first-come first-served;
 *                            the newest running request is preempted when pages run out,
 *                            and nothing waiting is admitted in a round that preempted.
 *
 * Everything here runs on the host and touches no GPU memory.  Pointers returned in
 * tide_ctb_round stay valid until the next tide_ctb_step or tide_ctb_destroy on the
 * same scheduler.  A scheduler object must not be used by two threads at once.
 * Return values are the tide_status codes of tide.h.
 */
#ifndef TIDE_CTB_H_
#define TIDE_CTB_H_

#include <stdint.h>

#include "tide.h"

#ifdef __cplusplus
extern "C" {
#endif

enum {
  TIDE_CTB_POLICY_CTB = 0,
  TIDE_CTB_POLICY_REQUEST = 1
};

enum {
  TIDE_CTB_OP_EXTEND = 0,
  TIDE_CTB_OP_DECODE = 1
};

enum {
  TIDE_CTB_EV_ADMIT = 0,   /* CTB: task admitted; request policy: task started */
  TIDE_CTB_EV_PAUSE = 1,   /* CTB: task paused; request policy: request preempted */
  TIDE_CTB_EV_RESUME = 2,  /* CTB: task resumed; request policy: request admitted to run */
  TIDE_CTB_EV_FINISH = 3   /* the task finished its last turn */
};

typedef struct tide_ctb_config {
  int32_t policy;          /* TIDE_CTB_POLICY_* */
  int32_t num_ranks;       /* >= 1 rollout ranks, each with its own pool */
  int32_t pages_per_rank;  /* >= 1 pages of 16 tokens per rank */
  int32_t budget_tokens;   /* CTB token budget per rank, 1 .. pages_per_rank * 16 */
  int32_t max_running;     /* >= 1 tasks that run an op per rank and round */
  int32_t max_in_flight;   /* request policy: tasks started and not finished, >= 1 */
  int32_t env_capacity;    /* CTB: admitted, unfinished tasks over all ranks; 0 = no limit */
  int32_t max_rounds;      /* tide_ctb_step returns TIDE_ERR_CAPACITY past this round */
} tide_ctb_config;

typedef struct tide_ctb_op {
  int32_t rank;
  int32_t kind;            /* TIDE_CTB_OP_* */
  int32_t task;
  int32_t start;           /* extend: retained prefix P; decode: position of the token */
  int32_t count;           /* extend: E; decode: 1 */
  int32_t num_pages;       /* the task's pages after the op: ceil((start + count) / 16) */
  int64_t page_offset;     /* its page ids: pages[page_offset .. page_offset + num_pages) */
} tide_ctb_op;

typedef struct tide_ctb_event {
  int32_t kind;            /* TIDE_CTB_EV_* */
  int32_t task;
  int32_t rank;
  int32_t reserved;
} tide_ctb_event;

typedef struct tide_ctb_round {
  int32_t round;           /* index of the round just run */
  int32_t done;            /* 1 once every task has finished */
  int32_t num_ops;
  int32_t num_events;
  int64_t num_pages;
  const tide_ctb_op* ops;          /* in execution order */
  const int32_t* pages;            /* page ids referenced by ops */
  const tide_ctb_event* events;    /* in the order they happened */
} tide_ctb_round;

typedef struct tide_ctb_stats {
  int64_t rounds;
  int64_t extend_ops;
  int64_t decode_ops;
  int64_t hit_tokens;      /* sum of extend starts: positions whose K/V were reused */
  int64_t queried_tokens;  /* sum of extend start + count: the prefix-cache hit rate is
                              hit_tokens / queried_tokens */
  int64_t extend_tokens;   /* sum of extend counts: rows prefilled */
  int64_t input_tokens;    /* prompt + observation tokens of the trace (the minimum) */
  int64_t pauses;
  int64_t resumes;
  int64_t admits;
} tide_ctb_stats;

/* Creates a scheduler for a trace of num_tasks trajectories in arrival order.
 *   group[t], is_eval[t]          GRPO group (0 .. num_groups-1) and evaluation flag
 *   group_size[g]                 trajectories in group g (for the completion ratio)
 *   turn_start[num_tasks + 1]     turns of task t are turn_start[t] .. turn_start[t+1]-1
 *   new_tokens, gen_tokens, env_rounds [turn_start[num_tasks]]
 *                                 per turn: input tokens appended first (turn 0: the
 *                                 prompt, >= 1), tokens generated (>= 1), and rounds the
 *                                 environment takes after the turn (>= 1; unused after
 *                                 the last turn)
 * All arrays are host memory and are copied.  Trajectories of one group must share the
 * prompt length, and with the CTB policy every task's full context must fit the budget
 * (else it could never run): TIDE_ERR_INVALID_ARG otherwise.  *sim_out receives the
 * scheduler, to be released with tide_ctb_destroy.  TIDE_ERR_CAPACITY if out of host
 * memory. */
TIDE_API int tide_ctb_create(const tide_ctb_config* cfg, int32_t num_tasks, const int32_t* group,
                    const int32_t* is_eval, int32_t num_groups, const int32_t* group_size,
                    const int32_t* turn_start, const int32_t* new_tokens,
                    const int32_t* gen_tokens, const int32_t* env_rounds, void** sim_out);

/* Runs one round and describes it in *out.  Calling it after the last task finished
 * returns TIDE_OK with an empty round and done = 1. */
TIDE_API int tide_ctb_step(void* sim, tide_ctb_round* out);

/* Totals since creation. */
TIDE_API int tide_ctb_get_stats(const void* sim, tide_ctb_stats* out);

/* Releases the scheduler (NULL is accepted). */
TIDE_API int tide_ctb_destroy(void* sim);

#ifdef __cplusplus
}
#endif

#endif /* TIDE_CTB_H_ */
