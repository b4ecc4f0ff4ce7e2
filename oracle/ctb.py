"""Continuous Task Batching scheduler, plain and slow (TEST INFRASTRUCTURE ONLY).

This is the oracle for the native scheduler in libtide.so.  Only tests/ and the
benchmark's CPU baseline use it; nothing in the product path imports it.  It recomputes
every quantity from scratch each time it is needed (usage, priorities, argmin/argmax over
sets), so that each step can be checked against the paper by eye.

What it follows (Section 4):
  * token-aware admission (4.1): each rank is a token budget pool; a new task is admitted
    only when the rank's headroom holds its group's probed first-turn footprint;
    footprints are refreshed at every round;
  * Algorithm 1 (Semantic-Aware CTB Scheduling): per rank, while usage exceeds the budget,
    pause the active task of least priority; while usage is below it, resume the
    highest-priority paused task that fits, else admit a new task, else stop;
  * the priority P(t) = w1 I_eval + w2 G_completion + w3 I_active + w4 L_context with the
    weights read lexicographically (the preemption taxonomy table orders the four terms
    strictly: task type > group completion > execution state > context length);
  * worker affinity (4.2): a paused task resumes on the rank that holds its cached pages,
    and a group's trajectories are admitted to the rank its first trajectory went to.

The baseline is request-level continuous batching with prefix caching and a fixed task
concurrency (the "F9/F10" settings of Section 6.5): every turn is a request; a finished
request's pages stay cached in LRU order until reused; FCFS admission; the newest running
request is preempted when pages run out.

Engine model shared by both policies (one round = one engine iteration):
  1. environment completions: a task whose environment finishes this round gets its next
     turn's input tokens (pending) and generation count;
  2. scheduling (the policy);
  3. execution: a selected task either extends (P = tokens whose K/V are still in its
     pages, E = the rest of its context plus its pending input) or decodes one token;
  4. a task that has generated its turn's tokens waits for its environment, or finishes.
Pages are 16 tokens.  A rank's pool is a FIFO free list plus an LRU list of cached pages
(content still valid).  Taking a cached page from the LRU head invalidates it and every
later page of the same task, since a prefix hit needs all earlier pages.

Readings where the paper is silent are listed in the docstrings of the functions that
take them.  Parity unpinned: none -- see tests/test_ctb_oracle.py for the pins.
"""
from __future__ import annotations

from collections import deque
from fractions import Fraction

PAGE = 16
POLICY_CTB = 0
POLICY_REQUEST = 1

OP_EXTEND = 0
OP_DECODE = 1

EV_ADMIT = 0    # CTB: new task admitted / request policy: task started
EV_PAUSE = 1    # CTB: paused (preempted) / request policy: request preempted
EV_RESUME = 2   # CTB: resumed / request policy: request admitted to run
EV_FINISH = 3   # task finished its last turn


def pages(n: int) -> int:
    return (n + PAGE - 1) // PAGE


class Config:
    def __init__(self, policy=POLICY_CTB, num_ranks=1, pages_per_rank=1024, budget_tokens=None,
                 max_running=256, max_in_flight=1024, env_capacity=0, max_rounds=1_000_000):
        self.policy = policy
        self.num_ranks = num_ranks
        self.pages_per_rank = pages_per_rank
        self.budget_tokens = pages_per_rank * PAGE if budget_tokens is None else budget_tokens
        self.max_running = max_running
        self.max_in_flight = max_in_flight
        self.env_capacity = env_capacity
        self.max_rounds = max_rounds


class Task:
    def __init__(self, tid, group, is_eval, turns):
        self.id = tid
        self.group = group
        self.is_eval = is_eval
        self.turns = turns          # [(new, gen, env)]
        self.state = "new"          # new | active | paused | done   (request policy: see below)
        self.rank = -1
        self.turn = 0
        self.ctx = 0                # tokens in the sequence so far
        self.kv_valid = 0           # leading tokens whose K/V are in the task's pages
        self.pending_new = 0        # input tokens of the current turn not yet appended
        self.to_gen = 0             # tokens still to generate in the current turn
        self.env_done = -1          # round at which the environment answers (-1: not waiting)
        self.pages = []             # page ids in logical order (held or cached)


class Pool:
    """One rank's pages: FIFO free list, LRU list of cached pages, owner of every page."""

    def __init__(self, n):
        self.free = deque(range(n))
        self.lru = []               # head (index 0) = least recently released
        self.owner = {}             # page -> (task, logical index), for held and cached pages
        self.later_free = []        # freed by this round's ops: reusable from the next round
        self.later_lru = []         # released by this round's ops: evictable from the next round

    def alloc(self, task, tasks):
        if self.free:
            page = self.free.popleft()
        else:
            page = self.lru.pop(0)
            victim, idx = self.owner.pop(page)
            v = tasks[victim]
            # the victim keeps only the pages before idx; later ones are useless now
            for j in range(idx + 1, len(v.pages)):
                p = v.pages[j]
                self.lru.remove(p)
                del self.owner[p]
                self.free.append(p)
            v.pages = v.pages[:idx]
            v.kv_valid = min(v.kv_valid, idx * PAGE)
        self.owner[page] = (task.id, len(task.pages))
        task.pages.append(page)
        return page

    def release(self, task, later=False):
        """Held pages become cached; the last page is released first, so it is taken
        first and the longest prefix survives.  `later`: released by an op of the round
        being executed, so they join the LRU list when the round ends."""
        for p in reversed(task.pages):
            (self.later_lru if later else self.lru).append(p)

    def reclaim(self, task):
        """A task's cached pages become held again."""
        for p in task.pages:
            self.lru.remove(p)

    def drop(self, task):
        """A finished task's pages go back to the free list when the round ends.  Reading:
        a round is one batched engine iteration, so no op of the round may rewrite a page
        another op of the same round reads; pages an op gives up become reusable in the
        next round (as an engine frees a finished request's blocks after its step)."""
        for p in task.pages:
            del self.owner[p]
            self.later_free.append(p)
        task.pages = []
        task.kv_valid = 0

    def end_round(self):
        self.free.extend(self.later_free)
        self.lru.extend(self.later_lru)
        self.later_free = []
        self.later_lru = []


class Sim:
    def __init__(self, cfg: Config, trace_tasks, group_size):
        """trace_tasks: [(group, is_eval, [(new, gen, env), ...])] in arrival order."""
        self.cfg = cfg
        self.tasks = [Task(i, g, e, turns) for i, (g, e, turns) in enumerate(trace_tasks)]
        self.group_size = list(group_size)
        self.group_done = [0] * len(self.group_size)
        self.group_rank = [-1] * len(self.group_size)
        self.pools = [Pool(cfg.pages_per_rank) for _ in range(cfg.num_ranks)]
        self.round = 0
        self.events = []            # (round, kind, task, rank)
        self.ops = []               # (round, rank, kind, task, P, E or pos, tuple(pages))
        self.new_queue = deque(range(len(self.tasks)))
        # request policy state
        self.waiting = [deque() for _ in range(cfg.num_ranks)]
        self.running = [[] for _ in range(cfg.num_ranks)]
        self.in_flight = 0
        self.stats = {"rounds": 0, "extend_ops": 0, "decode_ops": 0, "hit_tokens": 0,
                      "queried_tokens": 0, "extend_tokens": 0, "input_tokens": 0,
                      "pauses": 0, "resumes": 0, "admits": 0}
        for t in self.tasks:
            self.stats["input_tokens"] += sum(n for n, _, _ in t.turns)
        self._check_fits()

    # ---------------------------------------------------------------- helpers
    def _check_fits(self):
        """Inputs the model needs: at least one turn, a prompt, at least one generated
        token per turn, environments that take at least one round, one prompt length per
        group (the probe stands for the whole group), and a budget that one task alone
        never outgrows (else it could never run)."""
        cfg = self.cfg
        if cfg.num_ranks < 1 or cfg.pages_per_rank < 1 or cfg.max_running < 1:
            raise ValueError("bad configuration")
        if cfg.budget_tokens > cfg.pages_per_rank * PAGE:
            raise ValueError("budget exceeds the pool")
        prompt = {}
        for t in self.tasks:
            if not t.turns or t.turns[0][0] < 1:
                raise ValueError("task %d: no prompt" % t.id)
            if any(a < 1 or e < 1 or n < 0 for n, a, e in t.turns):
                raise ValueError("task %d: bad turn" % t.id)
            if prompt.setdefault(t.group, t.turns[0][0]) != t.turns[0][0]:
                raise ValueError("group %d: prompts differ" % t.group)
            need = PAGE * pages(sum(n + a for n, a, _ in t.turns) + 1)
            if cfg.policy == POLICY_CTB and need > cfg.budget_tokens:
                raise ValueError("task %d needs %d tokens, the budget is %d"
                                 % (t.id, need, cfg.budget_tokens))
            if need > cfg.pages_per_rank * PAGE:
                raise ValueError("task %d needs %d tokens, a rank holds %d"
                                 % (t.id, need, cfg.pages_per_rank * PAGE))

    def done(self):
        return all(t.state == "done" for t in self.tasks)

    def footprint(self, t):
        """Tokens the task may hold by the end of this round (page granular): its context,
        its pending input, and one decoded token if it still generates."""
        return PAGE * pages(t.ctx + t.pending_new + (1 if t.to_gen > 0 else 0))

    def usage(self, r):
        return sum(self.footprint(t) for t in self.tasks if t.state == "active" and t.rank == r)

    def probe(self, t):
        """Probed footprint of a new task: the first-turn usage (prompt + first generation)
        of its group's first trajectory (Section 4.1).  Reading: the probe is the group's
        first trajectory in arrival order, and its cost is not simulated."""
        first = next(x for x in self.tasks if x.group == t.group)
        n, a, _ = first.turns[0]
        return PAGE * pages(n + a + 1)

    def executing(self, t):
        """I_active: the task has work now (it is not waiting for its environment)."""
        return 1 if (t.pending_new > 0 or t.to_gen > 0) else 0

    def priority(self, t):
        """P(t) with lexicographic weights, then arrival order: a larger key is kept."""
        g = Fraction(self.group_done[t.group], self.group_size[t.group])
        return (t.is_eval, g, self.executing(t), t.ctx, -t.id)

    def event(self, kind, t, r):
        self.events.append((self.round, kind, t.id, r))

    # ---------------------------------------------------------------- round steps
    def env_completions(self):
        for t in self.tasks:
            if t.env_done == self.round:
                t.env_done = -1
                t.turn += 1
                n, a, _ = t.turns[t.turn]
                t.pending_new = n
                t.to_gen = a
                if self.cfg.policy == POLICY_REQUEST:
                    self.waiting[t.rank].append(t.id)

    def schedule_ctb(self):
        """Algorithm 1, one pass over the ranks."""
        B = self.cfg.budget_tokens
        for r in range(self.cfg.num_ranks):
            pool = self.pools[r]
            while self.usage(r) > B:
                act = [t for t in self.tasks if t.state == "active" and t.rank == r]
                t = min(act, key=self.priority)
                t.state = "paused"
                pool.release(t)
                self.stats["pauses"] += 1
                self.event(EV_PAUSE, t, r)
            while self.usage(r) < B:
                u = self.usage(r)
                fit = [t for t in self.tasks if t.state == "paused" and t.rank == r
                       and u + self.footprint(t) <= B]
                if fit:
                    # reading: "fits" selects among the paused tasks that fit
                    t = max(fit, key=self.priority)
                    t.state = "active"
                    pool.reclaim(t)
                    self.stats["resumes"] += 1
                    self.event(EV_RESUME, t, r)
                    continue
                t = self._next_new(r)
                if t is not None and self._admissible(t, r, u):
                    self.new_queue.remove(t.id)
                    t.state = "active"
                    t.rank = r
                    if self.group_rank[t.group] < 0:
                        self.group_rank[t.group] = r
                    n, a, _ = t.turns[0]
                    t.pending_new, t.to_gen = n, a
                    self.stats["admits"] += 1
                    self.event(EV_ADMIT, t, r)
                    continue
                break

    def _next_new(self, r):
        """The first new task (arrival order) that may go to rank r under group affinity."""
        for tid in self.new_queue:
            t = self.tasks[tid]
            if self.group_rank[t.group] in (-1, r):
                return t
        return None

    def _admissible(self, t, r, u):
        if u + self.probe(t) > self.cfg.budget_tokens:
            return False
        if self.cfg.env_capacity > 0:
            live = sum(1 for x in self.tasks if x.state in ("active", "paused"))
            if live >= self.cfg.env_capacity:
                return False
        return True

    def execute_ctb(self):
        for r in range(self.cfg.num_ranks):
            work = [t for t in self.tasks if t.state == "active" and t.rank == r
                    and (t.pending_new > 0 or t.to_gen > 0 or t.kv_valid < t.ctx)]
            work.sort(key=self.priority, reverse=True)
            for t in work[: self.cfg.max_running]:
                self.run_op(t, r)

    def run_op(self, t, r):
        pool = self.pools[r]
        if t.kv_valid < t.ctx or t.pending_new > 0:
            P = t.kv_valid
            E = t.ctx + t.pending_new - P
            while len(t.pages) < pages(P + E):
                pool.alloc(t, self.tasks)
            self.ops.append((self.round, r, OP_EXTEND, t.id, P, E, tuple(t.pages)))
            self.stats["extend_ops"] += 1
            self.stats["hit_tokens"] += P
            self.stats["queried_tokens"] += P + E
            self.stats["extend_tokens"] += E
            t.ctx += t.pending_new
            t.pending_new = 0
            t.kv_valid = t.ctx
        else:
            pos = t.ctx
            while len(t.pages) < pages(pos + 1):
                pool.alloc(t, self.tasks)
            self.ops.append((self.round, r, OP_DECODE, t.id, pos, 1, tuple(t.pages)))
            self.stats["decode_ops"] += 1
            t.ctx += 1
            t.kv_valid = t.ctx
            t.to_gen -= 1
            if t.to_gen == 0:
                self.end_turn(t, r)

    def end_turn(self, t, r):
        if t.turn == len(t.turns) - 1:
            self.pools[r].drop(t)
            t.state = "done"
            self.group_done[t.group] += 1
            self.event(EV_FINISH, t, r)
            if self.cfg.policy == POLICY_REQUEST:
                self.running[r].remove(t.id)
                self.in_flight -= 1
        else:
            t.env_done = self.round + t.turns[t.turn][2]
            if self.cfg.policy == POLICY_REQUEST:
                # the turn's request is finished: its pages stay cached, nothing is held
                self.running[r].remove(t.id)
                self.pools[r].release(t, later=True)
                t.state = "paused"

    # ---------------------------------------------------------------- request policy
    def schedule_request(self):
        """Request-level batching.  Reading of the engine (vLLM-like, the Section 6.5 baseline):
        a fixed number of tasks in flight; a new task goes to the rank with the fewest tasks
        in flight; per rank, running requests first get the page their next token needs,
        preempting the newest running request (to the front of the queue) when pages run
        out; then waiting requests are admitted first-come first-served while the batch has
        room and their pages fit."""
        while self.new_queue and self.in_flight < self.cfg.max_in_flight:
            t = self.tasks[self.new_queue.popleft()]
            counts = [sum(1 for x in self.tasks if x.rank == r and x.state != "done"
                          and x.state != "new") for r in range(self.cfg.num_ranks)]
            r = min(range(self.cfg.num_ranks), key=lambda i: (counts[i], i))
            t.rank = r
            t.state = "paused"       # not running, pages (none yet) evictable
            n, a, _ = t.turns[0]
            t.pending_new, t.to_gen = n, a
            self.in_flight += 1
            self.stats["admits"] += 1
            self.event(EV_ADMIT, t, r)
            self.waiting[r].append(t.id)
        for r in range(self.cfg.num_ranks):
            pool = self.pools[r]
            avail = len(pool.free) + len(pool.lru)
            need = 0
            preempted = False
            i = 0
            while i < len(self.running[r]):
                t = self.tasks[self.running[r][i]]
                want = self.op_pages(t) - len(t.pages)
                while need + want > avail:
                    preempted = True
                    v = self.tasks[self.running[r].pop()]
                    pool.release(v)
                    v.state = "paused"
                    avail += len(v.pages)
                    self.stats["pauses"] += 1
                    self.event(EV_PAUSE, v, r)
                    self.waiting[r].appendleft(v.id)
                    if v is t:
                        want = 0
                        break
                if t.state == "active":
                    need += want
                    i += 1
            # as in vLLM, nothing waiting is admitted in a round that preempted
            while (self.waiting[r] and not preempted
                   and len(self.running[r]) < self.cfg.max_running):
                t = self.tasks[self.waiting[r][0]]
                cached = len(t.pages)
                want = self.op_pages(t) - cached
                if need + want > avail - cached:
                    break
                self.waiting[r].popleft()
                pool.reclaim(t)
                avail -= cached
                need += want
                t.state = "active"
                self.running[r].append(t.id)
                self.stats["resumes"] += 1
                self.event(EV_RESUME, t, r)

    def op_pages(self, t):
        """Pages the task holds after this round's op (extend or one decoded token)."""
        if t.kv_valid < t.ctx or t.pending_new > 0:
            return pages(t.ctx + t.pending_new)
        return pages(t.ctx + 1)

    def execute_request(self):
        for r in range(self.cfg.num_ranks):
            for tid in list(self.running[r]):
                self.run_op(self.tasks[tid], r)

    # ---------------------------------------------------------------- driver
    def step(self, after_schedule=None):
        """One engine round.  Returns the ops issued in it.  `after_schedule(self)`, if
        given, runs between scheduling and execution (tests check invariants there)."""
        first = len(self.ops)
        self.env_completions()
        if self.cfg.policy == POLICY_CTB:
            self.schedule_ctb()
            if after_schedule:
                after_schedule(self)
            self.execute_ctb()
        else:
            self.schedule_request()
            if after_schedule:
                after_schedule(self)
            self.execute_request()
        for pool in self.pools:
            pool.end_round()
        self.round += 1
        self.stats["rounds"] = self.round
        return self.ops[first:]

    def run(self):
        while not self.done():
            if self.round >= self.cfg.max_rounds:
                raise RuntimeError("no progress after %d rounds" % self.round)
            self.step()
        return self


def trace_tasks(trace):
    """[(group, is_eval, [(new, gen, env), ...])] of a workloads.traces.Trace."""
    out = []
    for t in range(trace.num_tasks):
        a, b = int(trace.turn_start[t]), int(trace.turn_start[t + 1])
        turns = [(int(trace.new_tokens[k]), int(trace.gen_tokens[k]), int(trace.env_rounds[k]))
                 for k in range(a, b)]
        out.append((int(trace.group[t]), int(trace.is_eval[t]), turns))
    return out


def simulate(trace, cfg: Config) -> Sim:
    return Sim(cfg, trace_tasks(trace), trace.group_size).run()
