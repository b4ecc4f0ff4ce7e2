"""Pins of the scheduling oracle (oracle/ctb.py), CPU only.

Each pin ties the oracle to something other than its own code:
  * the preemption taxonomy table of Section 4.2 (eval > group completion > executing >
    context length), checked one term at a time on hand-built states;
  * Algorithm 1's order (resume paused tasks before admitting new ones; admission by the
    probed footprint of Section 4.1);
  * prefix-cache semantics of the pool (the last page goes first; losing page i loses
    every later page);
  * closed-form timelines when nothing contends for memory (both policies);
  * a page-content replay: every op's retained prefix must still hold the task's own K/V,
    which is what makes resuming equal to recomputing (Sections 2.2, 5.2).
"""
import random

import numpy as np
import pytest

from oracle import ctb as C
import workloads.traces as T


def _sim(tasks, group_size=None, **cfg):
    gs = group_size or [sum(1 for g, _, _ in tasks if g == i)
                        for i in range(max(g for g, _, _ in tasks) + 1)]
    return C.Sim(C.Config(**cfg), tasks, gs)


def _set(t, ctx, state="active", rank=0, pending=0, to_gen=0, env_done=-1):
    t.state, t.rank, t.ctx, t.kv_valid = state, rank, ctx, ctx
    t.pending_new, t.to_gen, t.env_done = pending, to_gen, env_done


def _hold(sim, t):
    pool = sim.pools[t.rank]
    while len(t.pages) < C.pages(t.ctx):
        pool.alloc(t, sim.tasks)
    if t.state == "paused":
        pool.release(t)


def _evicted(sim):
    return [e[2] for e in sim.events if e[1] == C.EV_PAUSE]


# ------------------------------------------------------------------ taxonomy, term by term
def _two_active(a_kw, b_kw, a_group=0, b_group=1, a_eval=0, b_eval=0, done=(0, 0), sizes=(2, 2)):
    """Two active tasks on one rank whose footprints together exceed the budget by one
    page, so Algorithm 1 must pause exactly one of them."""
    tasks = [(a_group, a_eval, [(64, 4, 5)] * 2), (b_group, b_eval, [(64, 4, 5)] * 2),
             (a_group, 0, [(64, 1, 1)]), (b_group, 0, [(64, 1, 1)])]
    sim = C.Sim(C.Config(pages_per_rank=64), tasks, list(sizes))
    a, b = sim.tasks[0], sim.tasks[1]
    _set(a, **a_kw)
    _set(b, **b_kw)
    for t in (a, b):
        _hold(sim, t)
    sim.tasks[2].state = sim.tasks[3].state = "done"
    sim.group_done = list(done)
    sim.new_queue.clear()
    sim.cfg.budget_tokens = sim.footprint(a) + sim.footprint(b) - C.PAGE
    sim.schedule_ctb()
    return _evicted(sim)


def test_eval_task_is_kept_over_everything_else():
    # task 1 is an eval task waiting on its environment with a short context; task 0 is a
    # training task that is executing, has a longer context and a half-finished group
    ev = _two_active(dict(ctx=400, to_gen=3), dict(ctx=32, env_done=9), b_eval=1,
                     done=(1, 0))
    assert ev == [0]


def test_group_completion_outranks_execution_state_and_length():
    ev = _two_active(dict(ctx=400, to_gen=3), dict(ctx=32, env_done=9), done=(0, 1))
    assert ev == [0]


def test_executing_task_is_kept_over_a_waiting_one():
    ev = _two_active(dict(ctx=400, env_done=9), dict(ctx=32, to_gen=2))
    assert ev == [0]


def test_longer_context_is_kept():
    ev = _two_active(dict(ctx=48, env_done=9), dict(ctx=400, env_done=9))
    assert ev == [0]


def test_group_completion_is_a_ratio():
    # 1 of 2 finished (0.5) outranks 1 of 4 finished (0.25)
    ev = _two_active(dict(ctx=32, env_done=9), dict(ctx=400, env_done=9), done=(1, 1),
                     sizes=(2, 4))
    assert ev == [1]


# ------------------------------------------------------------------ Algorithm 1 order
def test_resume_before_admit_and_fit_rule():
    # budget 8 pages; task 3 active (2 pages, waiting on its environment); task 0 paused
    # with 3 pages, task 1 paused with 7 (no room next to task 3), task 2 new (probe 2
    # pages).  Task 1 has the higher priority (longer context) but does not fit, so task 0
    # is resumed; with task 1 still not fitting, the new task is admitted (reading: the
    # resume branch picks among the paused tasks that fit).
    tasks = [(0, 0, [(40, 2, 3), (8, 1, 1)]), (1, 0, [(100, 2, 3), (8, 1, 1)]),
             (2, 0, [(16, 1, 1)]), (3, 0, [(32, 1, 3), (8, 1, 1)])]
    sim = _sim(tasks, pages_per_rank=16, budget_tokens=8 * 16)
    t0, t1, t3 = sim.tasks[0], sim.tasks[1], sim.tasks[3]
    _set(t3, 32, env_done=5)
    _set(t0, 40, state="paused", env_done=7)
    _set(t1, 100, state="paused", env_done=7)
    for t in (t3, t0, t1):
        _hold(sim, t)
    for i in (0, 1, 3):
        sim.new_queue.remove(i)
    sim.schedule_ctb()
    assert [(e[1], e[2]) for e in sim.events] == [(C.EV_RESUME, 0), (C.EV_ADMIT, 2)]
    # with room for both paused tasks, both are resumed (highest priority first) before
    # the new task is admitted
    tasks = tasks[:3]
    sim2 = _sim(tasks, pages_per_rank=12)
    for t, ctx in ((sim2.tasks[0], 40), (sim2.tasks[1], 100)):
        _set(t, ctx, state="paused", env_done=7)
        _hold(sim2, t)
    sim2.new_queue.remove(0)
    sim2.new_queue.remove(1)
    sim2.schedule_ctb()
    assert [(e[1], e[2]) for e in sim2.events] == [(C.EV_RESUME, 1), (C.EV_RESUME, 0),
                                                  (C.EV_ADMIT, 2)]


def test_admission_uses_the_group_probe():
    # group 0's first trajectory generates 100 tokens in its first turn: probe =
    # pages(20 + 100 + 1) = 8 pages.  Task 2 holds 3 pages of the rank.  With a budget of
    # 10 pages the headroom (7) cannot take the group's second trajectory, although its
    # prompt needs only 2 pages; with 11 pages it can.
    tasks = [(0, 0, [(20, 100, 1)]), (0, 0, [(20, 1, 1)]), (1, 0, [(48, 1, 2), (1, 1, 1)])]
    for budget, admitted in ((10, []), (11, [(C.EV_ADMIT, 1)])):
        sim = _sim(tasks, pages_per_rank=16, budget_tokens=budget * 16)
        sim.new_queue.clear()
        sim.new_queue.append(1)
        sim.tasks[0].state = "done"
        _set(sim.tasks[2], 48, env_done=4)
        _hold(sim, sim.tasks[2])
        sim.schedule_ctb()
        assert [(e[1], e[2]) for e in sim.events] == admitted


def test_group_affinity_across_ranks():
    # two ranks with room for one task each: group 0 starts on rank 0 and group 1 on
    # rank 1; group 0's second trajectory waits for rank 0 even when rank 1 frees first
    tasks = [(0, 0, [(16, 5, 1)]), (1, 0, [(16, 1, 1)]), (0, 0, [(16, 1, 1)])]
    sim = _sim(tasks, num_ranks=2, pages_per_rank=2).run()
    placed = {e[2]: e[3] for e in sim.events if e[1] == C.EV_ADMIT}
    assert placed == {0: 0, 1: 1, 2: 0}
    admit = {e[2]: e[0] for e in sim.events if e[1] == C.EV_ADMIT}
    finish = {e[2]: e[0] for e in sim.events if e[1] == C.EV_FINISH}
    assert finish[1] < finish[0] and admit[2] == finish[0] + 1


# ------------------------------------------------------------------ pool semantics
def test_pool_releases_last_page_first_and_loses_suffixes():
    tasks = [(0, 0, [(64, 1, 1)]), (1, 0, [(64, 1, 1)])]
    sim = _sim(tasks, pages_per_rank=6)
    a, b = sim.tasks
    _set(a, 64, state="paused")
    _hold(sim, a)                 # pages 0..3, cached; LRU = [3, 2, 1, 0]
    _set(b, 0)
    assert list(sim.pools[0].free) == [4, 5]
    for _ in range(3):            # two free pages, then a's last page
        sim.pools[0].alloc(b, sim.tasks)
    assert b.pages == [4, 5, 3] and a.pages == [0, 1, 2] and a.kv_valid == 48
    sim.pools[0].release(b)       # LRU = [2, 1, 0, 3, 5, 4]
    c = sim.tasks[1]
    assert sim.pools[0].lru == [2, 1, 0, 3, 5, 4]
    # taking a's page at index 1 (second from the head after page 2) loses index 2 too
    sim.pools[0].lru = [1, 2, 0, 3, 5, 4]
    page = sim.pools[0].alloc(c, sim.tasks)
    assert page == 1 and a.pages == [0] and a.kv_valid == 16
    assert list(sim.pools[0].free) == [2] and 2 not in sim.pools[0].lru


# ------------------------------------------------------------------ closed forms
def _random_tasks(rng, n, groups, turns=(1, 4), new=(1, 90), gen=(1, 12), env=(1, 9)):
    out = []
    prompts = [rng.randint(*new) for _ in range(groups)]
    for i in range(n):
        g = i % groups
        k = rng.randint(*turns)
        ts = [(prompts[g] if j == 0 else rng.randint(*new), rng.randint(*gen),
               rng.randint(*env)) for j in range(k)]
        out.append((g, int(g % 3 == 0), ts))
    return out


@pytest.mark.parametrize("policy", [C.POLICY_CTB, C.POLICY_REQUEST])
def test_uncontended_timeline_is_closed_form(policy):
    rng = random.Random(5)
    tasks = _random_tasks(rng, 12, 4)
    sim = _sim(tasks, policy=policy, pages_per_rank=4096, max_running=64).run()
    # every task starts in round 0; turn k extends once, decodes gen_k tokens, then waits
    # env_k rounds: it finishes in round sum(gen) + sum(env of all but the last turn)
    finish = {e[2]: e[0] for e in sim.events if e[1] == C.EV_FINISH}
    for i, (_, _, ts) in enumerate(tasks):
        assert finish[i] == sum(a for _, a, _ in ts) + sum(e for _, _, e in ts[:-1])
    assert sim.stats["pauses"] == 0
    # nothing is ever recomputed: extends are exactly the input tokens, and every later
    # turn hits its whole history
    assert sim.stats["extend_tokens"] == sum(n for _, _, ts in tasks for n, _, _ in ts)
    hits = 0
    for _, _, ts in tasks:
        ctx = 0
        for k, (n, a, _) in enumerate(ts):
            hits += ctx
            ctx += n + a
    assert sim.stats["hit_tokens"] == hits


def test_policies_agree_without_contention():
    rng = random.Random(9)
    tasks = _random_tasks(rng, 10, 3)
    a = _sim(tasks, policy=C.POLICY_CTB, pages_per_rank=4096).run()
    b = _sim(tasks, policy=C.POLICY_REQUEST, pages_per_rank=4096).run()
    # the same work in the same rounds (the order inside a round and the page ids differ)
    assert sorted(o[:6] for o in a.ops) == sorted(o[:6] for o in b.ops)


def test_one_task_in_flight_runs_tasks_back_to_back():
    rng = random.Random(3)
    tasks = _random_tasks(rng, 5, 5)
    sim = _sim(tasks, policy=C.POLICY_REQUEST, pages_per_rank=4096, max_in_flight=1).run()
    finish = {e[2]: e[0] for e in sim.events if e[1] == C.EV_FINISH}
    start = 0
    for i, (_, _, ts) in enumerate(tasks):
        dur = sum(a for _, a, _ in ts) + sum(e for _, _, e in ts[:-1])
        assert finish[i] == start + dur
        start = finish[i] + 1


# ------------------------------------------------------------------ whole-run invariants
def _replay_contents(sim, tasks):
    """Replays the op list against page contents: page p holds (task, position) per slot.
    Every op must find its own rows in front of its start, and the sequence of each task
    must be built exactly once in order.  Returns the number of positions checked."""
    content = {}
    ctx = [0] * len(tasks)
    checked = 0
    # the ops of one round run as batched kernel calls: no two of them may share a page
    by_round = {}
    for rnd, r, kind, t, start, count, pg in sim.ops:
        for p in pg:
            assert by_round.setdefault((rnd, r, p), t) == t, (rnd, r, p)
    for rnd, r, kind, t, start, count, pg in sim.ops:
        for pos in range(start):
            assert content.get((r, pg[pos // 16], pos % 16)) == (t, pos), (rnd, t, pos)
            checked += 1
        for pos in range(start, start + count):
            content[(r, pg[pos // 16], pos % 16)] = (t, pos)
        ctx[t] = max(ctx[t], start + count)
        if kind == C.OP_DECODE:
            assert count == 1
    for t, (_, _, ts) in enumerate(tasks):
        assert ctx[t] == sum(n + a for n, a, _ in ts)
    return checked


@pytest.mark.parametrize("policy,ranks,pages,seed", [
    (C.POLICY_CTB, 1, 40, 1), (C.POLICY_CTB, 2, 30, 2), (C.POLICY_CTB, 3, 24, 3),
    (C.POLICY_REQUEST, 1, 24, 4), (C.POLICY_REQUEST, 2, 20, 5)])
def test_contended_runs_keep_every_invariant(policy, ranks, pages, seed):
    rng = random.Random(seed)
    tasks = _random_tasks(rng, 24, 6)
    sim = _sim(tasks, policy=policy, num_ranks=ranks, pages_per_rank=pages, max_running=6,
               max_in_flight=10)
    def check(s):
        held = {}
        for t in s.tasks:
            if t.state == "active":
                for p in t.pages:
                    assert (t.rank, p) not in held
                    held[(t.rank, p)] = t.id
                if policy == C.POLICY_CTB:
                    assert len(t.pages) * 16 <= s.footprint(t)
        if policy == C.POLICY_CTB:
            # after Algorithm 1 every rank is within its budget
            for r in range(ranks):
                assert s.usage(r) <= s.cfg.budget_tokens
        for r in range(ranks):
            pool = s.pools[r]
            n_held = sum(len(t.pages) for t in s.tasks if t.state == "active" and t.rank == r)
            assert n_held + len(pool.free) + len(pool.lru) == pages

    while not sim.done():
        sim.step(check)
        assert sim.round < 20000
    # the pools are small enough to force pausing and recomputation
    assert sim.stats["pauses"] > 0
    assert sim.stats["extend_tokens"] > sim.stats["input_tokens"]
    assert _replay_contents(sim, tasks) > 0
    decoded = sum(1 for o in sim.ops if o[2] == C.OP_DECODE)
    assert decoded == sum(a for _, _, ts in tasks for _, a, _ in ts)


def test_trace_generator_shapes():
    tr = T.make_trace("webshop_step")
    assert tr.num_tasks == 32 * 8 + 200 * 4 and int(tr.is_eval.sum()) == 800
    nt = np.diff(tr.turn_start)
    assert nt.min() >= 3 and nt.max() <= 13 and 7 < nt.mean() < 9
    assert 2400 <= tr.final_lens.mean() <= 3400
    # trajectories of one group share the prompt
    for g in range(len(tr.group_size)):
        firsts = tr.new_tokens[tr.turn_start[:-1][tr.group == g]]
        assert (firsts == firsts[0]).all() and len(firsts) == tr.group_size[g]


def test_reusing_a_page_inside_its_round_is_caught(monkeypatch):
    """Planted mistake: pages an op gives up become reusable within the same round.  The
    batched execution of a round would then let one op overwrite K/V another op of the
    round reads; the page-content replay must reject such schedules."""
    def drop_now(self, task):
        for p in task.pages:
            del self.owner[p]
            self.free.append(p)
        task.pages = []
        task.kv_valid = 0
    release = C.Pool.release
    monkeypatch.setattr(C.Pool, "drop", drop_now)
    monkeypatch.setattr(C.Pool, "release", lambda self, task, later=False: release(self, task))
    rng = random.Random(1)
    tasks = _random_tasks(rng, 24, 6)
    sim = _sim(tasks, policy=C.POLICY_CTB, pages_per_rank=40, max_running=6).run()
    with pytest.raises(AssertionError):
        _replay_contents(sim, tasks)
