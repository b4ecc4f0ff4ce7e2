"""The native task-batching scheduler (libtide.so, include/tide_ctb.h) against the plain
oracle (oracle/ctb.py), CPU only.

Integer work, so the bar is exact: the same ops (round, rank, kind, task, start, count,
page ids), the same events in the same order, the same totals.  Small traces cover both
policies, one to three ranks, tight and loose pools, the engine batch limit, the
environment-capacity constraint and evaluation tasks; the WebShop-shaped step is compared
whole at the pool size the benchmark uses.
"""
import random

import numpy as np
import pytest

from oracle import ctb as C
import paper_2608_10402_amd.ctb as N
import workloads.traces as T


def _native_run(trace, **cfg):
    s = N.Scheduler.from_trace(trace, **cfg)
    ops, events = [], []
    for r in s.rounds():
        for i, o in enumerate(r.ops):
            ops.append((r.round, int(o["rank"]), int(o["kind"]), int(o["task"]), int(o["start"]),
                        int(o["count"]), tuple(int(p) for p in r.op_pages(i))))
        for e in r.events:
            events.append((r.round, int(e["kind"]), int(e["task"]), int(e["rank"])))
    st = s.stats()
    s.close()
    return ops, events, st


def _oracle_run(trace, **cfg):
    sim = C.simulate(trace, C.Config(**cfg))
    return sim.ops, sim.events, sim.stats


def _random_trace(seed, n, groups, turns=(1, 5), new=(1, 120), gen=(1, 14), env=(1, 12),
                  eval_frac=0.3):
    rng = random.Random(seed)
    prompts = [rng.randint(*new) for _ in range(groups)]
    evals = [int(rng.random() < eval_frac) for _ in range(groups)]
    tasks = []
    for i in range(n):
        g = rng.randrange(groups)
        k = rng.randint(*turns)
        ts = [(prompts[g] if j == 0 else rng.randint(*new), rng.randint(*gen), rng.randint(*env))
              for j in range(k)]
        tasks.append((g, ts))
    used = sorted({g for g, _ in tasks})
    remap = {g: i for i, g in enumerate(used)}
    tasks = [(remap[g], ts) for g, ts in tasks]
    is_eval = [evals[used[g]] for g, _ in tasks]
    return T.custom_trace(tasks, is_eval=is_eval, seed=seed)


CASES = [
    # (seed, tasks, groups, config)
    (1, 30, 8, dict(policy=0, pages_per_rank=48, max_running=8)),
    (2, 30, 8, dict(policy=0, pages_per_rank=40, budget_tokens=560, max_running=4)),
    (3, 40, 10, dict(policy=0, num_ranks=2, pages_per_rank=36, max_running=6)),
    (4, 40, 10, dict(policy=0, num_ranks=3, pages_per_rank=40, max_running=5, env_capacity=9)),
    (5, 30, 6, dict(policy=0, pages_per_rank=4096)),
    (6, 30, 8, dict(policy=1, pages_per_rank=48, max_running=8, max_in_flight=12)),
    (7, 30, 8, dict(policy=1, pages_per_rank=36, max_running=5, max_in_flight=30)),
    (8, 40, 10, dict(policy=1, num_ranks=2, pages_per_rank=36, max_running=6, max_in_flight=16)),
    (9, 40, 10, dict(policy=1, num_ranks=3, pages_per_rank=40, max_running=4, max_in_flight=7)),
    (10, 30, 6, dict(policy=1, pages_per_rank=4096, max_in_flight=1)),
]


@pytest.mark.parametrize("seed,n,groups,cfg", CASES, ids=[str(c[0]) for c in CASES])
def test_native_scheduler_matches_oracle(seed, n, groups, cfg):
    tr = _random_trace(seed, n, groups)
    o_ops, o_ev, o_st = _oracle_run(tr, **cfg)
    n_ops, n_ev, n_st = _native_run(tr, **cfg)
    assert n_ev == o_ev
    assert n_ops == o_ops
    assert n_st == o_st


def test_native_scheduler_matches_oracle_on_shrunk_webshop():
    tr = T.make_trace(T.TRACE_SPECS["webshop_step"].shrunk(6, 20, 4))
    for cfg in (dict(policy=0, pages_per_rank=1024, max_running=32),
                dict(policy=1, pages_per_rank=1024, max_running=32, max_in_flight=64)):
        o = _oracle_run(tr, **cfg)
        n = _native_run(tr, **cfg)
        assert n[1] == o[1] and n[0] == o[0] and n[2] == o[2]


def test_native_rejects_bad_traces():
    tr = _random_trace(1, 4, 2)
    with pytest.raises(N.TideError):   # budget above the pool
        N.Scheduler.from_trace(tr, pages_per_rank=4, budget_tokens=65)
    with pytest.raises(N.TideError):   # a task that can never fit
        N.Scheduler.from_trace(tr, pages_per_rank=2)
    bad = T.custom_trace([(0, [(10, 1, 1)]), (0, [(11, 1, 1)])])
    with pytest.raises(N.TideError):   # one group, two prompt lengths
        N.Scheduler.from_trace(bad)
    bad = T.custom_trace([(0, [(10, 0, 1)])])
    with pytest.raises(N.TideError):   # a turn that generates nothing
        N.Scheduler.from_trace(bad)


def test_step_after_the_end_is_empty():
    tr = _random_trace(2, 3, 2)
    s = N.Scheduler.from_trace(tr, pages_per_rank=4096)
    rounds = list(s.rounds())
    assert rounds[-1].done
    extra = s.step()
    assert extra.done and extra.ops.size == 0 and extra.events.size == 0


def _digest_native(trace, **cfg):
    import hashlib
    h = hashlib.sha256()
    s = N.Scheduler.from_trace(trace, **cfg)
    for r in s.rounds():
        for i, o in enumerate(r.ops):
            h.update(np.array([r.round, o["rank"], o["kind"], o["task"], o["start"], o["count"]],
                              np.int64).tobytes())
            h.update(r.op_pages(i).astype(np.int64).tobytes())
        for e in r.events:
            h.update(np.array([r.round, e["kind"], e["task"], e["rank"]], np.int64).tobytes())
    st = s.stats()
    s.close()
    return h.hexdigest(), st


def _digest_oracle(trace, **cfg):
    import hashlib
    h = hashlib.sha256()
    sim = C.simulate(trace, C.Config(**cfg))
    by_round = {}
    for o in sim.ops:
        by_round.setdefault(o[0], []).append(o)
    evs = {}
    for e in sim.events:
        evs.setdefault(e[0], []).append(e)
    for rnd in range(sim.round):
        for o in by_round.get(rnd, []):
            h.update(np.array(o[:6], np.int64).tobytes())
            h.update(np.array(o[6], np.int64).tobytes())
        for e in evs.get(rnd, []):
            h.update(np.array(e, np.int64).tobytes())
    return h.hexdigest(), sim.stats


@pytest.mark.parametrize("cfg", [dict(policy=0), dict(policy=1, max_in_flight=1024)],
                         ids=["ctb", "request_f1024"])
def test_native_matches_oracle_on_the_full_webshop_step(cfg):
    """The benchmark's workload at full size (1056 trajectories, ~2,000 rounds): every op,
    page id and event, compared through a SHA-256 over both streams."""
    tr = T.make_trace("webshop_step")
    cfg = dict(pages_per_rank=57344, max_running=256, **cfg)
    assert _digest_native(tr, **cfg) == _digest_oracle(tr, **cfg)


@pytest.mark.parametrize("cfg", [dict(policy=0, pages_per_rank=1000, max_running=48),
                                 dict(policy=1, pages_per_rank=1000, max_running=48,
                                      max_in_flight=64)], ids=["ctb", "request_f64"])
def test_native_rounds_never_share_a_page(cfg):
    """What the batched GPU replay relies on: the ops of one round touch disjoint pages,
    and every op's pages hold exactly its own context up to its start."""
    tr = T.make_trace(T.TRACE_SPECS["webshop_step"].shrunk(4, 12, 4))
    s = N.Scheduler.from_trace(tr, **cfg)
    content = {}
    for r in s.rounds():
        owner = {}
        for i, o in enumerate(r.ops):
            t, st, ct = int(o["task"]), int(o["start"]), int(o["count"])
            pg = r.op_pages(i)
            for p in pg:
                assert owner.setdefault(int(p), t) == t, (r.round, int(p))
            for pos in range(0, st, 7):
                assert content.get((int(pg[pos // 16]), pos % 16)) == (t, pos)
            for pos in range(st, st + ct):
                content[(int(pg[pos // 16]), pos % 16)] = (t, pos)
    s.close()
