"""Seeded synthetic multi-turn rollout traces for the task-batching scheduler.

A trace is a rollout step: GRPO groups of trajectories (training groups and evaluation
groups), each trajectory a sequence of turns.  Turn k of a trajectory first appends
`new_tokens[k]` input tokens (the prompt for k = 0, the environment's observation after
that), then generates `gen_tokens[k]` tokens one at a time, then waits `env_rounds[k]`
engine rounds for the environment (not after its last turn).  Trajectories of one group
share the prompt length.  Shapes follow the task-statistics table of Appendix C (WebShop:
about 8 turns and 3400 tokens per trajectory) and the single-instance step of Section 6.5
(32 training groups of 8 and 200 evaluation groups of 4 trajectories).

K/V/Q rows of trajectory t at position p come from the same counter-based generator as
the attention workloads (stream b = t), so a row never depends on the schedule: resuming
over retained pages and recomputing give the same K/V.

This module only draws inputs; it holds no scheduling or attention logic.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace

import numpy as np

from . import _native
from .configs import TENSOR_K, TENSOR_Q, TENSOR_V


@dataclass(frozen=True)
class TraceSpec:
    key: str
    index: int
    text: str
    train_groups: int
    train_group_size: int
    eval_groups: int
    eval_group_size: int
    turns: tuple        # ("uniform", lo, hi) turns per trajectory
    prompt: tuple       # ("uniform", lo, hi) tokens, one draw per group
    obs: tuple          # ("uniform", lo, hi) observation tokens per later turn
    gen: tuple          # ("uniform", lo, hi) generated tokens per turn
    env: tuple          # ("uniform", lo, hi) engine rounds the environment takes
    num_q_heads: int = 28
    num_kv_heads: int = 4
    head_dim: int = 128
    salt: int = 0

    def shrunk(self, train_groups: int, eval_groups: int, length_div: int,
               salt: int = 1) -> "TraceSpec":
        def div(law, floor=1):
            return (law[0], max(floor, law[1] // length_div), max(floor, law[2] // length_div))
        return replace(self, train_groups=train_groups, eval_groups=eval_groups,
                       prompt=div(self.prompt), obs=div(self.obs), gen=div(self.gen),
                       env=div(self.env), salt=salt)


TRACE_SPECS = {
    "webshop_step": TraceSpec(
        key="webshop_step", index=50,
        text=("One rollout step shaped like WebShop: 32 training groups x 8 and 200 evaluation "
              "groups x 4 trajectories (1056), 3-13 turns, prompt 400-800 tokens per group, "
              "observations 150-450 tokens, 20-80 generated tokens per turn, environment "
              "10-60 engine rounds; Qwen2.5-7B attention shape (28 q / 4 kv heads, d=128)"),
        train_groups=32, train_group_size=8, eval_groups=200, eval_group_size=4,
        turns=("uniform", 3, 13), prompt=("uniform", 400, 800), obs=("uniform", 150, 450),
        gen=("uniform", 20, 80), env=("uniform", 10, 60)),
}


@dataclass
class Trace:
    spec: TraceSpec
    group: np.ndarray        # int32 [N]   GRPO group of each trajectory
    is_eval: np.ndarray      # int32 [N]   1 = evaluation trajectory
    group_size: np.ndarray   # int32 [num_groups]
    turn_start: np.ndarray   # int32 [N+1] turns of trajectory t: turn_start[t] .. [t+1]-1
    new_tokens: np.ndarray   # int32 [num_turns]
    gen_tokens: np.ndarray   # int32 [num_turns]
    env_rounds: np.ndarray   # int32 [num_turns]
    seeds: dict

    @property
    def num_tasks(self) -> int:
        return int(self.group.size)

    def final_len(self, t: int) -> int:
        a, b = int(self.turn_start[t]), int(self.turn_start[t + 1])
        return int(self.new_tokens[a:b].sum() + self.gen_tokens[a:b].sum())

    @property
    def final_lens(self) -> np.ndarray:
        return np.array([self.final_len(t) for t in range(self.num_tasks)], np.int64)

    def rows(self, which: str, t: int, p0: int, p1: int) -> np.ndarray:
        """bf16 bits of rows p0..p1-1 of trajectory t: [n, heads, d]."""
        tensor = {"q": TENSOR_Q, "k": TENSOR_K, "v": TENSOR_V}[which]
        heads = self.spec.num_q_heads if which == "q" else self.spec.num_kv_heads
        d = self.spec.head_dim
        n = max(0, p1 - p0)
        flat = _native.normal_bf16(self.seeds[tensor], tensor, t, p0 * heads * d, n * heads * d)
        return flat.reshape(n, heads, d)

    def segments(self, which: str, tasks, p0, p1) -> np.ndarray:
        """Rows p0[i]..p1[i]-1 of trajectory tasks[i], concatenated: [sum n, heads, d]."""
        tensor = {"q": TENSOR_Q, "k": TENSOR_K, "v": TENSOR_V}[which]
        heads = self.spec.num_q_heads if which == "q" else self.spec.num_kv_heads
        d = self.spec.head_dim
        p0 = np.asarray(p0, np.int64)
        n = np.asarray(p1, np.int64) - p0
        flat = _native.normal_bf16_segments(self.seeds[tensor], tensor,
                                            np.asarray(tasks, np.uint32),
                                            (p0 * heads * d).astype(np.uint64), n * heads * d)
        return flat.reshape(-1, heads, d)


def make_trace(spec: TraceSpec | str) -> Trace:
    """Draw one trace.  Same spec => same trace."""
    if isinstance(spec, str):
        spec = TRACE_SPECS[spec]
    ss = np.random.SeedSequence([2608, 10402, spec.index, spec.salt])
    c_order, c_len, c_q, c_k, c_v = ss.spawn(5)
    sizes = [spec.train_group_size] * spec.train_groups + [spec.eval_group_size] * spec.eval_groups
    evals = [0] * spec.train_groups + [1] * spec.eval_groups
    # groups arrive in a seeded order; a group's trajectories arrive together
    order = np.random.Generator(np.random.PCG64(c_order)).permutation(len(sizes))
    rng = np.random.Generator(np.random.PCG64(c_len))

    def u(law, n=None):
        return rng.integers(law[1], law[2], size=n, endpoint=True)

    group, is_eval, turn_start = [], [], [0]
    new_tokens, gen_tokens, env_rounds = [], [], []
    group_size = np.zeros(len(sizes), np.int32)
    for gi, g in enumerate(order):
        group_size[gi] = sizes[g]
        prompt = int(u(spec.prompt))
        for _ in range(sizes[g]):
            k = int(u(spec.turns))
            group.append(gi)
            is_eval.append(evals[g])
            new_tokens.extend([prompt] + [int(x) for x in u(spec.obs, k - 1)])
            gen_tokens.extend(int(x) for x in u(spec.gen, k))
            env_rounds.extend(int(x) for x in u(spec.env, k))
            turn_start.append(turn_start[-1] + k)

    def seed64(c):
        w = c.generate_state(2, np.uint32)
        return int(w[0]) | (int(w[1]) << 32)

    return Trace(spec=spec, group=np.array(group, np.int32), is_eval=np.array(is_eval, np.int32),
                 group_size=group_size, turn_start=np.array(turn_start, np.int32),
                 new_tokens=np.array(new_tokens, np.int32),
                 gen_tokens=np.array(gen_tokens, np.int32),
                 env_rounds=np.array(env_rounds, np.int32),
                 seeds={TENSOR_Q: seed64(c_q), TENSOR_K: seed64(c_k), TENSOR_V: seed64(c_v)})


def custom_trace(tasks, group_size=None, is_eval=None, num_q_heads=4, num_kv_heads=2,
                 head_dim=64, seed=0) -> Trace:
    """A trace with explicit turns: tasks[t] = (group, [(new, gen, env), ...])."""
    group, turn_start, new, gen, env = [], [0], [], [], []
    for g, turns in tasks:
        group.append(int(g))
        for n, a, e in turns:
            new.append(int(n)); gen.append(int(a)); env.append(int(e))
        turn_start.append(turn_start[-1] + len(turns))
    ng = max(group) + 1 if group else 0
    if group_size is None:
        group_size = np.bincount(np.array(group, np.int64), minlength=ng)
    if is_eval is None:
        is_eval = [0] * len(group)
    spec = TraceSpec(key="custom_trace", index=400 + seed, text="explicit turns",
                     train_groups=0, train_group_size=0, eval_groups=0, eval_group_size=0,
                     turns=(), prompt=(), obs=(), gen=(), env=(), num_q_heads=num_q_heads,
                     num_kv_heads=num_kv_heads, head_dim=head_dim, salt=seed)
    ss = np.random.SeedSequence([2608, 10402, spec.index, spec.salt])
    c_q, c_k, c_v = ss.spawn(3)

    def seed64(c):
        w = c.generate_state(2, np.uint32)
        return int(w[0]) | (int(w[1]) << 32)

    return Trace(spec=spec, group=np.array(group, np.int32), is_eval=np.array(is_eval, np.int32),
                 group_size=np.asarray(group_size, np.int32),
                 turn_start=np.array(turn_start, np.int32), new_tokens=np.array(new, np.int32),
                 gen_tokens=np.array(gen, np.int32), env_rounds=np.array(env, np.int32),
                 seeds={TENSOR_Q: seed64(c_q), TENSOR_K: seed64(c_k), TENSOR_V: seed64(c_v)})
