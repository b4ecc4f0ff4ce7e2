"""Binding of the host-side task-batching scheduler (include/tide_ctb.h), and an engine
loop that executes its rounds with the attention kernels.

The scheduler (Algorithm 1 of Section 4, or the request-level baseline) is native code
in libtide.so; this module marshals its inputs and reads back each round's ops.
`Replay` then runs those ops on one rank's page pool: for every extend op the new rows
are appended and attended over the retained prefix (tide_kv_append + tide_extend_attn),
for every decode op one row is appended and decoded in one fused call
(tide_decode_append_attn).
Row contents come from a caller-supplied function, so the loop holds no model.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import _lib
from ._lib import TideError
from .kvcache import PagedKV

POLICY_CTB = 0
POLICY_REQUEST = 1
OP_EXTEND = 0
OP_DECODE = 1
EV_ADMIT, EV_PAUSE, EV_RESUME, EV_FINISH = 0, 1, 2, 3
PAGE = 16


class tide_ctb_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "policy", "num_ranks", "pages_per_rank", "budget_tokens", "max_running",
        "max_in_flight", "env_capacity", "max_rounds")]


class tide_ctb_op(ctypes.Structure):
    _fields_ = [("rank", ctypes.c_int32), ("kind", ctypes.c_int32), ("task", ctypes.c_int32),
                ("start", ctypes.c_int32), ("count", ctypes.c_int32),
                ("num_pages", ctypes.c_int32), ("page_offset", ctypes.c_int64)]


class tide_ctb_event(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("task", ctypes.c_int32), ("rank", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class tide_ctb_round(ctypes.Structure):
    _fields_ = [("round", ctypes.c_int32), ("done", ctypes.c_int32),
                ("num_ops", ctypes.c_int32), ("num_events", ctypes.c_int32),
                ("num_pages", ctypes.c_int64), ("ops", ctypes.POINTER(tide_ctb_op)),
                ("pages", ctypes.POINTER(ctypes.c_int32)),
                ("events", ctypes.POINTER(tide_ctb_event))]


class tide_ctb_stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in (
        "rounds", "extend_ops", "decode_ops", "hit_tokens", "queried_tokens", "extend_tokens",
        "input_tokens", "pauses", "resumes", "admits")]


_OP_DTYPE = np.dtype([("rank", "<i4"), ("kind", "<i4"), ("task", "<i4"), ("start", "<i4"),
                      ("count", "<i4"), ("num_pages", "<i4"), ("page_offset", "<i8")])
_EV_DTYPE = np.dtype([("kind", "<i4"), ("task", "<i4"), ("rank", "<i4"), ("reserved", "<i4")])
assert _OP_DTYPE.itemsize == ctypes.sizeof(tide_ctb_op)


class Round:
    """One scheduled round: numpy copies of its ops, page ids and events."""

    def __init__(self, r: tide_ctb_round):
        self.round = int(r.round)
        self.done = bool(r.done)
        self.ops = _copy(r.ops, r.num_ops, _OP_DTYPE)
        self.pages = _copy(r.pages, r.num_pages, np.dtype("<i4"))
        self.events = _copy(r.events, r.num_events, _EV_DTYPE)

    def op_pages(self, i: int) -> np.ndarray:
        o = self.ops[i]
        return self.pages[o["page_offset"]: o["page_offset"] + o["num_pages"]]


def _copy(ptr, n, dtype):
    n = int(n)
    if n == 0:
        return np.zeros(0, dtype)
    buf = ctypes.string_at(ctypes.cast(ptr, ctypes.c_void_p), n * dtype.itemsize)
    return np.frombuffer(buf, dtype=dtype).copy()


class Scheduler:
    """tide_ctb_create / tide_ctb_step / tide_ctb_get_stats / tide_ctb_destroy."""

    def __init__(self, group, is_eval, group_size, turn_start, new_tokens, gen_tokens,
                 env_rounds, policy=POLICY_CTB, num_ranks=1, pages_per_rank=1024,
                 budget_tokens=None, max_running=256, max_in_flight=1024, env_capacity=0,
                 max_rounds=10_000_000):
        lib = _lib.load()
        arrs = [np.ascontiguousarray(a, dtype=np.int32) for a in
                (group, is_eval, group_size, turn_start, new_tokens, gen_tokens, env_rounds)]
        self._keep = arrs
        g, e, gs, ts, nt, gt, er = arrs
        self.config = tide_ctb_config(
            policy, num_ranks, pages_per_rank,
            pages_per_rank * PAGE if budget_tokens is None else budget_tokens, max_running,
            max_in_flight, env_capacity, max_rounds)
        h = ctypes.c_void_p()
        st = lib.tide_ctb_create(ctypes.byref(self.config), int(g.size), g.ctypes.data,
                                 e.ctypes.data, int(gs.size), gs.ctypes.data, ts.ctypes.data,
                                 nt.ctypes.data, gt.ctypes.data, er.ctypes.data, ctypes.byref(h))
        if st != 0:
            raise TideError(st, "tide_ctb_create")
        self._h = h
        self._lib = lib

    @classmethod
    def from_trace(cls, trace, **cfg):
        return cls(trace.group, trace.is_eval, trace.group_size, trace.turn_start,
                   trace.new_tokens, trace.gen_tokens, trace.env_rounds, **cfg)

    def step(self) -> Round:
        r = tide_ctb_round()
        st = self._lib.tide_ctb_step(self._h, ctypes.byref(r))
        if st != 0:
            raise TideError(st, "tide_ctb_step")
        return Round(r)

    def rounds(self):
        """Yields rounds until every task has finished."""
        while True:
            r = self.step()
            yield r
            if r.done:
                return

    def stats(self) -> dict:
        s = tide_ctb_stats()
        st = self._lib.tide_ctb_get_stats(self._h, ctypes.byref(s))
        if st != 0:
            raise TideError(st, "tide_ctb_get_stats")
        return {name: int(getattr(s, name)) for name, _ in tide_ctb_stats._fields_}

    def close(self):
        if self._h is not None:
            self._lib.tide_ctb_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Replay:
    """Runs one rank's scheduled ops on a PagedKV pool with the attention kernels.

    rows(which, tasks, p0, p1) must return rows p0[i]..p1[i]-1 of every task tasks[i],
    concatenated: [sum n, heads, d] with heads the query heads for "q" and the KV heads
    for "k" / "v" -- either as a bf16 device tensor, or as bf16 bit patterns (uint16
    numpy) that are uploaded.  Each round's inputs are ready before its kernels are
    queued, so per-stage events bracket only the library calls (their work-list uploads
    and kernels).
    """

    def __init__(self, kv: PagedKV, rows, rank: int = 0, with_lse: bool = False):
        self.kv = kv
        self.rows = rows
        self.rank = rank
        self.with_lse = with_lse
        self.ms = {"extend": 0.0, "decode": 0.0}   # event time of each stage, summed
        self.tokens = {"extend": 0, "decode": 0}
        self.flops = 0.0      # algorithmic extend FLOPs
        self.kv_bytes = 0.0   # algorithmic decode bytes (K/V read once per task and head)
        self.calls = 0
        self._events = []

    def _table(self, rnd: Round, idx) -> np.ndarray:
        n = [int(rnd.ops[i]["num_pages"]) for i in idx]
        bt = np.zeros((len(idx), max(n)), np.int32)
        for j, i in enumerate(idx):
            bt[j, : n[j]] = rnd.op_pages(i)
        return bt

    def _up(self, rows) -> torch.Tensor:
        if isinstance(rows, torch.Tensor):
            return rows
        t = torch.from_numpy(np.ascontiguousarray(rows).view(np.int16))
        return t.to(self.kv.device).view(torch.bfloat16)

    def run(self, rnd: Round, timed: bool = True) -> dict:
        """Executes the round's ops of this rank.  Returns the device outputs:
        {"extend": (op indices, out, lse), "decode": (op indices, out, lse)}."""
        kv, dev = self.kv, self.kv.device
        d = self.kv.dims
        ops = rnd.ops
        mine = np.nonzero(ops["rank"] == self.rank)[0]
        result = {}
        for kind, name in ((OP_EXTEND, "extend"), (OP_DECODE, "decode")):
            idx = mine[ops["kind"][mine] == kind]
            if idx.size == 0:
                continue
            tasks = ops["task"][idx]
            start = ops["start"][idx].astype(np.int32)
            count = ops["count"][idx].astype(np.int32)
            bt = torch.from_numpy(self._table(rnd, idx)).to(dev)
            k = self._up(self.rows("k", tasks, start, start + count))
            v = self._up(self.rows("v", tasks, start, start + count))
            q = self._up(self.rows("q", tasks, start, start + count))
            out = torch.empty_like(q)
            lse = (torch.empty((q.shape[0], q.shape[1]), dtype=torch.float32, device=dev)
                   if self.with_lse else None)
            if timed:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
            if kind == OP_EXTEND:
                ws = kv.workspace(max(
                    _lib.tide_workspace_size(_lib.TIDE_OP_KV_APPEND, start, count, d),
                    _lib.tide_workspace_size(_lib.TIDE_OP_EXTEND, start, count, d)))
            else:
                kv_len = (start + 1).astype(np.int32)
                ws = kv.workspace(_lib.tide_workspace_size(_lib.TIDE_OP_DECODE, kv_len, None, d))
            if timed:
                e0.record()
            if kind == OP_EXTEND:
                _lib.tide_kv_append(k, v, kv.k_pool, kv.v_pool, bt, start, count, d, ws)
                _lib.tide_extend_attn(q, kv.k_pool, kv.v_pool, bt, start, count, d, out, lse, ws)
                pe = start.astype(np.float64), count.astype(np.float64)
                self.flops += 4.0 * d.head_dim * d.num_q_heads * float(
                    np.sum(pe[1] * pe[0] + pe[1] * (pe[1] + 1) / 2))
            else:
                # one token per task: the append is fused into the decode call
                _lib.tide_decode_append_attn(q, k, v, kv.k_pool, kv.v_pool, bt, kv_len, d, out,
                                             lse, 0, ws)
                self.kv_bytes += float(np.sum(kv_len)) * d.num_kv_heads * d.head_dim * 4
            if timed:
                e1.record()
                self._events.append((name, e0, e1))
            self.tokens[name] += int(count.sum())
            self.calls += 1
            result[name] = (idx, out, lse)
        return result

    def collect(self):
        """Waits for the queued rounds and adds their stage times."""
        torch.cuda.synchronize()
        for name, e0, e1 in self._events:
            self.ms[name] += e0.elapsed_time(e1)
        self._events = []
