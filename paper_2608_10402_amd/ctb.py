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
    numpy) that are uploaded.  A source whose rows live on the device may also offer
    locate(tasks, p0, p1) -> locator and fetch(which, locator) -> tensor, so that a
    round can be prepared (locators, block tables) before it is executed.  Each round's
    inputs are ready before its kernels are queued, so per-stage events bracket only the
    library calls (their work-list uploads and kernels).
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

    def _to_device(self, arr: np.ndarray) -> torch.Tensor:
        """Host array -> device through a pinned copy, so that the host does not wait for
        the GPU to drain (a copy from pageable memory synchronises the stream): the host
        queues the next rounds while the GPU runs, and the events time GPU work only."""
        t = torch.from_numpy(np.ascontiguousarray(arr))
        if self.kv.device.type != "cuda":
            return t.to(self.kv.device)
        return t.pin_memory().to(self.kv.device, non_blocking=True)

    def _up(self, rows) -> torch.Tensor:
        if isinstance(rows, torch.Tensor):
            return rows
        return self._to_device(np.ascontiguousarray(rows).view(np.int16)).view(torch.bfloat16)

    def prepare(self, rnd: Round) -> list:
        """Everything a round needs on the device, taken from the scheduler's round while
        it is valid: per op kind the op indices, lengths, block table (on the device), the
        rows to attend (a device-side locator when the row source offers one, see
        `execute`) and the workspace size.  Preparing every round first and executing them
        afterwards keeps host work out of the timed calls."""
        ops = rnd.ops
        d = self.kv.dims
        mine = np.nonzero(ops["rank"] == self.rank)[0]
        prepared = []
        for kind, name in ((OP_EXTEND, "extend"), (OP_DECODE, "decode")):
            idx = mine[ops["kind"][mine] == kind]
            if idx.size == 0:
                continue
            tasks = ops["task"][idx].copy()
            start = ops["start"][idx].astype(np.int32)
            count = ops["count"][idx].astype(np.int32)
            if kind == OP_EXTEND:
                ws = max(_lib.tide_workspace_size(_lib.TIDE_OP_KV_APPEND, start, count, d),
                         _lib.tide_workspace_size(_lib.TIDE_OP_EXTEND, start, count, d))
            else:
                ws = _lib.tide_workspace_size(_lib.TIDE_OP_DECODE, (start + 1).astype(np.int32),
                                              None, d)
            loc = (self.rows.locate(tasks, start, start + count)
                   if hasattr(self.rows, "locate") else None)
            prepared.append(dict(kind=kind, name=name, idx=idx, tasks=tasks, start=start,
                                 count=count, bt=self._to_device(self._table(rnd, idx)),
                                 loc=loc, ws=ws))
        return prepared

    def execute(self, prepared: list, timed: bool = True) -> dict:
        """Runs prepared rounds' ops.  Rows come from rows.fetch(which, locator) when the
        source offers `locate`/`fetch` (device-resident rows), else from rows(which, tasks,
        p0, p1).  Returns {"extend": (op indices, out, lse), "decode": (...)}."""
        kv, dev = self.kv, self.kv.device
        d = self.kv.dims
        result = {}
        for p in prepared:
            kind, name, start, count, bt = p["kind"], p["name"], p["start"], p["count"], p["bt"]
            if p["loc"] is not None:
                k, v, q = (self.rows.fetch(w, p["loc"]) for w in ("k", "v", "q"))
            else:
                k, v, q = (self._up(self.rows(w, p["tasks"], start, start + count))
                           for w in ("k", "v", "q"))
            out = torch.empty_like(q)
            lse = (torch.empty((q.shape[0], q.shape[1]), dtype=torch.float32, device=dev)
                   if self.with_lse else None)
            ws = kv.workspace(p["ws"])
            if timed:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
            if kind == OP_EXTEND:
                _lib.tide_kv_append(k, v, kv.k_pool, kv.v_pool, bt, start, count, d, ws)
                _lib.tide_extend_attn(q, kv.k_pool, kv.v_pool, bt, start, count, d, out, lse, ws)
                pe = start.astype(np.float64), count.astype(np.float64)
                self.flops += 4.0 * d.head_dim * d.num_q_heads * float(
                    np.sum(pe[1] * pe[0] + pe[1] * (pe[1] + 1) / 2))
            else:
                # one token per task: the append is fused into the decode call
                kv_len = (start + 1).astype(np.int32)
                _lib.tide_decode_append_attn(q, k, v, kv.k_pool, kv.v_pool, bt, kv_len, d, out,
                                             lse, 0, ws)
                self.kv_bytes += float(np.sum(kv_len)) * d.num_kv_heads * d.head_dim * 4
            if timed:
                e1.record()
                self._events.append((name, e0, e1))
            self.tokens[name] += int(count.sum())
            self.calls += 1
            result[name] = (p["idx"], out, lse)
        return result

    def reserve(self, prepared_rounds) -> None:
        """Grows the pool's workspace to what the prepared rounds need, so that no
        allocation happens while they execute."""
        need = [p["ws"] for rnd in prepared_rounds for p in rnd]
        if need:
            self.kv.workspace(max(need))

    def run(self, rnd: Round, timed: bool = True) -> dict:
        """prepare + execute of one round."""
        return self.execute(self.prepare(rnd), timed)

    def collect(self):
        """Waits for the queued rounds and adds their stage times."""
        torch.cuda.synchronize()
        for name, e0, e1 in self._events:
            self.ms[name] += e0.elapsed_time(e1)
        self._events = []
