"""Test-side glue: put a seeded workload on the GPU through the library's own calls,
and compare results with the oracle.

The GPU pool is filled only by tide_kv_append (first the retained prefix, then the new
tokens), the oracle pool only by the oracle's own append; the two never exchange data.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import oracle_pins
import paper_2608_10402_amd as tide
import workloads as W

MAX_ABS_TOL = 2e-2   # bf16 outputs vs fp64 oracle: max |error|
MEAN_ABS_TOL = 2e-3  # and mean |error|
LSE_TOL = 1e-3


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def dev_bf16(bits: np.ndarray, device="cuda") -> torch.Tensor:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return torch.from_numpy(bits.view(np.int16)).to(device).view(torch.bfloat16)


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def host_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


class DeviceWorkload:
    """Device pools of a workload, with the prefix already appended."""

    def __init__(self, wl: W.Workload, device="cuda"):
        self.wl = wl
        s = wl.spec
        self.kv = tide.PagedKV(wl.num_pages, s.num_q_heads, s.num_kv_heads, s.head_dim,
                               wl.block_table, wl.sm_scale, device=device)
        zeros = np.zeros(wl.num_tasks, np.int32)
        if wl.shared_lens is not None:
            # GRPO groups: a group's prompt pages are written once (through its first
            # task), then every trajectory's own positions up to the decoded token
            shared = np.repeat(wl.shared_lens, np.diff(wl.group_start)).astype(np.int32)
            first = np.zeros(wl.num_tasks, np.int32)
            first[wl.group_start[:-1]] = wl.shared_lens
            rng = [(0, int(n)) for n in first]
            if first.sum() > 0:
                self.kv.append(dev_bf16(wl.packed("k", rng)), dev_bf16(wl.packed("v", rng)),
                               zeros, first)
            own = (wl.prefix_lens - shared).astype(np.int32)
            rng = [(int(a), int(a + n)) for a, n in zip(shared, own)]
            if own.sum() > 0:
                self.kv.append(dev_bf16(wl.packed("k", rng)), dev_bf16(wl.packed("v", rng)),
                               shared, own)
        elif wl.prefix_lens.sum() > 0:
            self.kv.append(dev_bf16(wl.packed("k", wl.prefix_ranges())),
                           dev_bf16(wl.packed("v", wl.prefix_ranges())), zeros, wl.prefix_lens)
        if wl.stale_lens is not None:
            # sliding-window prune: the pages still hold the context as it was before the
            # prune (encoded at the old positions); the resume writes over it
            n = (wl.stale_lens - wl.prefix_lens).astype(np.int32)
            if n.sum() > 0:
                self.kv.append(dev_bf16(wl.stale_packed("k")), dev_bf16(wl.stale_packed("v")),
                               wl.prefix_lens, n)

    def append_extend(self):
        wl = self.wl
        self.kv.append(dev_bf16(wl.packed("k", wl.extend_ranges())),
                       dev_bf16(wl.packed("v", wl.extend_ranges())), wl.prefix_lens,
                       wl.extend_lens)

    def extend(self, lse=True):
        wl = self.wl
        q = dev_bf16(wl.packed("q", wl.extend_ranges()))
        l = torch.empty((q.shape[0], q.shape[1]), dtype=torch.float32, device=q.device) if lse else None
        out = self.kv.extend(q, wl.prefix_lens, wl.extend_lens, lse=l)
        return out, l

    def prefill(self, lse=True):
        wl = self.wl
        q = dev_bf16(wl.packed("q", wl.full_ranges()))
        l = torch.empty((q.shape[0], q.shape[1]), dtype=torch.float32, device=q.device) if lse else None
        out = self.kv.prefill(q, wl.seq_lens, lse=l)
        return out, l


def oracle_pools(wl: W.Workload):
    return oracle_pins.oracle_pools_for(wl)


def assert_close(gpu: torch.Tensor, ref: np.ndarray, what: str, max_tol=MAX_ABS_TOL,
                 mean_tol=MEAN_ABS_TOL):
    g = host_f64(gpu)
    assert g.shape == ref.shape, (what, g.shape, ref.shape)
    assert np.isfinite(g).all(), "%s: non-finite GPU output" % what
    err = np.abs(g - ref)
    mx, mean = float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0
    log("%s: max abs err %.3e, mean abs err %.3e over %d values" % (what, mx, mean, err.size))
    assert mx <= max_tol, "%s: max abs error %.4g > %.4g" % (what, mx, max_tol)
    assert mean <= mean_tol, "%s: mean abs error %.4g > %.4g" % (what, mean, mean_tol)


def assert_lse(gpu: torch.Tensor, ref: np.ndarray, what: str, tol=LSE_TOL):
    g = gpu.cpu().numpy().astype(np.float64)
    err = np.abs(g - ref)
    mx = float(err.max()) if err.size else 0.0
    log("%s: lse max abs err %.3e" % (what, mx))
    assert mx <= tol, "%s: lse error %.4g > %.4g" % (what, mx, tol)


def oracle_task_pool(wl: W.Workload, b: int, n_pos: int):
    """Oracle pool images holding task b alone (positions 0 .. n_pos - 1, its own page
    order), written by the oracle's own append from the seeded generator."""
    s = wl.spec
    n_pages = -(-n_pos // 16)
    perm = np.random.default_rng(b + 17).permutation(n_pages).astype(np.int32)
    bt = perm.reshape(1, -1)
    kp, vp = oracle.new_pools(n_pages, s.num_kv_heads, s.head_dim)
    oracle.kv_append(wl.k_rows(b, 0, n_pos), wl.v_rows(b, 0, n_pos), kp, vp, bt,
                     np.array([0], np.int32), np.array([n_pos], np.int32))
    return kp, vp, bt


def oracle_task_rows(wl: W.Workload, b: int, rows, upto: int | None = None, pool=None):
    """fp64 oracle for selected query positions of task b, from a compact pool that holds
    only task b (its own append, its own page order).  `rows` are absolute positions;
    each attends to keys 0..row.  `upto` = number of positions to place (default: the
    last requested row + 1); `pool` = (kp, vp, bt) from oracle_task_pool, reused.
    Returns (sorted rows, out [n, Hq, d], lse [n, Hq])."""
    s = wl.spec
    rows = np.asarray(sorted(rows), dtype=np.int64)
    n_pos = int(upto if upto is not None else rows.max() + 1)
    kp, vp, bt = pool if pool is not None else oracle_task_pool(wl, b, n_pos)
    q = np.concatenate([wl.q_rows(b, int(r), int(r) + 1) for r in rows])
    out, lse = oracle.attention(q, rows, kp, vp, bt, np.array([0], np.int32),
                                np.array([n_pos], np.int32), s.num_q_heads, wl.sm_scale)
    return rows, out, lse


def sample_tasks(wl: W.Workload, k: int, seed: int = 0):
    """The longest and shortest task plus seeded others (k in total, distinct)."""
    L = wl.seq_lens
    picks = [int(np.argmax(L)), int(np.argmin(L))]
    rng = np.random.default_rng(seed)
    for b in rng.permutation(wl.num_tasks):
        if len(picks) >= k:
            break
        if int(b) not in picks:
            picks.append(int(b))
    return picks[:k]
