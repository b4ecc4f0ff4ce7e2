"""Full-size parity: the workloads at their real sizes, in the launch configuration
the benchmark times (automatic work lists and split counts), checked on sampled rows
that the fp64 oracle recomputes one by one, plus invariants checked on every row.

For each sampled task the oracle rebuilds that task alone in a compact pool of its own
(its own append, its own page order) from the seeded generator; the GPU ran on the
full fragmented pool.  Physical placement does not change the result (pinned for the
oracle on the CPU), so the comparison is exact up to the GPU's bf16 rounding.
"""
import gc
import os

import numpy as np
import pytest
import torch

import workloads as W
from gpu_harness import (DeviceWorkload, assert_close, assert_lse, dev_bf16, host_bits, log,
                         oracle_task_rows, sample_tasks)

pytestmark = pytest.mark.gpu


def _free():
    gc.collect()
    torch.cuda.empty_cache()


def _check_extend_rows(wl, out, lse, tasks, rows_per_task=3, seed=0, what="extend"):
    rng = np.random.default_rng(seed)
    indptr = np.concatenate([[0], np.cumsum(wl.extend_lens)])
    got, ref, got_l, ref_l = [], [], [], []
    for b in tasks:
        p, e = int(wl.prefix_lens[b]), int(wl.extend_lens[b])
        if e == 0:
            continue
        local = sorted(set([0, e - 1] + rng.integers(0, e, size=rows_per_task).tolist()))
        pos, o, l = oracle_task_rows(wl, b, [p + j for j in local], upto=p + e)
        rows = torch.as_tensor([int(indptr[b]) + j for j in local], device=out.device)
        got.append(out[rows])
        got_l.append(lse[rows])
        ref.append(o)
        ref_l.append(l)
    assert_close(torch.cat(got), np.concatenate(ref), "%s %s sampled" % (wl.spec.key, what))
    assert_lse(torch.cat(got_l), np.concatenate(ref_l), "%s %s sampled" % (wl.spec.key, what))


def _check_append_pages(wl, dw, tasks, upto_fn):
    """The GPU pool holds each sampled task's K/V at (BT[b][p//16], p%16), bit for bit."""
    kp = dw.kv.k_pool
    vp = dw.kv.v_pool
    for b in tasks:
        n = upto_fn(b)
        pages = torch.as_tensor(wl.block_table[b, : -(-n // 16)].astype(np.int64), device=kp.device)
        gk = host_bits(kp[pages])  # [npages, Hkv, 16, d]
        gv = host_bits(vp[pages])  # [npages, Hkv, 16, d]
        k = wl.k_rows(b, 0, n)
        v = wl.v_rows(b, 0, n)
        pos = np.arange(n)
        assert np.array_equal(gk[pos // 16, :, pos % 16, :], k), "task %d K pages" % b
        assert np.array_equal(gv[pos // 16, :, pos % 16, :], v), "task %d V pages" % b


@pytest.fixture(scope="module")
def agent_resume():
    wl = W.make_workload("agent_resume_7b")
    log("agent_resume_7b: T_ext=%d sumL=%d" % (wl.extend_lens.sum(), wl.seq_lens.sum()))
    dw = DeviceWorkload(wl)
    dw.append_extend()
    torch.cuda.synchronize()
    yield wl, dw
    del dw
    _free()


def test_agent_resume_extend(agent_resume):
    wl, dw = agent_resume
    out, lse = dw.extend()
    _check_extend_rows(wl, out, lse, sample_tasks(wl, 4, seed=1))
    _check_append_pages(wl, dw, sample_tasks(wl, 2, seed=2), lambda b: int(wl.seq_lens[b]))


def test_agent_resume_one_task_split(agent_resume):
    """The bench's one-task resume: the longest-prefix task alone, which the planner runs
    split-KV (a few dozen items for 256 CUs).  Sampled rows against the oracle, and the
    split rows against the same task's rows from the plain plan."""
    wl, dw = agent_resume
    b = int(np.argmax(wl.prefix_lens))
    indptr = np.concatenate([[0], np.cumsum(wl.extend_lens)]).astype(np.int64)
    q = dev_bf16(wl.packed("q", wl.extend_ranges()))[int(indptr[b]):int(indptr[b + 1])]
    ext = np.zeros(wl.num_tasks, np.int32)
    ext[b] = wl.extend_lens[b]
    outs = {}
    for mode in ("1", "0"):
        os.environ["TIDE_EXTEND_SPLIT"] = mode
        try:
            lse = torch.empty((q.shape[0], q.shape[1]), dtype=torch.float32, device=q.device)
            outs[mode] = (dw.kv.extend(q, wl.prefix_lens, ext, lse=lse), lse)
        finally:
            os.environ.pop("TIDE_EXTEND_SPLIT", None)
    torch.cuda.synchronize()
    p, e = int(wl.prefix_lens[b]), int(wl.extend_lens[b])
    rng = np.random.default_rng(5)
    local = sorted(set([0, e - 1] + rng.integers(0, e, size=6).tolist()))
    pos, o, l = oracle_task_rows(wl, b, [p + j for j in local], upto=p + e)
    rows = torch.as_tensor(local, device=q.device)
    out_s, lse_s = outs["1"]
    assert_close(out_s[rows], o, "agent_resume_7b one-task split sampled")
    assert_lse(lse_s[rows], l, "agent_resume_7b one-task split sampled")
    d = (out_s.float() - outs["0"][0].float()).abs()
    log("one-task split vs plain: max %.3g mean %.3g" % (d.max().item(), d.mean().item()))
    assert d.max().item() <= 2e-2 and d.mean().item() <= 2e-3


def test_agent_resume_prefill_and_equivalence(agent_resume):
    """Full re-prefill: sampled rows (prefix region too) against the oracle, and every
    extend row equal to the matching re-prefill row (the equivalence a cache hit relies on)."""
    wl, dw = agent_resume
    full, full_lse = dw.prefill()
    ext, _ = dw.extend(lse=False)
    indptr = np.concatenate([[0], np.cumsum(wl.seq_lens)])
    rng = np.random.default_rng(3)
    got, ref = [], []
    for b in sample_tasks(wl, 3, seed=4):
        L = int(wl.seq_lens[b])
        local = sorted(set([0, 1, L - 1] + rng.integers(0, L, size=3).tolist()))
        _, o, _ = oracle_task_rows(wl, b, local, upto=L)
        got.append(full[torch.as_tensor([int(indptr[b]) + j for j in local], device=full.device)])
        ref.append(o)
    assert_close(torch.cat(got), np.concatenate(ref), "agent_resume_7b prefill sampled")
    # every extend row vs the re-prefill row of the same position
    sel = np.concatenate([np.arange(int(indptr[b] + wl.prefix_lens[b]), int(indptr[b + 1]))
                          for b in range(wl.num_tasks)])
    d = (ext.float() - full[torch.as_tensor(sel, device=full.device)].float()).abs()
    log("agent_resume_7b extend vs prefill rows: max %.3e mean %.3e" % (d.max().item(), d.mean().item()))
    assert d.max().item() <= 2e-2 and d.mean().item() <= 2e-3


def test_agent_resume_decode(agent_resume):
    wl, dw = agent_resume
    last = np.cumsum(wl.extend_lens) - 1
    q = wl.packed("q", [(int(l) - 1, int(l)) for l in wl.seq_lens])
    lse = torch.empty((wl.num_tasks, wl.spec.num_q_heads), dtype=torch.float32, device="cuda")
    out = dw.kv.decode(dev_bf16(q), wl.seq_lens, lse=lse)
    tasks = sample_tasks(wl, 4, seed=5)
    ref = [oracle_task_rows(wl, b, [int(wl.seq_lens[b]) - 1])[1:] for b in tasks]
    sel = torch.as_tensor(tasks, device="cuda")
    assert_close(out[sel], np.concatenate([r[0] for r in ref]), "agent_resume_7b decode sampled")
    assert_lse(lse[sel], np.concatenate([r[1] for r in ref]), "agent_resume_7b decode sampled")
    del last


def test_resumed_decode_fullsize():
    wl = W.make_workload("resumed_decode")
    log("resumed_decode: sum ctx=%d" % wl.seq_lens.sum())
    dw = DeviceWorkload(wl)
    dw.append_extend()  # the decoded token's own K/V
    q = wl.packed("q", wl.extend_ranges())
    qd = dev_bf16(q)
    lse = torch.empty((wl.num_tasks, wl.spec.num_q_heads), dtype=torch.float32, device="cuda")
    out = dw.kv.decode(qd, wl.seq_lens, lse=lse)
    tasks = sample_tasks(wl, 6, seed=6)
    ref = [oracle_task_rows(wl, b, [int(wl.seq_lens[b]) - 1])[1:] for b in tasks]
    sel = torch.as_tensor(tasks, device="cuda")
    assert_close(out[sel], np.concatenate([r[0] for r in ref]), "resumed_decode sampled")
    assert_lse(lse[sel], np.concatenate([r[1] for r in ref]), "resumed_decode sampled")
    # every task: split count does not matter beyond fp32 rounding
    out1 = dw.kv.decode(qd, wl.seq_lens, num_splits=1)
    d = (out.float() - out1.float()).abs().max().item()
    log("resumed_decode auto vs 1 split: max %.3e" % d)
    assert d <= 1e-2
    _check_append_pages(wl, dw, tasks[:2], lambda b: int(wl.seq_lens[b]))
    del dw
    _free()


def test_multimodal_resume_fullsize():
    wl = W.make_workload("multimodal_resume")
    log("multimodal_resume: T_ext=%d sumL=%d" % (wl.extend_lens.sum(), wl.seq_lens.sum()))
    dw = DeviceWorkload(wl)
    dw.append_extend()
    out, lse = dw.extend()
    _check_extend_rows(wl, out, lse, sample_tasks(wl, 4, seed=7))
    del dw
    _free()


def _check_stale_pages(wl, dw, tasks):
    """Past the resumed end the pages still hold the pre-prune context, bit for bit."""
    kp, vp = dw.kv.k_pool, dw.kv.v_pool
    for b in tasks:
        n, s = int(wl.seq_lens[b]), int(wl.stale_lens[b])
        pos = np.arange(n, s)
        pages = torch.as_tensor(wl.block_table[b, pos // 16].astype(np.int64), device=kp.device)
        slots = torch.as_tensor(pos % 16, device=kp.device)
        gk = host_bits(kp[pages, :, slots, :])  # [n, Hkv, d]
        gv = host_bits(vp[pages, :, slots, :])  # [n, Hkv, d]
        assert np.array_equal(gk, wl.stale_rows("k", b, n, s)), "task %d stale K" % b
        assert np.array_equal(gv, wl.stale_rows("v", b, n, s)), "task %d stale V" % b


def test_multimodal_prune_resume_fullsize():
    """Resume after the sliding-window prune: the re-encoded tail is appended over pages
    holding the pre-prune context, then extend over the prompt; sampled rows against the
    oracle (which never saw the stale context), the written pages bit for bit, the stale
    slots past the end untouched, and extend rows equal to the re-prefill's."""
    wl = W.make_workload("multimodal_prune_resume")
    log("multimodal_prune_resume: T_ext=%d sumL=%d stale=%d" % (
        wl.extend_lens.sum(), wl.seq_lens.sum(), wl.stale_lens.sum()))
    dw = DeviceWorkload(wl)
    dw.append_extend()
    out, lse = dw.extend()
    tasks = sample_tasks(wl, 4, seed=12)
    _check_extend_rows(wl, out, lse, tasks)
    _check_append_pages(wl, dw, tasks[:2], lambda b: int(wl.seq_lens[b]))
    _check_stale_pages(wl, dw, tasks)
    full, _ = dw.prefill(lse=False)
    indptr_e = np.concatenate([[0], np.cumsum(wl.extend_lens)])
    indptr_f = np.concatenate([[0], np.cumsum(wl.seq_lens)])
    for b in tasks:
        p, e = int(wl.prefix_lens[b]), int(wl.extend_lens[b])
        a = out[int(indptr_e[b]):int(indptr_e[b]) + e].float()
        f = full[int(indptr_f[b]) + p:int(indptr_f[b]) + p + e].float()
        assert (a - f).abs().max().item() <= 2e-2, b
    del dw, out, lse, full
    _free()


def test_long_horizon_fullsize():
    """Append the resumed tokens into a 90%-occupied pool, extend, then 8 rounds of
    (append one token, decode)."""
    wl = W.make_workload("long_horizon")
    log("long_horizon: T_ext=%d sumL=%d pages=%d" % (wl.extend_lens.sum(), wl.seq_lens.sum(),
                                                     wl.num_pages))
    dw = DeviceWorkload(wl)
    dw.append_extend()
    out, lse = dw.extend()
    tasks = sample_tasks(wl, 3, seed=8)
    _check_extend_rows(wl, out, lse, tasks, rows_per_task=2)
    del out, lse
    dec = []
    for step in range(wl.spec.decode_steps):
        rng = wl.decode_ranges(step)
        pos = wl.seq_lens + step
        dw.kv.append(dev_bf16(wl.packed("k", rng)), dev_bf16(wl.packed("v", rng)), pos,
                     np.ones(wl.num_tasks, np.int32))
        dec.append(dw.kv.decode(dev_bf16(wl.packed("q", rng)), pos + 1))
    torch.cuda.synchronize()
    sel = torch.as_tensor(tasks, device="cuda")
    got = torch.stack([d[sel] for d in dec], dim=1)  # [tasks, steps, Hq, d]
    ref = []
    for b in tasks:
        L = int(wl.seq_lens[b])
        _, o, _ = oracle_task_rows(wl, b, [L + s for s in range(wl.spec.decode_steps)],
                                   upto=L + wl.spec.decode_steps)
        ref.append(o)
    assert_close(got.reshape(-1, *got.shape[2:]), np.concatenate(ref), "long_horizon decode steps")
    _check_append_pages(wl, dw, tasks[:2], lambda b: int(wl.final_lens[b]))
    del dw, dec
    _free()
