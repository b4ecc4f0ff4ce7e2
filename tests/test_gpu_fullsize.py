"""Full-size parity: the workloads at their real sizes, in the launch configuration
the benchmark times (automatic work lists and split counts), checked against the fp64
oracle on every task: each task's first and last new row plus seeded ones, all query
heads, and every decode row.

For each task the oracle rebuilds that task alone in a compact pool of its own (its own
append, its own page order) from the seeded generator; the GPU ran on the full
fragmented pool.  Physical placement does not change the result (pinned for the oracle
on the CPU), so the comparison is exact up to the GPU's bf16 rounding.  The slots the
resume wrote are compared with that pool bit for bit.
"""
import gc
import os

import numpy as np
import pytest
import torch

import workloads as W
from gpu_harness import (DeviceWorkload, assert_close, assert_lse, dev_bf16, host_bits, log,
                         oracle_task_pool, oracle_task_rows, sample_tasks)

pytestmark = pytest.mark.gpu


def _free():
    gc.collect()
    torch.cuda.empty_cache()


SEEDED_ROWS = 4  # per task, besides its first and last new row


def _local_rows(e: int, rng, extra: int = SEEDED_ROWS):
    return sorted(set([0, e - 1] + rng.integers(0, e, size=extra).tolist()))


def _check_written_slots(wl, dw, b, pool, lo, hi, what):
    """GPU pool slots of positions lo .. hi-1 of task b equal the oracle pool's, bit for bit."""
    if hi <= lo:
        return
    kp_o, vp_o, bt_o = pool
    pos = np.arange(lo, hi)
    dev = dw.kv.k_pool.device
    pages = torch.as_tensor(wl.block_table[b, pos // 16].astype(np.int64), device=dev)
    slots = torch.as_tensor(pos % 16, device=dev)
    op = bt_o[0, pos // 16]
    assert np.array_equal(host_bits(dw.kv.k_pool[pages, :, slots, :]), kp_o[op, :, pos % 16, :]), \
        "%s task %d K slots %d..%d" % (what, b, lo, hi)
    assert np.array_equal(host_bits(dw.kv.v_pool[pages, :, slots, :]), vp_o[op, :, pos % 16, :]), \
        "%s task %d V slots %d..%d" % (what, b, lo, hi)


def _check_extend_all(wl, dw, out, lse, seed=0, what="extend", extra_positions=None,
                      extra_check=None):
    """Every task: rows {0, E-1} plus SEEDED_ROWS seeded ones against the oracle (all
    heads), and the slots the resume wrote bit for bit.  extra_positions(b) adds
    positions to the same oracle call (with its pool), whose results go to
    extra_check(b, positions, out, lse)."""
    rng = np.random.default_rng(seed)
    indptr = np.concatenate([[0], np.cumsum(wl.extend_lens)])
    got, ref, got_l, ref_l = [], [], [], []
    n_rows = 0
    for b in range(wl.num_tasks):
        p, e = int(wl.prefix_lens[b]), int(wl.extend_lens[b])
        more = list(extra_positions(b)) if extra_positions else []
        if e == 0 and not more:
            continue
        local = _local_rows(e, rng) if e else []
        upto = max([p + e] + [x + 1 for x in more])
        pool = oracle_task_pool(wl, b, upto)
        pos, o, l = oracle_task_rows(wl, b, [p + j for j in local] + more, upto=upto, pool=pool)
        k = len(local)  # extend positions sort before the later extra ones
        if k:
            rows = torch.as_tensor([int(indptr[b]) + j for j in local], device=out.device)
            got.append(out[rows])
            got_l.append(lse[rows])
            ref.append(o[:k])
            ref_l.append(l[:k])
            n_rows += k
        if more:
            extra_check(b, pos[k:], o[k:], l[k:])
        _check_written_slots(wl, dw, b, pool, p, p + e, what)
        del pool
    log("%s %s: %d tasks, %d rows" % (wl.spec.key, what, wl.num_tasks, n_rows))
    assert_close(torch.cat(got), np.concatenate(ref), "%s %s all tasks" % (wl.spec.key, what))
    assert_lse(torch.cat(got_l), np.concatenate(ref_l), "%s %s all tasks" % (wl.spec.key, what))


def _check_decode_all(wl, out, lse, what):
    """Every task's decode row (the last context position) against the oracle."""
    o_all, l_all = [], []
    for b in range(wl.num_tasks):
        L = int(wl.seq_lens[b])
        _, o, l = oracle_task_rows(wl, b, [L - 1], upto=L)
        o_all.append(o)
        l_all.append(l)
    assert_close(out, np.concatenate(o_all), "%s %s all %d tasks" % (wl.spec.key, what, wl.num_tasks))
    assert_lse(lse, np.concatenate(l_all), "%s %s all %d tasks" % (wl.spec.key, what, wl.num_tasks))


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
    _check_extend_all(wl, dw, out, lse, seed=1)
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
    got, ref, got_l, ref_l = [], [], [], []
    for b in range(wl.num_tasks):  # every task: rows 0, 1, L-1 and seeded ones
        L = int(wl.seq_lens[b])
        local = sorted(set([0, 1, L - 1] + rng.integers(0, L, size=SEEDED_ROWS).tolist()))
        _, o, l = oracle_task_rows(wl, b, local, upto=L)
        sel_rows = torch.as_tensor([int(indptr[b]) + j for j in local], device=full.device)
        got.append(full[sel_rows])
        got_l.append(full_lse[sel_rows])
        ref.append(o)
        ref_l.append(l)
    assert_close(torch.cat(got), np.concatenate(ref), "agent_resume_7b prefill all tasks")
    assert_lse(torch.cat(got_l), np.concatenate(ref_l), "agent_resume_7b prefill all tasks")
    # every extend row vs the re-prefill row of the same position
    sel = np.concatenate([np.arange(int(indptr[b] + wl.prefix_lens[b]), int(indptr[b + 1]))
                          for b in range(wl.num_tasks)])
    d = (ext.float() - full[torch.as_tensor(sel, device=full.device)].float()).abs()
    log("agent_resume_7b extend vs prefill rows: max %.3e mean %.3e" % (d.max().item(), d.mean().item()))
    assert d.max().item() <= 2e-2 and d.mean().item() <= 2e-3


def test_agent_resume_decode(agent_resume):
    wl, dw = agent_resume
    q = wl.packed("q", [(int(l) - 1, int(l)) for l in wl.seq_lens])
    lse = torch.empty((wl.num_tasks, wl.spec.num_q_heads), dtype=torch.float32, device="cuda")
    out = dw.kv.decode(dev_bf16(q), wl.seq_lens, lse=lse)
    _check_decode_all(wl, out, lse, "decode")


def test_resumed_decode_fullsize():
    wl = W.make_workload("resumed_decode")
    log("resumed_decode: sum ctx=%d" % wl.seq_lens.sum())
    dw = DeviceWorkload(wl)
    dw.append_extend()  # the decoded token's own K/V
    q = wl.packed("q", wl.extend_ranges())
    qd = dev_bf16(q)
    lse = torch.empty((wl.num_tasks, wl.spec.num_q_heads), dtype=torch.float32, device="cuda")
    out = dw.kv.decode(qd, wl.seq_lens, lse=lse)
    _check_decode_all(wl, out, lse, "decode")
    tasks = sample_tasks(wl, 2, seed=6)
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
    _check_extend_all(wl, dw, out, lse, seed=7)
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
    _check_extend_all(wl, dw, out, lse, seed=12)
    _check_append_pages(wl, dw, tasks[:2], lambda b: int(wl.seq_lens[b]))
    _check_stale_pages(wl, dw, range(wl.num_tasks))
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
    """Append the resumed tokens into a 90%-occupied pool, extend, then 8 decode steps,
    each appending its token inside the attention call (tide_decode_append_attn), as the
    benchmark runs them.  Every task: extend rows and all 8 decode rows against the
    oracle, and every slot the resume and the decode steps wrote."""
    wl = W.make_workload("long_horizon")
    log("long_horizon: T_ext=%d sumL=%d pages=%d" % (wl.extend_lens.sum(), wl.seq_lens.sum(),
                                                     wl.num_pages))
    dw = DeviceWorkload(wl)
    dw.append_extend()
    out, lse = dw.extend()
    steps = wl.spec.decode_steps
    dec, dec_l = [], []
    for step in range(steps):
        rng = wl.decode_ranges(step)
        pos = wl.seq_lens + step
        l = torch.empty((wl.num_tasks, wl.spec.num_q_heads), dtype=torch.float32, device="cuda")
        dec.append(dw.kv.decode_append(dev_bf16(wl.packed("q", rng)), dev_bf16(wl.packed("k", rng)),
                                       dev_bf16(wl.packed("v", rng)), pos + 1, lse=l))
        dec_l.append(l)
    torch.cuda.synchronize()
    got = torch.stack(dec, dim=1)      # [tasks, steps, Hq, d]
    got_l = torch.stack(dec_l, dim=1)  # [tasks, steps, Hq]
    ref, ref_l = {}, {}

    def keep(b, positions, o, l):
        assert list(positions) == [int(wl.seq_lens[b]) + s for s in range(steps)]
        ref[b], ref_l[b] = o, l

    def decode_positions(b):
        return [int(wl.seq_lens[b]) + s for s in range(steps)]

    _check_extend_all(wl, dw, out, lse, seed=8, extra_positions=decode_positions,
                      extra_check=keep)
    order = list(range(wl.num_tasks))
    assert_close(got.reshape(-1, *got.shape[2:]), np.concatenate([ref[b] for b in order]),
                 "long_horizon decode steps, all tasks")
    assert_lse(got_l.reshape(-1, got_l.shape[2]), np.concatenate([ref_l[b] for b in order]),
               "long_horizon decode steps, all tasks")
    for b in sample_tasks(wl, 4, seed=9):
        pool = oracle_task_pool(wl, b, int(wl.final_lens[b]))
        _check_written_slots(wl, dw, b, pool, int(wl.seq_lens[b]), int(wl.final_lens[b]),
                             "decode append")
    _check_append_pages(wl, dw, sample_tasks(wl, 2, seed=10), lambda b: int(wl.final_lens[b]))
    del dw, dec, out, lse
    _free()
