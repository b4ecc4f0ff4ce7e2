"""GPU parity against the fp64 oracle through the C ABI (needs an MI355X).

Sizes: the tiny workload at full size, the others shrunk so the oracle computes every
row in seconds while still spanning many 64-key tiles, several token blocks per task and
ragged page/tile tails; plus explicit edge cases (empty extends, fresh tasks, single
keys, page and tile boundaries, GQA groups 1..16, head_dim 64 and 128, resumes written
over a pruned context).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_harness import (DeviceWorkload, assert_close, assert_lse, dev_bf16, host_bits,
                         log, oracle_pools)

pytestmark = pytest.mark.gpu

S = W.SPECS
EXTEND_WORKLOADS = {
    "tiny_extend": lambda: W.make_workload(S["tiny_extend"]),
    "agent_resume_7b_small": lambda: W.make_workload(S["agent_resume_7b"].shrunk(6, 8)),
    "multimodal_resume_small": lambda: W.make_workload(S["multimodal_resume"].shrunk(4, 16)),
    "long_horizon_small": lambda: W.make_workload(S["long_horizon"].shrunk(3, 48)),
    "g1_boundaries": lambda: W.custom_workload(8, 8, 128, [0, 16, 63, 64, 65], [1, 0, 1, 63, 130]),
    "g16_d64": lambda: W.custom_workload(32, 2, 64, [0, 200, 15], [300, 1, 17], seed=1),
    "g3_d64": lambda: W.custom_workload(12, 4, 64, [1, 127, 0], [127, 1, 0], seed=2),
    "g4_long": lambda: W.custom_workload(4, 1, 128, [1000], [37], seed=3),
    "g8_outliers": lambda: W.custom_workload(16, 2, 128, [300, 5], [90, 200], seed=4,
                                             outlier_frac=0.1),
    # sliding-window prune resume: the new rows are written over pages that still hold the
    # pre-prune context, which must neither leak into the attention nor survive in a
    # written slot; an empty prompt, page-aligned prompts, a resumed end that lands on a
    # page boundary (task 3: 64 + 176) and ragged ends inside a stale page
    "prune_resume_small": lambda: W.make_workload(S["multimodal_prune_resume"].shrunk(4, 16)),
    "prune_edges_d64": lambda: W.custom_prune_workload(
        16, 4, 64, [0, 16, 37, 64],
        [[0] * 10, [3, 40, 0, 7, 1, 12, 33, 2, 9, 5], [5] * 10, [2] + [1] * 9],
        image_tokens=33, seed=2),
}


@pytest.fixture(scope="module", params=sorted(EXTEND_WORKLOADS))
def case(request):
    name = request.param
    log("workload %s" % name)
    wl = EXTEND_WORKLOADS[name]()
    log("  P=%s E=%s Hq=%d Hkv=%d d=%d pages=%d" % (
        wl.prefix_lens.tolist()[:8], wl.extend_lens.tolist()[:8], wl.spec.num_q_heads,
        wl.spec.num_kv_heads, wl.spec.head_dim, wl.num_pages))
    dw = DeviceWorkload(wl)
    dw.append_extend()
    kp, vp = oracle_pools(wl)
    torch.cuda.synchronize()
    return name, wl, dw, kp, vp


def test_append_bitexact(case):
    name, wl, dw, kp, vp = case
    gk = host_bits(dw.kv.k_pool)
    gv = host_bits(dw.kv.v_pool)
    assert np.array_equal(gk, kp), "%s: K pool differs from the oracle image" % name
    assert np.array_equal(gv, vp), "%s: V pool differs from the oracle image" % name


def test_extend_parity(case):
    name, wl, dw, kp, vp = case
    out, lse = dw.extend()
    q = wl.packed("q", wl.extend_ranges())
    ref, ref_lse = oracle.extend(q, kp, vp, wl.block_table, wl.prefix_lens, wl.extend_lens,
                                 wl.spec.num_q_heads, wl.sm_scale)
    assert_close(out, ref, "%s extend" % name)
    assert_lse(lse, ref_lse, "%s extend" % name)


def test_prefill_parity(case):
    name, wl, dw, kp, vp = case
    out, lse = dw.prefill()
    q = wl.packed("q", wl.full_ranges())
    ref, ref_lse = oracle.prefill(q, kp, vp, wl.block_table, wl.seq_lens, wl.spec.num_q_heads,
                                  wl.sm_scale)
    assert_close(out, ref, "%s prefill" % name)
    assert_lse(lse, ref_lse, "%s prefill" % name)


def test_extend_matches_prefill_rows(case):
    """Invariant (a) on the GPU: resume over the retained prefix == re-prefill rows."""
    name, wl, dw, kp, vp = case
    ext, _ = dw.extend(lse=False)
    full, _ = dw.prefill(lse=False)
    e = ext.float().cpu().numpy()
    f = full.float().cpu().numpy()
    row_e = row_f = 0
    for b in range(wl.num_tasks):
        p, n = int(wl.prefix_lens[b]), int(wl.extend_lens[b])
        d = np.abs(e[row_e:row_e + n] - f[row_f + p:row_f + p + n])
        assert d.size == 0 or d.max() <= 2e-2, (name, b, d.max())
        row_e += n
        row_f += p + n


def test_deterministic(case):
    name, wl, dw, kp, vp = case
    a, la = dw.extend()
    b, lb = dw.extend()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert torch.equal(la, lb)


def test_page_placement_invariance():
    """Moving physical pages (and remapping the table) changes no output bit."""
    wl = W.make_workload(S["agent_resume_7b"].shrunk(4, 16))
    perm = np.random.default_rng(7).permutation(wl.num_pages).astype(np.int32)
    outs = []
    for w in (wl, wl.remap_pages(perm)):
        dw = DeviceWorkload(w)
        dw.append_extend()
        o, l = dw.extend()
        outs.append((o.view(torch.int16).cpu(), l.cpu()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


# ---- decode -------------------------------------------------------------------------------
DECODE_WORKLOADS = {
    "resumed_decode_small": lambda: W.make_workload(S["resumed_decode"].shrunk(16, 6)),
    "decode_edges_g8": lambda: W.custom_workload(32, 4, 128, [0, 15, 16, 31, 32, 2047, 2048, 700],
                                                 [1] * 8, seed=5),
    "decode_g16_d64": lambda: W.custom_workload(16, 1, 64, [0, 100, 999], [1, 1, 1], seed=6),
    "decode_g1": lambda: W.custom_workload(4, 4, 128, [3000, 1], [1, 1], seed=7),
    # d = 64 with 2,048+ work items, so the 8-wave workgroups of large launches run
    "decode_d64_2k_items": lambda: W.custom_workload(16, 2, 64,
                                                     [2000 + 7 * (i % 40) for i in range(256)],
                                                     [1] * 256, seed=8),
}


@pytest.fixture(scope="module", params=sorted(DECODE_WORKLOADS))
def dcase(request):
    name = request.param
    log("decode workload %s" % name)
    wl = DECODE_WORKLOADS[name]()
    dw = DeviceWorkload(wl)
    dw.append_extend()  # the token being decoded is appended first
    kp, vp = oracle_pools(wl)
    q = wl.packed("q", wl.extend_ranges())  # one row per task
    ref, ref_lse = oracle.decode(q, kp, vp, wl.block_table, wl.seq_lens, wl.spec.num_q_heads,
                                 wl.sm_scale)
    torch.cuda.synchronize()
    return name, wl, dw, q, ref, ref_lse


@pytest.mark.parametrize("splits", [0, 1, 2, 7, 64, 100])
def test_decode_parity(dcase, splits):
    name, wl, dw, q, ref, ref_lse = dcase
    qd = dev_bf16(q)
    lse = torch.empty((q.shape[0], q.shape[1]), dtype=torch.float32, device="cuda")
    out = dw.kv.decode(qd, wl.seq_lens, num_splits=splits, lse=lse)
    assert_close(out, ref, "%s decode splits=%d" % (name, splits))
    assert_lse(lse, ref_lse, "%s decode splits=%d" % (name, splits))


def test_decode_matches_extend_e1(dcase):
    name, wl, dw, q, ref, ref_lse = dcase
    qd = dev_bf16(q)
    a = dw.kv.decode(qd, wl.seq_lens).float()
    b = dw.kv.extend(qd, wl.prefix_lens, wl.extend_lens).float()
    assert (a - b).abs().max().item() <= 2e-2


def test_long_horizon_sequence():
    """Append the resumed tokens, extend, then 8 rounds of (append one token, decode)."""
    wl = W.make_workload(S["long_horizon"].shrunk(3, 96))
    dw = DeviceWorkload(wl)
    dw.append_extend()
    out, _ = dw.extend(lse=False)
    kp, vp = oracle_pools(wl)
    ref, _ = oracle.extend(wl.packed("q", wl.extend_ranges()), kp, vp, wl.block_table,
                           wl.prefix_lens, wl.extend_lens, wl.spec.num_q_heads, wl.sm_scale)
    assert_close(out, ref, "long_horizon extend")
    for step in range(wl.spec.decode_steps):
        pos = wl.seq_lens + step
        rng = wl.decode_ranges(step)
        kn, vn = wl.packed("k", rng), wl.packed("v", rng)
        one = np.ones(wl.num_tasks, np.int32)
        dw.kv.append(dev_bf16(kn), dev_bf16(vn), pos, one)
        oracle.kv_append(kn, vn, kp, vp, wl.block_table, pos, one)
        q = wl.packed("q", rng)
        o = dw.kv.decode(dev_bf16(q), pos + 1)
        r, _ = oracle.decode(q, kp, vp, wl.block_table, pos + 1, wl.spec.num_q_heads, wl.sm_scale)
        assert_close(o, r, "long_horizon decode step %d" % step)
    torch.cuda.synchronize()
    assert np.array_equal(host_bits(dw.kv.k_pool), kp)
    assert np.array_equal(host_bits(dw.kv.v_pool), vp)


@pytest.mark.parametrize("splits", [0, 1, 2, 3, 40])
def test_decode_every_row_merged_once(splits):
    """Every decode row is written exactly by one of: the task's only split (1 split),
    the split that finishes its (task, kv head) last (few splits per task: 2, 3), or the
    merge kernel (many: 40, and the automatic plan at this size).  Outputs and LSE start
    as NaN on every call, so a row nobody wrote shows; repeated calls are bit-identical
    (merges sum in split order, whichever split arrives last) and match the oracle.  64
    tasks of mixed lengths spread the splits of one task over many CUs and XCDs."""
    rng = np.random.default_rng(31)
    prefix = [int(x) for x in rng.integers(0, 5000, size=64)]
    prefix[:4] = [0, 15, 31, 4095]
    wl = W.custom_workload(28, 4, 128, prefix, [1] * 64, seed=11)
    dw = DeviceWorkload(wl)
    dw.append_extend()
    kp, vp = oracle_pools(wl)
    q = wl.packed("q", wl.extend_ranges())
    ref, ref_lse = oracle.decode(q, kp, vp, wl.block_table, wl.seq_lens, wl.spec.num_q_heads,
                                 wl.sm_scale)
    qd = dev_bf16(q)
    outs = []
    for _ in range(3):
        out = torch.full_like(qd, float("nan"))
        lse = torch.full((q.shape[0], q.shape[1]), float("nan"), dtype=torch.float32, device="cuda")
        dw.kv.decode(qd, wl.seq_lens, num_splits=splits, out=out, lse=lse)
        torch.cuda.synchronize()
        assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
        outs.append((out, lse))
    assert_close(outs[0][0], ref, "decode merged in kernel, splits=%d" % splits)
    assert_lse(outs[0][1], ref_lse, "decode merged in kernel, splits=%d" % splits)
    for o, l in outs[1:]:
        assert torch.equal(o.view(torch.int16), outs[0][0].view(torch.int16))
        assert torch.equal(l, outs[0][1])
