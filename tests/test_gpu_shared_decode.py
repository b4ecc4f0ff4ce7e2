"""Shared-prefix (GRPO group) decode on the GPU.

tide_decode_attn_shared must return what tide_decode_attn returns: decode attention of
each trajectory over its whole context.  Only how the shared prompt pages are read
differs (once per group of up to 16 / G trajectories).  Checked against the fp64 oracle
and against plain decode, on small and edge-case groups and on the full-size workload.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_harness import (DeviceWorkload, assert_close, assert_lse, dev_bf16, log, oracle_pools,
                         oracle_task_rows, sample_tasks)

pytestmark = pytest.mark.gpu
S = W.SPECS

# groups of 1, 3, 8, 17 and 2 trajectories (17 > 16 / G = 4: split into several items),
# nothing shared, one page shared, long prompts, and trajectories whose whole context but
# the decoded token is the shared prompt (own length 1)
MIXED_OWN = [5] + [1, 7, 40] + [33, 1, 2, 900, 64, 17, 300, 5] + list(range(1, 18)) + [1, 2000]
WORKLOADS = {
    "grpo_small": lambda: W.make_workload(S["grpo_group_decode"].shrunk(24, 8)),
    "groups_mixed_g4": lambda: W.custom_group_workload(32, 8, 128, [1, 3, 8, 17, 2],
                                                       [0, 16, 1024, 160, 96], MIXED_OWN, seed=3),
    "groups_g16_d64": lambda: W.custom_group_workload(16, 1, 64, [3, 2], [512, 32],
                                                      [1, 20, 300, 1, 5], seed=4),
    "groups_g1_16wide": lambda: W.custom_group_workload(4, 4, 128, [16, 5], [2048, 0],
                                                        [1] * 8 + [3] * 8 + [100] * 5, seed=5),
    # d = 64 with 2,048+ work items, so the 8-wave workgroups of large launches run
    "groups_d64_2k_items": lambda: W.custom_group_workload(
        16, 2, 64, [8] * 64, [1024] * 64, [1 + (37 * i) % 1500 for i in range(512)], seed=6),
}


@pytest.fixture(scope="module", params=sorted(WORKLOADS))
def gcase(request):
    name = request.param
    log("shared-prefix decode workload %s" % name)
    wl = WORKLOADS[name]()
    dw = DeviceWorkload(wl)
    dw.append_extend()  # each trajectory's decoded token
    kp, vp = oracle_pools(wl)
    q = wl.packed("q", wl.extend_ranges())
    ref, ref_lse = oracle.decode(q, kp, vp, wl.block_table, wl.seq_lens, wl.spec.num_q_heads,
                                 wl.sm_scale)
    torch.cuda.synchronize()
    return name, wl, dw, q, ref, ref_lse


@pytest.mark.parametrize("splits", [0, 1, 3])
def test_shared_decode_parity(gcase, splits):
    name, wl, dw, q, ref, ref_lse = gcase
    lse = torch.empty((q.shape[0], q.shape[1]), dtype=torch.float32, device="cuda")
    out = dw.kv.decode_shared(dev_bf16(q), wl.seq_lens, wl.group_start, wl.shared_lens,
                              num_splits=splits, lse=lse)
    assert_close(out, ref, "%s shared decode splits=%d" % (name, splits))
    assert_lse(lse, ref_lse, "%s shared decode splits=%d" % (name, splits))


def test_shared_matches_plain_decode(gcase):
    name, wl, dw, q, ref, ref_lse = gcase
    qd = dev_bf16(q)
    a = dw.kv.decode(qd, wl.seq_lens).float()
    b = dw.kv.decode_shared(qd, wl.seq_lens, wl.group_start, wl.shared_lens).float()
    diff = (a - b).abs().max().item()
    log("%s shared vs plain decode: max abs diff %.3e" % (name, diff))
    assert diff <= 1e-2


def test_shared_decode_fullsize():
    """grpo_group_decode at full size: every trajectory against plain decode, eight
    trajectories (the longest, the shortest, seeded others) against the oracle."""
    wl = W.make_workload("grpo_group_decode")
    dw = DeviceWorkload(wl)
    dw.append_extend()
    q = wl.packed("q", wl.extend_ranges())
    qd = dev_bf16(q)
    plain = dw.kv.decode(qd, wl.seq_lens)
    shared = dw.kv.decode_shared(qd, wl.seq_lens, wl.group_start, wl.shared_lens)
    diff = (plain.float() - shared.float()).abs().max().item()
    log("grpo_group_decode shared vs plain: max abs diff %.3e" % diff)
    assert diff <= 1e-2
    for b in sample_tasks(wl, 8, seed=11):
        pos = int(wl.seq_lens[b]) - 1
        _, ref, _ = oracle_task_rows(wl, b, [pos], upto=pos + 1)
        assert_close(shared[b:b + 1], ref, "grpo_group_decode task %d" % b)
