"""Decode with the append of the decoded token fused in (tide_decode_append_attn).

The fused call must leave the pool and return the output of tide_kv_append of the
newest token followed by tide_decode_attn, bit for bit: the split that covers the newest
position uses the same values a pool load would have given it.  Checked against that
two-call sequence on a copy of the same pool, and against the fp64 oracle, for split
counts 0, 1 and 3 and for the positions where the newest token lands on a page edge.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_harness import (DeviceWorkload, assert_close, assert_lse, dev_bf16, host_bits, log,
                         oracle_pools)

pytestmark = pytest.mark.gpu
S = W.SPECS

def _newest_token_on_page0():
    """Task 0's newest token lands on physical page 0, and every task's context ends in
    the first page of its last 32-key step, so the second page of that step lies past
    the context.  Such pages are never read (a zero-range load), so no wave can bring a
    copy of page 0 into its CU's L1 before the fused append writes it."""
    wl = W.custom_workload(16, 4, 128, [40, 100, 7, 200, 0, 72, 136, 1000, 520], [1] * 9,
                           seed=24)
    assert ((wl.seq_lens % 32 >= 1) & (wl.seq_lens % 32 <= 16)).all()
    p = int(wl.block_table[0, (wl.seq_lens[0] - 1) // 16])
    perm = np.arange(wl.num_pages, dtype=np.int32)
    perm[p], perm[0] = 0, p
    return wl.remap_pages(perm)


# contexts (including the decoded token): 1 (the token is the whole context), 16 (last
# slot of the first page), 17 (first slot of the second page), 32, 33, 2049; GQA 1..16
CASES = {
    "newest_on_page0": _newest_token_on_page0,
    "resumed_decode_small": lambda: W.make_workload(S["resumed_decode"].shrunk(12, 16)),
    "edges_g4_d128": lambda: W.custom_workload(16, 4, 128, [0, 15, 16, 31, 32, 2048, 100],
                                               [1] * 7, seed=21),
    "edges_g16_d64": lambda: W.custom_workload(16, 1, 64, [0, 15, 16, 500], [1] * 4, seed=22),
    "g1_d128": lambda: W.custom_workload(4, 4, 128, [47, 3, 300], [1] * 3, seed=23),
    # d = 64 with 2,048+ work items, so the 8-wave workgroups of large launches run
    "d64_2k_items": lambda: W.custom_workload(16, 2, 64, [2000 + 7 * (i % 40) for i in range(256)],
                                              [1] * 256, seed=25),
}


@pytest.fixture(scope="module", params=sorted(CASES))
def dcase(request):
    name = request.param
    log("fused append+decode workload %s" % name)
    wl = CASES[name]()
    assert (wl.extend_lens == 1).all()
    kp, vp = oracle_pools(wl)
    q = wl.packed("q", wl.extend_ranges())
    ref, ref_lse = oracle.decode(q, kp, vp, wl.block_table, wl.seq_lens, wl.spec.num_q_heads,
                                 wl.sm_scale)
    return name, wl, q, ref, ref_lse


@pytest.mark.parametrize("splits", [0, 1, 3])
def test_fused_equals_append_then_decode(dcase, splits):
    name, wl, q, ref, ref_lse = dcase
    a = DeviceWorkload(wl)  # prefix appended
    b = DeviceWorkload(wl)
    kn = dev_bf16(wl.packed("k", wl.extend_ranges()))
    vn = dev_bf16(wl.packed("v", wl.extend_ranges()))
    qd = dev_bf16(q)
    la = torch.empty((q.shape[0], q.shape[1]), dtype=torch.float32, device="cuda")
    lb = torch.empty_like(la)
    a.kv.append(kn, vn, wl.prefix_lens, wl.extend_lens)
    out_a = a.kv.decode(qd, wl.seq_lens, num_splits=splits, lse=la)
    out_b = b.kv.decode_append(qd, kn, vn, wl.seq_lens, num_splits=splits, lse=lb)
    torch.cuda.synchronize()
    assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16)), name
    assert torch.equal(la, lb), name
    assert np.array_equal(host_bits(a.kv.k_pool), host_bits(b.kv.k_pool)), name
    assert np.array_equal(host_bits(a.kv.v_pool), host_bits(b.kv.v_pool)), name
    assert_close(out_b, ref, "%s fused decode splits=%d" % (name, splits))
    assert_lse(lb, ref_lse, "%s fused decode splits=%d" % (name, splits))


def test_fused_pool_matches_oracle_image(dcase):
    """After the fused call the whole pool is the oracle's append image, untouched bytes
    (NaN canaries) included."""
    name, wl, q, ref, ref_lse = dcase
    b = DeviceWorkload(wl)
    kn = dev_bf16(wl.packed("k", wl.extend_ranges()))
    vn = dev_bf16(wl.packed("v", wl.extend_ranges()))
    b.kv.decode_append(dev_bf16(q), kn, vn, wl.seq_lens)
    torch.cuda.synchronize()
    kp, vp = oracle_pools(wl)
    assert np.array_equal(host_bits(b.kv.k_pool), kp), name
    assert np.array_equal(host_bits(b.kv.v_pool), vp), name


def test_fused_fullsize_resumed_decode():
    wl = W.make_workload("resumed_decode")
    a = DeviceWorkload(wl)
    b = DeviceWorkload(wl)
    kn = dev_bf16(wl.packed("k", wl.extend_ranges()))
    vn = dev_bf16(wl.packed("v", wl.extend_ranges()))
    qd = dev_bf16(wl.packed("q", wl.extend_ranges()))
    a.kv.append(kn, vn, wl.prefix_lens, wl.extend_lens)
    out_a = a.kv.decode(qd, wl.seq_lens)
    out_b = b.kv.decode_append(qd, kn, vn, wl.seq_lens)
    torch.cuda.synchronize()
    assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16))
    assert torch.equal(a.kv.k_pool.view(torch.int16), b.kv.k_pool.view(torch.int16))
    assert torch.equal(a.kv.v_pool.view(torch.int16), b.kv.v_pool.view(torch.int16))
