"""Extend attention with the KV-append fused in (tide_extend_append_attn).

The fused call must leave the pool and return the output (and LSE) of tide_kv_append of
the new tokens followed by tide_extend_attn, bit for bit: the attention reads keys at or
past each prefix straight from the new rows, which hold the bits the append would have
written.  Checked against that two-call sequence on a second copy of the same pool --
outputs, LSE, and the whole K and V pools including the untouched NaN canaries and the
stale slots of a pruned context -- under the planner's choice and with the split-KV plan
forced on and off, and against the fp64 oracle.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_harness import DeviceWorkload, assert_close, assert_lse, dev_bf16, host_bits, log, oracle_pools
from test_gpu_parity import EXTEND_WORKLOADS

pytestmark = pytest.mark.gpu

CASES = dict(EXTEND_WORKLOADS)
CASES["agent_resume_7b_one_task"] = lambda: W.custom_workload(28, 4, 128, [9000], [700], seed=6)


@pytest.fixture(scope="module", params=sorted(CASES))
def case(request):
    name = request.param
    wl = CASES[name]()
    log("fused append+extend workload %s: P=%s E=%s" % (name, wl.prefix_lens.tolist()[:6],
                                                       wl.extend_lens.tolist()[:6]))
    kp, vp = oracle_pools(wl)
    q = wl.packed("q", wl.extend_ranges())
    ref, ref_lse = oracle.extend(q, kp, vp, wl.block_table, wl.prefix_lens, wl.extend_lens,
                                 wl.spec.num_q_heads, wl.sm_scale)
    return name, wl, q, ref, ref_lse, kp, vp


@pytest.mark.parametrize("mode", [None, "0", "1"])
def test_fused_equals_append_then_extend(case, mode):
    name, wl, q, ref, ref_lse, kp, vp = case
    a = DeviceWorkload(wl)  # prefix (and any pre-prune context) appended
    b = DeviceWorkload(wl)
    kn = dev_bf16(wl.packed("k", wl.extend_ranges()))
    vn = dev_bf16(wl.packed("v", wl.extend_ranges()))
    qd = dev_bf16(q)
    rows, hq = q.shape[0], q.shape[1]
    la = torch.empty((rows, hq), dtype=torch.float32, device="cuda")
    lb = torch.full_like(la, float("nan"))
    saved = os.environ.get("TIDE_EXTEND_SPLIT")
    try:
        if mode is None:
            os.environ.pop("TIDE_EXTEND_SPLIT", None)
        else:
            os.environ["TIDE_EXTEND_SPLIT"] = mode
        a.kv.append(kn, vn, wl.prefix_lens, wl.extend_lens)
        out_a = a.kv.extend(qd, wl.prefix_lens, wl.extend_lens, lse=la)
        out_b = torch.full_like(out_a, float("nan"))
        b.kv.extend_append(qd, kn, vn, wl.prefix_lens, wl.extend_lens, out=out_b, lse=lb)
        torch.cuda.synchronize()
    finally:
        if saved is None:
            os.environ.pop("TIDE_EXTEND_SPLIT", None)
        else:
            os.environ["TIDE_EXTEND_SPLIT"] = saved
    what = "%s fused split=%s" % (name, mode)
    assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16)), what
    assert torch.equal(la, lb), what
    assert np.array_equal(host_bits(a.kv.k_pool), host_bits(b.kv.k_pool)), what
    assert np.array_equal(host_bits(a.kv.v_pool), host_bits(b.kv.v_pool)), what
    assert_close(out_b, ref, what)
    assert_lse(lb, ref_lse, what)


def test_fused_pool_matches_oracle_image(case):
    """After the fused call the whole pool is the oracle's append image (pre-prune context
    and canaries included)."""
    name, wl, q, ref, ref_lse, kp, vp = case
    b = DeviceWorkload(wl)
    kn = dev_bf16(wl.packed("k", wl.extend_ranges()))
    vn = dev_bf16(wl.packed("v", wl.extend_ranges()))
    b.kv.extend_append(dev_bf16(q), kn, vn, wl.prefix_lens, wl.extend_lens)
    torch.cuda.synchronize()
    assert np.array_equal(host_bits(b.kv.k_pool), kp), name
    assert np.array_equal(host_bits(b.kv.v_pool), vp), name


def test_fused_fullsize_agent_resume():
    """agent_resume_7b at full size: fused == append + extend, bit for bit."""
    wl = W.make_workload("agent_resume_7b")
    a = DeviceWorkload(wl)
    b = DeviceWorkload(wl)
    kn = dev_bf16(wl.packed("k", wl.extend_ranges()))
    vn = dev_bf16(wl.packed("v", wl.extend_ranges()))
    qd = dev_bf16(wl.packed("q", wl.extend_ranges()))
    a.kv.append(kn, vn, wl.prefix_lens, wl.extend_lens)
    out_a = a.kv.extend(qd, wl.prefix_lens, wl.extend_lens)
    out_b = b.kv.extend_append(qd, kn, vn, wl.prefix_lens, wl.extend_lens)
    torch.cuda.synchronize()
    assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16))
    assert torch.equal(a.kv.k_pool.view(torch.int16), b.kv.k_pool.view(torch.int16))
    assert torch.equal(a.kv.v_pool.view(torch.int16), b.kv.v_pool.view(torch.int16))
