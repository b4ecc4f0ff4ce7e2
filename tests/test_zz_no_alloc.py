"""Decode without allocation (tide_decode_attn_noalloc), called through the C ABI.

Two calls in a row share the library's static device scratch, the second with a smaller
input, then the first again: the scratch keeps the last call's contents, so each call
must clear what it relies on.  Every output and LSE equals tide_decode_attn's on the same
arguments bit for bit (same plan, same kernels), and matches the fp64 oracle within the
bf16 tolerance.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_10402_amd as tide
import workloads as W
from gpu_harness import DeviceWorkload, assert_close, assert_lse, dev_bf16, log, oracle_pools

pytestmark = pytest.mark.gpu
S = W.SPECS

CASES = [
    # (name, workload factory, num_splits)
    ("resumed_decode/4", lambda: W.make_workload(S["resumed_decode"].shrunk(64, 4)), 0),
    ("small_g4_d128", lambda: W.custom_workload(16, 4, 128, [0, 15, 16, 31, 300], [1] * 5,
                                                seed=31), 0),
    ("resumed_decode/4 again", lambda: W.make_workload(S["resumed_decode"].shrunk(64, 4)), 3),
    ("small_g16_d64", lambda: W.custom_workload(16, 1, 64, [7, 100, 2047], [1] * 3, seed=32), 0),
]


def _run(name, make, splits):
    wl = make()
    assert (wl.extend_lens == 1).all()
    log("noalloc decode %s: %d tasks, context %d..%d, splits %d"
        % (name, wl.num_tasks, wl.seq_lens.min(), wl.seq_lens.max(), splits))
    need = tide.tide_workspace_size(tide.TIDE_OP_DECODE, wl.seq_lens, None,
                                    tide.make_dims(wl.spec.num_q_heads, wl.spec.num_kv_heads,
                                                   wl.spec.head_dim, wl.sm_scale), splits)
    assert need <= tide.NOALLOC_SCRATCH_BYTES
    dw = DeviceWorkload(wl)
    dw.append_extend()  # the decoded token's own K/V
    q = wl.packed("q", wl.extend_ranges())
    qd = dev_bf16(q)
    h = wl.spec.num_q_heads
    l_ref = torch.empty((wl.num_tasks, h), dtype=torch.float32, device="cuda")
    l_na = torch.full_like(l_ref, float("nan"))
    out_ref = dw.kv.decode(qd, wl.seq_lens, num_splits=splits, lse=l_ref)
    out_na = torch.full_like(out_ref, float("nan"))
    dw.kv.decode_noalloc(qd, wl.seq_lens, num_splits=splits, out=out_na, lse=l_na)
    torch.cuda.synchronize()
    assert torch.equal(out_na.view(torch.int16), out_ref.view(torch.int16)), name
    assert torch.equal(l_na, l_ref), name
    kp, vp = oracle_pools(wl)
    ref, ref_lse = oracle.decode(q, kp, vp, wl.block_table, wl.seq_lens, h, wl.sm_scale)
    assert_close(out_na, ref, "noalloc decode %s" % name)
    assert_lse(l_na, ref_lse, "noalloc decode %s" % name)


def test_noalloc_decode_calls_in_a_row():
    for name, make, splits in CASES:
        _run(name, make, splits)
