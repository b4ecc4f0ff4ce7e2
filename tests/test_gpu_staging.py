"""Reuse of the pinned staging slots that carry each call's work list (needs an MI355X).

A call reuses one of the library's 16 staging slots only after the previous copy out of
it has read it: each copy workgroup sets a flag that the host checks, waiting a bounded
time and then synchronising the device.  Here a spin kernel holds the stream while 40
calls are queued behind it, so from the 17th call on every slot the host wants is still
unread; with TIDE_STAGING_WAIT_US=0 each such reuse takes the fallback at once.  Every
result must equal, bit for bit, the same call made on an idle device."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_harness import DeviceWorkload, dev_bf16

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("wait_us", ["0", None])
def test_slot_reuse_behind_a_busy_stream(monkeypatch, wait_us):
    wl = W.make_workload(W.SPECS["agent_resume_7b"].shrunk(6, 8))
    dw = DeviceWorkload(wl)
    dw.append_extend()
    kv = dw.kv
    P, E, L = wl.prefix_lens, wl.extend_lens, wl.seq_lens
    q = dev_bf16(wl.packed("q", wl.extend_ranges()))
    last = torch.as_tensor((np.cumsum(E) - 1).astype(np.int64), device="cuda")
    qd = q[last].contiguous()
    ref_e = kv.extend(q, P, E)
    ref_d = kv.decode(qd, L)
    torch.cuda.synchronize()

    if wait_us is not None:
        monkeypatch.setenv("TIDE_STAGING_WAIT_US", wait_us)
    torch.cuda._sleep(50_000_000)  # a bounded spin kernel (tens of ms) ahead of the calls
    outs = [(kv.extend(q, P, E), kv.decode(qd, L)) for _ in range(20)]
    torch.cuda.synchronize()
    for i, (oe, od) in enumerate(outs):
        assert torch.equal(oe.view(torch.int16), ref_e.view(torch.int16)), i
        assert torch.equal(od.view(torch.int16), ref_d.view(torch.int16)), i
