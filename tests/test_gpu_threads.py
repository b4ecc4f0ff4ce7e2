"""Two host threads calling the library at once (needs an MI355X).

Each thread has its own stream (default priority, as every stream here) and its own
workspaces, and runs extend, decode and an append into its own copy of the pool, 12
times over.  The library's only shared host state, the pinned staging ring, is guarded
by a mutex, and a work list is reused only after its copy completed; so every result
must equal, bit for bit, the same call made alone on the default stream."""
import threading

import numpy as np
import pytest
import torch

import paper_2608_10402_amd as tide
import workloads as W
from gpu_harness import DeviceWorkload, dev_bf16, log

_lib = tide._lib
pytestmark = pytest.mark.gpu


def test_two_threads_two_streams_match_serial():
    wl = W.make_workload(W.SPECS["agent_resume_7b"].shrunk(6, 8))
    dw = DeviceWorkload(wl)
    kv = dw.kv
    P, E, L = wl.prefix_lens, wl.extend_lens, wl.seq_lens
    k_new = dev_bf16(wl.packed("k", wl.extend_ranges()))
    v_new = dev_bf16(wl.packed("v", wl.extend_ranges()))
    q = dev_bf16(wl.packed("q", wl.extend_ranges()))
    last = torch.as_tensor((np.cumsum(E) - 1).astype(np.int64), device="cuda")
    qd = q[last].contiguous()
    prefix_pools = (kv.k_pool.clone(), kv.v_pool.clone())  # before the new tokens
    # serial reference, default stream
    kv.append(k_new, v_new, P, E)
    ref_ext = kv.extend(q, P, E)
    ref_dec = kv.decode(qd, L)
    torch.cuda.synchronize()
    ref_pools = (kv.k_pool.clone(), kv.v_pool.clone())

    ws_bytes = max(_lib.tide_workspace_size(_lib.TIDE_OP_EXTEND, P, E, kv.dims),
                   _lib.tide_workspace_size(_lib.TIDE_OP_KV_APPEND, P, E, kv.dims),
                   _lib.tide_workspace_size(_lib.TIDE_OP_DECODE, L, None, kv.dims))
    results, errors = {}, []

    def worker(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                ws_a = _lib.alloc_workspace(ws_bytes)
                ws_b = _lib.alloc_workspace(ws_bytes)
                kp, vp = prefix_pools[0].clone(), prefix_pools[1].clone()
                for rep in range(12):
                    out = torch.empty_like(q)
                    outd = torch.empty_like(qd)
                    _lib.tide_extend_attn(q, ref_pools[0], ref_pools[1], kv.block_table, P, E,
                                          kv.dims, out, None, ws_a, s)
                    _lib.tide_decode_attn(qd, ref_pools[0], ref_pools[1], kv.block_table, L,
                                          kv.dims, outd, None, 0, ws_b, s)
                    if rep == 5:
                        _lib.tide_kv_append(k_new, v_new, kp, vp, kv.block_table, P, E, kv.dims,
                                            ws_b, s)
                    results[(i, rep)] = (out, outd)
                s.synchronize()
                results[(i, "pools")] = (kp, vp)
        except Exception as e:  # reported by the main thread
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    bits = lambda t: t.view(torch.int16)
    for i in range(2):
        for rep in range(12):
            out, outd = results[(i, rep)]
            assert torch.equal(bits(out), bits(ref_ext)), (i, rep, "extend")
            assert torch.equal(bits(outd), bits(ref_dec)), (i, rep, "decode")
        kp, vp = results[(i, "pools")]
        assert torch.equal(bits(kp), bits(ref_pools[0])) and torch.equal(bits(vp), bits(ref_pools[1]))
    log("two threads x 12 rounds: extend, decode and append bit-identical to serial")
