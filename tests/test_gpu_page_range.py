"""Out-of-range page ids (needs an MI355X).

The ABI guarantees that a block-table entry outside [0, num_pages) is never dereferenced:
the attention kernels read it through a zero-range buffer descriptor (zeros, no memory
access), append writes nothing for it, and each sets an error flag in the workspace,
which TIDE_DEBUG_CHECKS=1 turns into TIDE_ERR_PAGE_RANGE.  Each
entry point is called with one bad entry (too large, then negative) in a page it reads or
writes -- extend under both the plain and the split-KV plan -- and must report the error;
the same calls on the valid table must not.
"""
import numpy as np
import pytest
import torch

from paper_2608_10402_amd import _lib
import workloads as W
from gpu_harness import DeviceWorkload, dev_bf16, log

pytestmark = pytest.mark.gpu


def _expect(fn, bad):
    if bad:
        with pytest.raises(_lib.TideError) as e:
            fn()
        assert e.value.status == _lib.TIDE_ERR_PAGE_RANGE
    else:
        fn()
    torch.cuda.synchronize()


@pytest.fixture(scope="module")
def setup():
    # task 1 has a long prefix, so that a lone task's extend takes the split-KV plan too
    wl = W.custom_workload(16, 4, 128, [300, 3000], [40, 5], seed=11)
    dw = DeviceWorkload(wl)
    dw.append_extend()
    torch.cuda.synchronize()
    return wl, dw


@pytest.mark.parametrize("bad_id", ["large", "negative"])
def test_attention_entry_points_report_bad_pages(setup, bad_id, monkeypatch):
    wl, dw = setup
    kv = dw.kv
    s = wl.spec
    good = wl.block_table.copy()
    bad = good.copy()
    bad[1, 10] = wl.num_pages + 7 if bad_id == "large" else -3  # a prefix page of task 1
    q_ext = dev_bf16(wl.packed("q", wl.extend_ranges()))
    q_full = dev_bf16(wl.packed("q", wl.full_ranges()))
    q_dec = q_ext[torch.as_tensor(np.cumsum(wl.extend_lens) - 1, device=q_ext.device)].contiguous()
    k_dec = torch.zeros((wl.num_tasks, s.num_kv_heads, s.head_dim), dtype=torch.bfloat16,
                        device=q_ext.device)
    monkeypatch.setenv("TIDE_DEBUG_CHECKS", "1")
    try:
        for table, is_bad in ((good, False), (bad, True)):
            kv.set_block_table(table)
            for mode in ("0", "1"):
                monkeypatch.setenv("TIDE_EXTEND_SPLIT", mode)
                _expect(lambda: kv.extend(q_ext, wl.prefix_lens, wl.extend_lens), is_bad)
            monkeypatch.delenv("TIDE_EXTEND_SPLIT")
            _expect(lambda: kv.prefill(q_full, wl.seq_lens), is_bad)
            _expect(lambda: kv.decode(q_dec, wl.seq_lens), is_bad)
            if not is_bad:
                continue
            # the fused call writes each task's position seq_len (inside its last mapped
            # page for these lengths) and reads the rest, page 10 of task 1 included
            _expect(lambda: kv.decode_append(q_dec, k_dec, k_dec,
                                             (wl.seq_lens + 1).astype(np.int32)), True)
        log("every attention entry point reported the %s page id" % bad_id)
    finally:
        kv.set_block_table(good)


def test_append_writes_nothing_for_a_bad_page(setup, monkeypatch):
    wl, dw = setup
    kv = dw.kv
    s = wl.spec
    b = 0
    last = int((wl.seq_lens[b] - 1) // 16)  # the page the next token of task 0 goes to
    bad = wl.block_table.copy()
    bad[b, last] = wl.num_pages + 1
    k_pool = kv.k_pool.clone()
    v_pool = kv.v_pool.clone()
    k_new = torch.ones((1, s.num_kv_heads, s.head_dim), dtype=torch.bfloat16, device=k_pool.device)
    monkeypatch.setenv("TIDE_DEBUG_CHECKS", "1")
    try:
        kv.set_block_table(bad[b:b + 1])
        _expect(lambda: kv.append(k_new, k_new, (wl.seq_lens[b:b + 1] - 1).astype(np.int32),
                                  np.ones(1, np.int32)), True)
        assert torch.equal(kv.k_pool.view(torch.int16), k_pool.view(torch.int16))
        assert torch.equal(kv.v_pool.view(torch.int16), v_pool.view(torch.int16))
    finally:
        kv.set_block_table(wl.block_table)


def test_shared_decode_reports_bad_pages(monkeypatch):
    wl = W.custom_group_workload(16, 4, 128, [4, 3], [256, 128], [40, 3, 17, 1, 90, 2, 33],
                                 seed=12)
    dw = DeviceWorkload(wl)
    torch.cuda.synchronize()
    q = dev_bf16(wl.packed("q", wl.extend_ranges()))
    bad = wl.block_table.copy()
    bad[0, 3] = -1  # a shared prompt page, read through the group's first task
    monkeypatch.setenv("TIDE_DEBUG_CHECKS", "1")
    dw.kv.decode_shared(q, wl.seq_lens, wl.group_start, wl.shared_lens)
    dw.kv.set_block_table(bad)
    _expect(lambda: dw.kv.decode_shared(q, wl.seq_lens, wl.group_start, wl.shared_lens), True)
