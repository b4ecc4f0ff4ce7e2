"""Split-KV extend and prefill against the fp64 oracle (needs an MI355X).

A call with few work items runs split-KV: long token blocks are cut into key-tile
chunks whose fp32 partials a merge kernel combines.  The plan is chosen from the lengths;
TIDE_EXTEND_SPLIT forces either plan so that both are checked on the same inputs:
against the oracle row by row (output and LSE), against each other, and for bitwise
repeatability.  Cases: one-task calls with long retained prefixes (the shape that
triggers the split), GQA groups 1, 7 and 16, head_dim 64 and 128, a fresh prefill whose
diagonal falls inside a chunk, ragged blocks and tiles, outlier keys that force running-max
rescales inside a chunk, and several tasks of which some are split and some are not.
"""
import pytest
import torch

import oracle
import workloads as W
from gpu_harness import DeviceWorkload, assert_close, assert_lse, log, oracle_pools

pytestmark = pytest.mark.gpu

CASES = {
    "g7_one_task": lambda: W.custom_workload(28, 4, 128, [5000], [300], seed=5),
    "g1_d64": lambda: W.custom_workload(8, 8, 64, [3000, 0], [70, 1], seed=6),
    "g16_d128": lambda: W.custom_workload(16, 1, 128, [2500], [40], seed=7),
    "g4_outliers": lambda: W.custom_workload(16, 4, 128, [4000], [100], seed=8, outlier_frac=0.1),
    "g7_fresh": lambda: W.custom_workload(28, 4, 128, [0], [1500], seed=9),
    "g8_mixed_d64": lambda: W.custom_workload(32, 4, 64, [6000, 17, 900, 0], [33, 200, 1, 65],
                                              seed=10),
}


@pytest.fixture(scope="module", params=sorted(CASES))
def scase(request):
    name = request.param
    wl = CASES[name]()
    log("split case %s: P=%s E=%s Hq=%d Hkv=%d d=%d" % (
        name, wl.prefix_lens.tolist(), wl.extend_lens.tolist(), wl.spec.num_q_heads,
        wl.spec.num_kv_heads, wl.spec.head_dim))
    dw = DeviceWorkload(wl)
    dw.append_extend()
    kp, vp = oracle_pools(wl)
    torch.cuda.synchronize()
    return name, wl, dw, kp, vp


def _run(monkeypatch, mode, fn):
    monkeypatch.setenv("TIDE_EXTEND_SPLIT", mode)
    out, lse = fn()
    torch.cuda.synchronize()
    return out, lse


@pytest.mark.parametrize("mode", ["1", "0"])
def test_extend_against_oracle(scase, mode, monkeypatch):
    name, wl, dw, kp, vp = scase
    out, lse = _run(monkeypatch, mode, dw.extend)
    ref, ref_lse = oracle.extend(wl.packed("q", wl.extend_ranges()), kp, vp, wl.block_table,
                                 wl.prefix_lens, wl.extend_lens, wl.spec.num_q_heads,
                                 wl.sm_scale)
    assert_close(out, ref, "%s extend (split=%s)" % (name, mode))
    assert_lse(lse, ref_lse, "%s extend (split=%s)" % (name, mode))


@pytest.mark.parametrize("mode", ["1", "0"])
def test_prefill_against_oracle(scase, mode, monkeypatch):
    name, wl, dw, kp, vp = scase
    out, lse = _run(monkeypatch, mode, dw.prefill)
    ref, ref_lse = oracle.prefill(wl.packed("q", wl.full_ranges()), kp, vp, wl.block_table,
                                  wl.seq_lens, wl.spec.num_q_heads, wl.sm_scale)
    assert_close(out, ref, "%s prefill (split=%s)" % (name, mode))
    assert_lse(lse, ref_lse, "%s prefill (split=%s)" % (name, mode))


def test_split_matches_plain_and_repeats(scase, monkeypatch):
    """The two plans agree to bf16 rounding, and each is bitwise repeatable."""
    name, wl, dw, kp, vp = scase
    o1, l1 = _run(monkeypatch, "1", dw.extend)
    o1b, l1b = _run(monkeypatch, "1", dw.extend)
    o0, l0 = _run(monkeypatch, "0", dw.extend)
    assert torch.equal(o1, o1b) and torch.equal(l1, l1b), name
    d = (o1.float() - o0.float()).abs()
    log("%s split vs plain: max %.3g mean %.3g, lse max %.3g" % (
        name, d.max().item(), d.mean().item(), (l1 - l0).abs().max().item()))
    assert d.max().item() <= 2e-2 and d.mean().item() <= 2e-3, name
    assert (l1 - l0).abs().max().item() <= 1e-3, name


def test_split_without_lse(scase, monkeypatch):
    """Without an LSE output the merge skips the exact sums; the rows are unchanged."""
    name, wl, dw, kp, vp = scase
    with_l, _ = _run(monkeypatch, "1", dw.extend)
    without, _ = _run(monkeypatch, "1", lambda: dw.extend(lse=False))
    assert torch.equal(with_l, without), name
