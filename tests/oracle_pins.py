"""Checks that tie the fp64 oracle to facts other than its own code.

Each pin takes a loaded oracle library (ctypes handle) so the same checks can be run
against deliberately broken builds of oracle.c (see test_oracle.py), proving that a
plausible mistake -- a dropped scale, a causal off-by-one, a wrong GQA map, a
transposed V layout, a wrong slot index, a wrong sign -- fails at least one of them.

Pins used:
  golden       hand-derived closed forms (tests/golden/closed_forms.txt)
  sdpa         torch.nn.functional.scaled_dot_product_attention in fp64 on dense,
               unpaged per-task tensors (an independent library implementation), with
               an explicit bottom-right causal mask
  uniform      Q = 0 gives equal weights: o = mean of visible v, lse = log(count);
               v[:, 0] = position makes o[0] = t/2 and catches causal off-by-ones
  constant_v   v rows all equal c gives o = c (the weights sum to 1)
  one_key      a single visible key gives o = v_0 exactly
  permutation  moving physical pages (and remapping the block table) changes nothing
  gqa_replica  replicating each kv head G times and running G = 1 changes nothing
  append       every appended element lands at (BT[b][p//16], p%16) and nothing else moves
"""
from __future__ import annotations

import math
import os

import numpy as np
import torch

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "closed_forms.txt")


# ---------------------------------------------------------------------------------------
# helpers (no attention arithmetic: conversions and data movement only)
def bf16_bits(x) -> np.ndarray:
    t = torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bits_to_f64(a) -> np.ndarray:
    a = np.asarray(a, dtype=np.uint16)
    return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def oracle_pools_for(wl: W.Workload, lib=None, upto: str = "seq"):
    """Oracle pool images holding every position of every task (prefix + extend),
    built with the oracle's own append: first the prefix rows, then the new rows.  For a
    prune resume the pre-prune context is appended after the prefix and before the new
    rows, which write over its start."""
    hkv, d = wl.spec.num_kv_heads, wl.spec.head_dim
    kp, vp = oracle.new_pools(wl.num_pages, hkv, d)
    zeros = np.zeros_like(wl.prefix_lens)
    oracle.kv_append(wl.packed("k", wl.prefix_ranges()), wl.packed("v", wl.prefix_ranges()),
                     kp, vp, wl.block_table, zeros, wl.prefix_lens, lib=lib)
    if wl.stale_lens is not None:
        oracle.kv_append(wl.stale_packed("k"), wl.stale_packed("v"), kp, vp, wl.block_table,
                         wl.prefix_lens, (wl.stale_lens - wl.prefix_lens).astype(np.int32),
                         lib=lib)
    oracle.kv_append(wl.packed("k", wl.extend_ranges()), wl.packed("v", wl.extend_ranges()),
                     kp, vp, wl.block_table, wl.prefix_lens, wl.extend_lens, lib=lib)
    return kp, vp


def parse_golden(path: str = GOLDEN):
    cases, cur = [], None
    with open(path) as f:
        for raw in f:
            line = raw.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "case":
                cur = {"name": tok[1], "k": {}, "v": {}, "q": {}, "o": {}, "lse": {}}
            elif tok[0] == "dims":
                cur["hq"], cur["hkv"], cur["d"] = int(tok[1]), int(tok[2]), int(tok[3])
                cur["scale"] = float(tok[4])
            elif tok[0] == "lens":
                cur["prefix"], cur["extend"] = int(tok[1]), int(tok[2])
            elif tok[0] in ("k", "v", "q", "o"):
                cur[tok[0]][(int(tok[1]), int(tok[2]))] = [float(x) for x in tok[3:]]
            elif tok[0] == "lse":
                cur["lse"][(int(tok[1]), int(tok[2]))] = float(tok[3])
            elif tok[0] == "end":
                cases.append(cur)
                cur = None
    return cases


# ---------------------------------------------------------------------------------------
def pin_golden(lib=None):
    for case in parse_golden():
        hq, hkv, d = case["hq"], case["hkv"], case["d"]
        p, e = case["prefix"], case["extend"]
        n = p + e
        k = np.zeros((n, hkv, d), np.float32)
        v = np.zeros((n, hkv, d), np.float32)
        for (pos, g), vals in case["k"].items():
            k[pos, g] = vals
        for (pos, g), vals in case["v"].items():
            v[pos, g] = vals
        q = np.zeros((e, hq, d), np.float32)
        for (r, h), vals in case["q"].items():
            q[r, h] = vals
        num_pages = 3
        bt = np.array([[2, 0]], np.int32)  # positions 0..15 live in physical page 2
        kp, vp = oracle.new_pools(num_pages, hkv, d)
        oracle.kv_append(bf16_bits(k), bf16_bits(v), kp, vp, bt, np.array([0], np.int32),
                         np.array([n], np.int32), lib=lib)
        out, lse = oracle.extend(bf16_bits(q), kp, vp, bt, np.array([p], np.int32),
                                 np.array([e], np.int32), hq, case["scale"], lib=lib)
        for (r, h), vals in case["o"].items():
            np.testing.assert_allclose(out[r, h], vals, rtol=0, atol=1e-13,
                                       err_msg="%s o[%d,%d]" % (case["name"], r, h))
        for (r, h), val in case["lse"].items():
            assert abs(lse[r, h] - val) < 1e-13, (case["name"], r, h, lse[r, h], val)


def _dense_sdpa(wl: W.Workload, b: int):
    """Reference output of task b's extend rows from torch SDPA on dense fp64 tensors."""
    p, e = int(wl.prefix_lens[b]), int(wl.extend_lens[b])
    L = p + e
    g = wl.spec.group
    q = torch.from_numpy(bits_to_f64(wl.q_rows(b, p, L))).permute(1, 0, 2)  # [Hq, E, d]
    k = torch.from_numpy(bits_to_f64(wl.k_rows(b, 0, L))).permute(1, 0, 2)  # [Hkv, L, d]
    v = torch.from_numpy(bits_to_f64(wl.v_rows(b, 0, L))).permute(1, 0, 2)
    k = k.repeat_interleave(g, dim=0).contiguous()
    v = v.repeat_interleave(g, dim=0).contiguous()
    rows = torch.arange(e).unsqueeze(1) + p
    cols = torch.arange(L).unsqueeze(0)
    mask = cols <= rows  # bottom-right aligned causal mask: row j sees keys 0..p+j
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask,
                                                         scale=wl.sm_scale)
    s = torch.matmul(q, k.transpose(1, 2)) * wl.sm_scale
    s = s.masked_fill(~mask, float("-inf"))
    lse = torch.logsumexp(s, dim=-1)
    return o.permute(1, 0, 2).numpy(), lse.transpose(0, 1).numpy()


def pin_sdpa(wl: W.Workload, lib=None, tol=1e-11):
    kp, vp = oracle_pools_for(wl, lib)
    q = wl.packed("q", wl.extend_ranges())
    out, lse = oracle.extend(q, kp, vp, wl.block_table, wl.prefix_lens, wl.extend_lens,
                             wl.spec.num_q_heads, wl.sm_scale, lib=lib)
    row = 0
    for b in range(wl.num_tasks):
        e = int(wl.extend_lens[b])
        if e == 0:
            continue
        ro, rl = _dense_sdpa(wl, b)
        np.testing.assert_allclose(out[row:row + e], ro, rtol=0, atol=tol, err_msg="task %d" % b)
        np.testing.assert_allclose(lse[row:row + e], rl, rtol=0, atol=tol, err_msg="lse %d" % b)
        row += e


def pin_uniform(lib=None):
    """Q = 0: every visible key has weight 1/(t+1).  v[p][0] = p, v[p][1] = -2p."""
    hq, hkv, d = 4, 2, 64
    prefix, extend = np.array([0, 21, 40], np.int32), np.array([19, 3, 24], np.int32)
    L = prefix + extend
    bt = np.array([[7, 3, 9, -1], [0, 5, -1, -1], [8, 1, 2, 4]], np.int32)
    kp, vp = oracle.new_pools(10, hkv, d)
    rng = np.random.default_rng(5)
    k = rng.standard_normal((int(L.sum()), hkv, d)).astype(np.float32)
    v = np.zeros((int(L.sum()), hkv, d), np.float32)
    at = 0
    for b in range(3):
        for pos in range(int(L[b])):
            v[at + pos, :, 0] = pos
            v[at + pos, :, 1] = -2 * pos
        at += int(L[b])
    oracle.kv_append(bf16_bits(k), bf16_bits(v), kp, vp, bt, np.zeros(3, np.int32), L, lib=lib)
    q = np.zeros((int(extend.sum()), hq, d), np.uint16)
    out, lse = oracle.extend(q, kp, vp, bt, prefix, extend, hq, 0.125, lib=lib)
    row = 0
    for b in range(3):
        for j in range(int(extend[b])):
            t = int(prefix[b]) + j
            assert np.allclose(out[row, :, 0], t / 2.0, rtol=0, atol=1e-12), (b, j, out[row, :, 0])
            assert np.allclose(out[row, :, 1], -float(t), rtol=0, atol=1e-12)
            assert np.allclose(out[row, :, 2:], 0.0, atol=0)
            assert np.allclose(lse[row], math.log(t + 1), rtol=0, atol=1e-12)
            row += 1


def pin_constant_v(lib=None):
    """v rows all equal to c: the output is c whatever the scores (weights sum to 1)."""
    hq, hkv, d = 6, 3, 64
    prefix, extend = np.array([50, 0], np.int32), np.array([30, 17], np.int32)
    L = prefix + extend
    need = [-(-int(x) // 16) for x in L]
    bt = np.full((2, max(need)), -1, np.int32)
    perm = np.random.default_rng(1).permutation(12).astype(np.int32)
    bt[0, :need[0]] = perm[:need[0]]
    bt[1, :need[1]] = perm[need[0]:need[0] + need[1]]
    kp, vp = oracle.new_pools(12, hkv, d)
    rng = np.random.default_rng(2)
    c = bf16_bits(rng.standard_normal((hkv, d)).astype(np.float32))
    k = bf16_bits(3 * rng.standard_normal((int(L.sum()), hkv, d)).astype(np.float32))
    v = np.broadcast_to(c, (int(L.sum()), hkv, d)).copy()
    oracle.kv_append(k, v, kp, vp, bt, np.zeros(2, np.int32), L, lib=lib)
    q = bf16_bits(rng.standard_normal((int(extend.sum()), hq, d)).astype(np.float32))
    out, _ = oracle.extend(q, kp, vp, bt, prefix, extend, hq, 1 / 8, lib=lib)
    expect = np.repeat(bits_to_f64(c), hq // hkv, axis=0)  # [hq, d]
    np.testing.assert_allclose(out, np.broadcast_to(expect, out.shape), rtol=1e-13, atol=1e-13)


def pin_one_key(lib=None):
    """A fresh task's first row sees only its own key: o = v_0, lse = scale * q.k_0."""
    hq, hkv, d = 2, 1, 128
    bt = np.array([[1]], np.int32)
    kp, vp = oracle.new_pools(2, hkv, d)
    rng = np.random.default_rng(3)
    k = bf16_bits(rng.standard_normal((1, hkv, d)))
    v = bf16_bits(rng.standard_normal((1, hkv, d)))
    q = bf16_bits(rng.standard_normal((1, hq, d)))
    oracle.kv_append(k, v, kp, vp, bt, np.array([0], np.int32), np.array([1], np.int32), lib=lib)
    out, lse = oracle.decode(q, kp, vp, bt, np.array([1], np.int32), hq, 0.5, lib=lib)
    for h in range(hq):
        assert np.array_equal(out[0, h], bits_to_f64(v[0, 0]))
        assert abs(lse[0, h] - 0.5 * float(bits_to_f64(q[0, h]) @ bits_to_f64(k[0, 0]))) < 1e-12


def pin_permutation(wl: W.Workload, lib=None):
    """Physical page placement does not change the result (bitwise in fp64)."""
    q = wl.packed("q", wl.extend_ranges())
    kp, vp = oracle_pools_for(wl, lib)
    a = oracle.extend(q, kp, vp, wl.block_table, wl.prefix_lens, wl.extend_lens,
                      wl.spec.num_q_heads, wl.sm_scale, lib=lib)
    perm = np.random.default_rng(11).permutation(wl.num_pages).astype(np.int32)
    wl2 = wl.remap_pages(perm)
    kp2, vp2 = oracle_pools_for(wl2, lib)
    b = oracle.extend(q, kp2, vp2, wl2.block_table, wl.prefix_lens, wl.extend_lens,
                      wl.spec.num_q_heads, wl.sm_scale, lib=lib)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def pin_gqa_replica(wl: W.Workload, lib=None):
    """Replicating kv head g to query heads g*G .. g*G+G-1 (G = 1) changes nothing."""
    hq, g = wl.spec.num_q_heads, wl.spec.group
    q = wl.packed("q", wl.extend_ranges())
    kp, vp = oracle_pools_for(wl, lib)
    a = oracle.extend(q, kp, vp, wl.block_table, wl.prefix_lens, wl.extend_lens, hq,
                      wl.sm_scale, lib=lib)
    kr = np.ascontiguousarray(np.repeat(kp, g, axis=1))
    vr = np.ascontiguousarray(np.repeat(vp, g, axis=1))
    b = oracle.extend(q, kr, vr, wl.block_table, wl.prefix_lens, wl.extend_lens, hq,
                      wl.sm_scale, lib=lib)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def pin_append(wl: W.Workload, lib=None):
    """Every new row lands at (BT[b][pos // 16], pos % 16); nothing else changes."""
    hkv, d = wl.spec.num_kv_heads, wl.spec.head_dim
    kp, vp = oracle.new_pools(wl.num_pages, hkv, d)
    kn = wl.packed("k", wl.extend_ranges())
    vn = wl.packed("v", wl.extend_ranges())
    oracle.kv_append(kn, vn, kp, vp, wl.block_table, wl.prefix_lens, wl.extend_lens, lib=lib)
    touched_k = np.zeros(kp.shape, bool)
    touched_v = np.zeros(vp.shape, bool)
    row = 0
    for b in range(wl.num_tasks):
        for j in range(int(wl.extend_lens[b])):
            pos = int(wl.prefix_lens[b]) + j
            page = int(wl.block_table[b, pos // 16])
            slot = pos % 16
            assert np.array_equal(kp[page, :, slot, :], kn[row]), (b, j)
            assert np.array_equal(vp[page, :, slot, :], vn[row]), (b, j)
            touched_k[page, :, slot, :] = True
            touched_v[page, :, slot, :] = True
            row += 1
    assert (kp[~touched_k] == oracle.CANARY).all()
    assert (vp[~touched_v] == oracle.CANARY).all()


def shrunk_workloads():
    """CPU-sized versions of the workloads (same structure, shorter lengths)."""
    s = W.SPECS
    return [
        W.make_workload(s["tiny_extend"]),
        W.make_workload(s["agent_resume_7b"].shrunk(num_tasks=3, length_div=64)),
        W.make_workload(s["resumed_decode"].shrunk(num_tasks=6, length_div=32)),
        W.make_workload(s["multimodal_resume"].shrunk(num_tasks=3, length_div=64)),
        W.make_workload(s["long_horizon"].shrunk(num_tasks=2, length_div=256)),
        W.make_workload(s["multimodal_prune_resume"].shrunk(num_tasks=3, length_div=32)),
    ]
