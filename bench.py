#!/usr/bin/env python3
"""Benchmark of the paged-KV resume-attention hot path on one MI355X.

One step is one pass over every stage of the path for the chosen workload (default
agent_resume_7b: 64 tasks, 28 query / 4 KV heads, head_dim 128, page 16, prefixes
U{2048..16384}, observations log-uniform 64..2048, fragmented page placement):

  extend workloads (agent_resume_7b, multimodal_resume, tiny_extend)
    1. KV-append of the new observation tokens           (tide_kv_append)
    2. extend attention over the retained prefix         (tide_extend_attn)
    3. decode attention of one token per task (split-K)  (tide_decode_attn)
    4. with --reprefill 1, the recompute a cache miss forces: KV-append of the whole
       history, then full causal re-prefill attention     (tide_kv_append, tide_full_prefill_attn)
  resumed_decode
    1. KV-append of each task's decoded token, 2. split-K decode over its context,
    3. the same two steps as one fused call (tide_decode_append_attn), for comparison
  long_horizon
    1. KV-append of the new tokens, 2. extend, 3. eight rounds of (append one token, decode)
  grpo_group_decode
    1. KV-append of each trajectory's decoded token, 2. shared-prefix decode
       (tide_decode_attn_shared), 3. plain decode of the same tokens, for comparison
  multimodal_prune_resume
    as the extend workloads, with the new rows written over pages that still hold the
    context from before the sliding-window prune
  webshop_step (the task-batching scheduler, Section 4)
    one rollout step of 1056 WebShop-shaped trajectories scheduled round by round by the
    native scheduler -- Continuous Task Batching, then request-level batching with 1024
    and 512 tasks in flight -- each round's ops executed by the kernels (append + extend
    for every (re)prefill, append + decode for every generated token) on one rank's pool
    of 57344 pages; the step is the whole replay, so --steps and --warmup do not apply.
    Every round is scheduled and its inputs placed on the device first; the timed pass
    then runs the rounds' calls, bracketed by HIP events

Inputs are resident in HBM before timing starts.  `ms_per_step` comes from HIP events
around K whole steps on the stream the library launches on.  Each stage is then repeated
K times back to back under one event pair, which gives its per-call cost (its work-list
upload, its kernels and launch gaps included); the rates below use those times.

Printed: one JSON line.  For extend workloads `value` is extend-attention throughput in
TFLOP/s over the unmasked (query, key) pairs (4*d flops per pair and query head); for
resumed_decode it is decode-attention GB/s of algorithmic bytes, and for grpo_group_decode
the shared-prefix decode's GB/s over the bytes it must read (each prompt once per group).  The line also carries
the other stages' rates, the speedup of extend over re-prefill, the roofline of the
dominant kernel, and the fp64 oracle timed on a bounded sample on the host.  For extend
workloads, `extra.one_task_resume` times a resume round of a single task (the longest
prefix) outside the step, under the plain plan and under the planner's choice, which
splits the keys of a call that has too few work items for the chip.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "extend-attn TFLOP/s (% bf16 peak); decode-attn GB/s (% HBM); speedup vs re-prefill"
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E
# rocprofv3 counter summaries (copy-calibrated FETCH_SIZE + WRITE_SIZE per launch), keyed by
# (workload, dominant kernel); each records the hash of the kernel source it was taken on.
PROFILE_SUMMARIES = {
    ("agent_resume_7b", "extend"): "attn_extend_agent_resume_7b_counters.txt",
    ("resumed_decode", "decode"): "decode_split_resumed_decode_counters.txt",
    ("grpo_group_decode", "shared_decode"): "decode_split_grpo_group_decode_counters.txt",
    ("multimodal_prune_resume", "extend"): "attn_extend_multimodal_prune_resume_counters.txt",
    ("multimodal_resume", "extend"): "attn_extend_multimodal_resume_counters.txt",
    ("long_horizon", "extend"): "attn_extend_long_horizon_counters.txt",
    ("long_horizon", "decode"): "decode_split_long_horizon_counters.txt",
    ("agent_resume_7b", "decode"): "decode_split_agent_resume_7b_counters.txt",
    ("multimodal_resume", "decode"): "decode_split_multimodal_resume_counters.txt",
    ("multimodal_prune_resume", "decode"): "decode_split_multimodal_prune_resume_counters.txt",
}


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="agent_resume_7b")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="wall-time budget of the oracle CPU baseline sample (0 disables it)")
    ap.add_argument("--one-task", type=int, default=1,
                    help="for extend workloads, also time a one-task resume outside the step "
                         "(1) or not (0; profiling runs use 0 so every launch is the step's)")
    ap.add_argument("--reprefill", type=int, default=1,
                    help="include the recompute comparison (append history + full prefill) "
                         "for extend workloads (1) or not (0)")
    return ap.parse_args()


def extend_flops(wl) -> float:
    p = wl.prefix_lens.astype(np.float64)
    e = wl.extend_lens.astype(np.float64)
    pairs = float(np.sum(e * p + e * (e + 1) / 2))
    return 4.0 * wl.spec.head_dim * wl.spec.num_q_heads * pairs


def prefill_flops(wl) -> float:
    l = wl.seq_lens.astype(np.float64)
    return 4.0 * wl.spec.head_dim * wl.spec.num_q_heads * float(np.sum(l * (l + 1) / 2))


def decode_bytes(wl, kv_lens) -> float:
    s = wl.spec
    kv = float(np.sum(kv_lens)) * s.num_kv_heads * s.head_dim * 2 * 2  # K and V once
    qo = wl.num_tasks * s.num_q_heads * s.head_dim * 2 * 2              # Q in, O out
    bt = float(np.sum(-(-np.asarray(kv_lens) // 16))) * 4                 # page ids read
    return kv + qo + bt


def shared_decode_bytes(wl) -> float:
    """Bytes a group-aware decode must read: each group's prompt K/V once, every
    trajectory's own K/V, Q, O and page ids."""
    s = wl.spec
    per_tok = s.num_kv_heads * s.head_dim * 2 * 2
    sizes = np.diff(wl.group_start)
    shared = np.repeat(wl.shared_lens, sizes).astype(np.float64)
    own = wl.seq_lens.astype(np.float64) - shared
    kv = (float(np.sum(wl.shared_lens)) + float(np.sum(own))) * per_tok
    qo = wl.num_tasks * s.num_q_heads * s.head_dim * 2 * 2
    bt = float(np.sum(-(-wl.seq_lens // 16))) * 4
    return kv + qo + bt


def append_bytes(wl, tokens: int) -> float:
    s = wl.spec
    return float(tokens) * s.num_kv_heads * s.head_dim * 2 * 2 * 2  # K+V, read + write


def source_digest() -> str:
    """sha256 over every kernel and host source in csrc/ (names and bytes, sorted by name)
    and the build script that holds the compiler flags: a counter summary is only valid for
    the exact build it was taken from."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_10402_amd", "csrc")
    files = sorted(os.listdir(csrc)) + ["../build.py"]
    for name in files:
        path = os.path.join(csrc, name)
        if os.path.isfile(path):
            h.update(os.path.basename(name).encode() + b"\0")
            h.update(open(path, "rb").read())
    return h.hexdigest()


def counter_traffic(workload: str, kernel: str):
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3 counter
    summary, or None when there is none or any source or build flag changed since."""
    entry = PROFILE_SUMMARIES.get((workload, kernel))
    if entry is None:
        return None
    path = os.path.join(ROOT, "profiles", entry)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    m_bytes = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_hash or not m_bytes:
        return None
    return float(m_bytes.group(1)) if source_digest() == m_hash.group(1) else None


def kernel_label(wl, stage: str) -> str:
    """The instantiation the stage's dominant kernel runs as, from the plan the library
    makes for these lengths (tide_plan_info_get): extend<D, lse, split, append>,
    decode_split<D, shared, append, waves per workgroup>."""
    import paper_2608_10402_amd as tide
    s = wl.spec
    dims = tide.make_dims(s.num_q_heads, s.num_kv_heads, s.head_dim, wl.sm_scale)
    d = s.head_dim
    if stage == "extend":
        info = tide.tide_plan_info_get(tide.TIDE_OP_EXTEND, wl.prefix_lens, wl.extend_lens, dims)
        return "extend_attn_kernel<%d, false, %s, false>" % (d, "true" if info["split"] else "false")
    if stage == "decode":
        kv = wl.seq_lens + (1 if s.decode_steps else 0)  # the first of the fused decode steps
        info = tide.tide_plan_info_get(tide.TIDE_OP_DECODE, kv, None, dims)
        return "decode_split_kernel<%d, false, %s, %d>%s" % (
            d, "true" if s.decode_steps else "false", info["waves_per_group"],
            " (merge in kernel)" if info["merge_in_kernel"] else " + decode_merge_kernel")
    return "decode_split_kernel<%d, true, false, 4|8 by item count> + decode_merge_kernel" % d


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _task_pool(wl, b: int, n_pos: int):
    """The oracle's pool image of task b alone (positions 0 .. n_pos - 1 in pages 0, 1, ..),
    built by the oracle's own append from the seeded generator."""
    import oracle
    s = wl.spec
    n_pages = max(1, -(-n_pos // 16))
    kp, vp = oracle.new_pools(n_pages, s.num_kv_heads, s.head_dim)
    bt = np.arange(n_pages, dtype=np.int32).reshape(1, -1)
    oracle.kv_append(wl.k_rows(b, 0, n_pos), wl.v_rows(b, 0, n_pos), kp, vp, bt,
                     np.array([0], np.int32), np.array([n_pos], np.int32))
    return kp, vp, bt


def _oracle_rows(wl, b: int, positions, n_pos: int, threads: int):
    """fp64 oracle for query positions of task b (each attends keys 0 .. its position);
    returns (out [n, Hq, d], seconds spent in the oracle itself)."""
    import oracle
    s = wl.spec
    kp, vp, bt = _task_pool(wl, b, n_pos)
    pos = np.asarray(positions, np.int64)
    q = np.concatenate([wl.q_rows(b, int(t), int(t) + 1) for t in pos])
    t0 = time.perf_counter()
    o, _ = oracle.attention(q, pos, kp, vp, bt, np.array([0], np.int32),
                            np.array([n_pos], np.int32), s.num_q_heads, wl.sm_scale,
                            nthreads=threads)
    return o, time.perf_counter() - t0


def cpu_baseline_extend(wl, budget_s: float, extra_rows: int = 46):
    """The fp64 oracle on a bounded sample of extend rows, timed on the host cores: every
    task's first and last new row plus `extra_rows` seeded ones, all query heads.  Only the
    oracle's own calls are timed (building each task's pool image is not)."""
    import oracle
    s = wl.spec
    threads = oracle.threads()
    rng = np.random.default_rng(2608)
    indptr = np.concatenate([[0], np.cumsum(wl.extend_lens)]).astype(np.int64)
    secs, flops, rows, outs = 0.0, 0.0, 0, []
    for b in rng.permutation(wl.num_tasks):
        b = int(b)
        p, e = int(wl.prefix_lens[b]), int(wl.extend_lens[b])
        if e == 0:
            continue
        local = sorted(set([0, e - 1] + rng.integers(0, e, size=extra_rows).tolist()))
        pos = [p + j for j in local]
        o, dt = _oracle_rows(wl, b, pos, p + e, threads)
        secs += dt
        flops += 4.0 * s.head_dim * s.num_q_heads * float(sum(t + 1 for t in pos))
        rows += len(pos)
        outs.append((np.array([indptr[b] + j for j in local], np.int64), o))
        if secs > budget_s:
            break
    full = extend_flops(wl)
    info = {"value": flops / secs / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": "%d of %d extend rows (each sampled task's first and last row plus %d "
                      "seeded ones), all %d query heads, fp64; %.1f s of oracle time"
                      % (rows, int(indptr[-1]), extra_rows, s.num_q_heads, secs),
            "seconds": round(secs, 2), "flops": flops,
            "extrapolated_full_config_s": round(secs * full / flops, 1),
            "extrapolation": "sample time x (full-config FLOPs / sample FLOPs); not measured"}
    return info, outs


def cpu_baseline_decode(wl, budget_s: float, steps: int = 1):
    """The fp64 oracle over the decode queries of every task (steps consecutive decode
    positions per task), timed on the host cores; GB/s over the same algorithmic bytes as
    the GPU figure.  Only the oracle's own calls are timed."""
    import oracle
    s = wl.spec
    threads = oracle.threads()
    secs, nbytes, tasks = 0.0, 0.0, 0
    for b in range(wl.num_tasks):
        L = int(wl.seq_lens[b])
        if steps == 1:  # the decoded token is the last of the context
            pos, n_pos = [L - 1], L
        else:           # decode steps after the resume: positions L .. L + steps - 1
            pos, n_pos = [L + i for i in range(steps)], L + steps
        _, dt = _oracle_rows(wl, b, pos, n_pos, threads)
        secs += dt
        kv = np.array([t + 1 for t in pos])
        nbytes += float(kv.sum()) * s.num_kv_heads * s.head_dim * 4 + \
            len(pos) * s.num_q_heads * s.head_dim * 4 + float((-(-kv // 16)).sum()) * 4
        tasks += 1
        if secs > budget_s:
            break
    info = {"value": nbytes / secs / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": "%s: %d of %d tasks x %d decode step(s), all %d query heads, fp64; "
                      "%.1f s of oracle time" % ("full coverage" if tasks == wl.num_tasks else
                                                 "sample", tasks, wl.num_tasks, steps,
                                                 s.num_q_heads, secs),
            "seconds": round(secs, 2), "bytes": nbytes}
    if tasks < wl.num_tasks:
        info["extrapolated_full_config_s"] = round(secs * wl.num_tasks / tasks, 1)
        info["extrapolation"] = "sample time x (all tasks / sampled tasks); not measured"
    return info


def extend_vs_prefill(wl, keep, torch):
    """Every extend row against the same row of the full re-prefill, both from the GPU at
    full size (resume and recompute must agree): the largest and mean absolute difference."""
    full_start = np.concatenate([[0], np.cumsum(wl.seq_lens)[:-1]])
    rows = np.concatenate([np.arange(fs + p, fs + p + e) for fs, p, e in
                           zip(full_start, wl.prefix_lens, wl.extend_lens)]).astype(np.int64)
    sel = keep["out_full"][torch.from_numpy(rows).to(keep["out_full"].device)]
    diff = (sel.float() - keep["out_ext"].float()).abs()
    return {"rows": int(rows.size), "max_abs_diff": float(diff.max().item()),
            "mean_abs_diff": float(diff.mean().item())}


class Stage:
    """One timed call of the step: a callable plus its algorithmic work.  in_step=False
    marks a comparison (the same work done another way), timed on its own but not part of
    the step."""

    def __init__(self, name, fn, flops=0.0, bytes_=0.0, in_step=True):
        self.name, self.fn, self.flops, self.bytes = name, fn, flops, bytes_
        self.in_step = in_step
        self.times = []


def build_stages(wl, kv, dev, args, torch, np_up):
    """The step for this workload: the list of stages, in order."""
    s = wl.spec
    zeros = np.zeros(wl.num_tasks, np.int32)
    ones = np.ones(wl.num_tasks, np.int32)
    stages = []
    keep = {}
    if s.kind in ("extend", "long_horizon", "prune_resume"):
        k_ext, v_ext = np_up(wl.packed("k", wl.extend_ranges())), np_up(wl.packed("v", wl.extend_ranges()))
        q_ext = np_up(wl.packed("q", wl.extend_ranges()))
        out_ext = torch.empty_like(q_ext)
        keep.update(q_ext=q_ext, out_ext=out_ext)
        stages.append(Stage("append_new", lambda: kv.append(k_ext, v_ext, wl.prefix_lens, wl.extend_lens),
                            bytes_=append_bytes(wl, int(wl.extend_lens.sum()))))
        stages.append(Stage("extend", lambda: kv.extend(q_ext, wl.prefix_lens, wl.extend_lens, out=out_ext),
                            flops=extend_flops(wl)))
        # the same resume with the append fused into the attention (tide_extend_append_attn)
        out_fused = torch.empty_like(q_ext)
        keep.update(out_fused_ext=out_fused)
        stages.append(Stage("fused_append_extend",
                            lambda: kv.extend_append(q_ext, k_ext, v_ext, wl.prefix_lens,
                                                     wl.extend_lens, out=out_fused),
                            flops=extend_flops(wl), in_step=False))
    if s.kind in ("extend", "prune_resume"):
        last = np.cumsum(wl.extend_lens) - 1
        q_dec = keep["q_ext"][torch.from_numpy(last.astype(np.int64)).to(dev)].contiguous()
        out_dec = torch.empty_like(q_dec)
        stages.append(Stage("decode", lambda: kv.decode(q_dec, wl.seq_lens, out=out_dec),
                            bytes_=decode_bytes(wl, wl.seq_lens)))
        if args.reprefill:
            k_full, v_full = np_up(wl.packed("k", wl.full_ranges())), np_up(wl.packed("v", wl.full_ranges()))
            q_full = np_up(wl.packed("q", wl.full_ranges()))
            out_full = torch.empty_like(q_full)
            keep.update(out_full=out_full)
            stages.append(Stage("append_history", lambda: kv.append(k_full, v_full, zeros, wl.seq_lens),
                                bytes_=append_bytes(wl, int(wl.seq_lens.sum()))))
            stages.append(Stage("prefill", lambda: kv.prefill(q_full, wl.seq_lens, out=out_full),
                                flops=prefill_flops(wl)))
    elif s.kind == "group_decode":
        k_new, v_new = np_up(wl.packed("k", wl.extend_ranges())), np_up(wl.packed("v", wl.extend_ranges()))
        q_dec = np_up(wl.packed("q", wl.extend_ranges()))
        out_s, out_p = torch.empty_like(q_dec), torch.empty_like(q_dec)
        stages.append(Stage("append_new", lambda: kv.append(k_new, v_new, wl.prefix_lens, wl.extend_lens),
                            bytes_=append_bytes(wl, wl.num_tasks)))
        stages.append(Stage("shared_decode",
                            lambda: kv.decode_shared(q_dec, wl.seq_lens, wl.group_start,
                                                     wl.shared_lens, out=out_s),
                            bytes_=shared_decode_bytes(wl)))
        stages.append(Stage("plain_decode", lambda: kv.decode(q_dec, wl.seq_lens, out=out_p),
                            bytes_=decode_bytes(wl, wl.seq_lens)))
        keep.update(out_shared=out_s, out_plain=out_p)
    elif s.kind == "decode":
        k_new, v_new = np_up(wl.packed("k", wl.extend_ranges())), np_up(wl.packed("v", wl.extend_ranges()))
        q_dec = np_up(wl.packed("q", wl.extend_ranges()))
        out_dec = torch.empty_like(q_dec)
        stages.append(Stage("append_new", lambda: kv.append(k_new, v_new, wl.prefix_lens, wl.extend_lens),
                            bytes_=append_bytes(wl, wl.num_tasks)))
        stages.append(Stage("decode", lambda: kv.decode(q_dec, wl.seq_lens, out=out_dec),
                            bytes_=decode_bytes(wl, wl.seq_lens)))
        out_fused = torch.empty_like(q_dec)
        stages.append(Stage("fused_append_decode",
                            lambda: kv.decode_append(q_dec, k_new, v_new, wl.seq_lens, out=out_fused),
                            bytes_=decode_bytes(wl, wl.seq_lens) + append_bytes(wl, wl.num_tasks)))
        keep.update(out_dec=out_dec, out_fused=out_fused)
    if s.kind == "long_horizon":
        # eight generated tokens per task, each appended and attended in one fused call
        # (tide_decode_append_attn); the bytes are the decode's plus the token's append
        for step in range(s.decode_steps):
            rng = wl.decode_ranges(step)
            pos = (wl.seq_lens + step).astype(np.int32)
            kn, vn, qn = (np_up(wl.packed(x, rng)) for x in ("k", "v", "q"))
            on = torch.empty_like(qn)
            stages.append(Stage("decode_%d" % step,
                                (lambda qn=qn, kn=kn, vn=vn, on=on, pos=pos:
                                 kv.decode_append(qn, kn, vn, pos + 1, out=on)),
                                bytes_=decode_bytes(wl, pos + 1) + append_bytes(wl, wl.num_tasks)))
    return stages, keep


def one_task_resume(wl, kv, keep, steps, torch, stream):
    """A resume round that holds a single task: the workload's longest-prefix task alone,
    timed under the plain plan and under the planner's own choice (which is split-KV when
    one task leaves most compute units idle).  Outside the timed step."""
    s = wl.spec
    b = int(np.argmax(wl.prefix_lens))
    indptr = np.concatenate([[0], np.cumsum(wl.extend_lens)]).astype(np.int64)
    q = keep["q_ext"][int(indptr[b]):int(indptr[b + 1])]
    out = torch.empty_like(q)
    ext = np.zeros(wl.num_tasks, np.int32)
    ext[b] = wl.extend_lens[b]
    p, e = float(wl.prefix_lens[b]), float(wl.extend_lens[b])
    flops = 4.0 * s.head_dim * s.num_q_heads * (e * p + e * (e + 1) / 2)
    res = {"task": b, "prefix": int(p), "extend": int(e)}
    saved = os.environ.get("TIDE_EXTEND_SPLIT")
    try:
        for name, mode in (("plain", "0"), ("auto", None)):
            if mode is None:
                os.environ.pop("TIDE_EXTEND_SPLIT", None)
            else:
                os.environ["TIDE_EXTEND_SPLIT"] = mode
            for _ in range(3):
                kv.extend(q, wl.prefix_lens, ext, out=out)
            ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            ea.record(stream)
            for _ in range(steps):
                kv.extend(q, wl.prefix_lens, ext, out=out)
            eb.record(stream)
            torch.cuda.synchronize()
            t = ea.elapsed_time(eb) / steps
            res[name + "_ms"] = round(t, 4)
            res[name + "_TFLOPs"] = round(flops / (t * 1e-3) / 1e12, 1)
    finally:
        if saved is None:
            os.environ.pop("TIDE_EXTEND_SPLIT", None)
        else:
            os.environ["TIDE_EXTEND_SPLIT"] = saved
    res["speedup_auto_vs_plain"] = round(res["plain_ms"] / res["auto_ms"], 3)
    return res


CTB_POOL_PAGES = 57344   # 917,504 tokens: a 7B model's KV budget on an 80 GB GPU
CTB_MAX_RUNNING = 256
CTB_POLICIES = (("ctb", dict(policy=0)), ("request_f1024", dict(policy=1, max_in_flight=1024)),
                ("request_f512", dict(policy=1, max_in_flight=512)))


class ResidentRows:
    """Every trajectory's Q/K/V rows, drawn once from the seeded generator and kept in HBM;
    a round's rows are gathered on the device (inputs resident before timing)."""

    def __init__(self, tr, dev, torch, chunk=64):
        s = tr.spec
        self.torch, self.dev = torch, dev
        lens = tr.final_lens.astype(np.int64)
        self.off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        total = int(self.off[-1])
        self.t = {}
        for which, heads in (("k", s.num_kv_heads), ("v", s.num_kv_heads), ("q", s.num_q_heads)):
            buf = torch.empty((total, heads, s.head_dim), dtype=torch.bfloat16, device=dev)
            for a in range(0, tr.num_tasks, chunk):
                b = min(tr.num_tasks, a + chunk)
                tasks = np.arange(a, b)
                bits = tr.segments(which, tasks, np.zeros(b - a, np.int64), lens[a:b])
                host = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16)
                buf[int(self.off[a]):int(self.off[b])].copy_(host)
            self.t[which] = buf
            print("# resident %s rows: %d x %d x %d" % (which, total, heads, s.head_dim),
                  file=sys.stderr, flush=True)

    def locate(self, tasks, p0, p1):
        """Device index of rows p0[i]..p1[i]-1 of every task tasks[i], concatenated."""
        p0 = np.asarray(p0, np.int64)
        n = np.asarray(p1, np.int64) - p0
        first = self.off[np.asarray(tasks, np.int64)] + p0
        base = np.concatenate([[0], np.cumsum(n)[:-1]])
        idx = np.repeat(first - base, n) + np.arange(int(n.sum()), dtype=np.int64)
        # pinned and non-blocking: a pageable copy would make the host wait for the GPU
        return self.torch.from_numpy(idx).pin_memory().to(self.dev, non_blocking=True)

    def fetch(self, which, loc):
        return self.t[which].index_select(0, loc)

    def __call__(self, which, tasks, p0, p1):
        return self.fetch(which, self.locate(tasks, p0, p1))


def run_ctb(args, torch, tide):
    """Scheduler workload: replay one rollout step under each policy with the kernels."""
    import paper_2608_10402_amd.ctb as N
    import workloads.traces as T
    tr = T.make_trace(args.workload)
    s = tr.spec
    dev = torch.device("cuda", 0)
    kv = tide.PagedKV(CTB_POOL_PAGES, s.num_q_heads, s.num_kv_heads, s.head_dim,
                      np.zeros((1, 1), np.int32), device=dev, fill_canary=False)
    t_setup = time.perf_counter()
    rows = ResidentRows(tr, dev, torch)
    setup_s = time.perf_counter() - t_setup
    # warm-up: the first rounds of the CTB schedule (kernel loads, workspace growth)
    warm = N.Scheduler.from_trace(tr, pages_per_rank=CTB_POOL_PAGES, max_running=CTB_MAX_RUNNING)
    rep = N.Replay(kv, rows)
    for i, rnd in enumerate(warm.rounds()):
        rep.run(rnd, timed=False)
        if i == 60:
            break
    warm.close()
    torch.cuda.synchronize()
    res = {}
    for name, cfg in CTB_POLICIES:
        t0 = time.perf_counter()
        sched = N.Scheduler.from_trace(tr, pages_per_rank=CTB_POOL_PAGES,
                                       max_running=CTB_MAX_RUNNING, **cfg)
        rep = N.Replay(kv, rows)
        # Pass 1: schedule every round and put its inputs on the device (block tables,
        # row locators); pass 2 executes them, so the timed calls carry no host work but
        # their own (the scheduler is timed on its own, in pass 1).
        sched_s = 0.0
        prepared = []
        it = sched.rounds()
        while True:
            a = time.perf_counter()
            rnd = next(it, None)
            sched_s += time.perf_counter() - a
            if rnd is None:
                break
            prepared.append(rep.prepare(rnd))
        rep.reserve(prepared)
        torch.cuda.synchronize()
        for r, pr in enumerate(prepared):
            rep.execute(pr)
            if r % 200 == 0:
                rep.collect()   # bounds the number of live events
            if r % 500 == 0:
                print("# %s: round %d" % (name, r), file=sys.stderr, flush=True)
        rep.collect()
        del prepared
        wall = time.perf_counter() - t0
        st = sched.stats()
        sched.close()
        att = rep.ms["extend"] + rep.ms["decode"]
        res[name] = {
            "rounds": st["rounds"], "kv_hit_rate": round(st["hit_tokens"] / st["queried_tokens"], 4),
            "prefill_tokens": st["extend_tokens"], "recomputed_tokens": st["extend_tokens"] - st["input_tokens"],
            "pauses": st["pauses"], "extend_ms": round(rep.ms["extend"], 1),
            "decode_ms": round(rep.ms["decode"], 1), "attention_ms": round(att, 1),
            "extend_TFLOPs": round(rep.flops / max(rep.ms["extend"], 1e-9) / 1e9, 1),
            "decode_GBps": round(rep.kv_bytes / max(rep.ms["decode"], 1e-9) / 1e6, 1),
            "decoded_tokens": rep.tokens["decode"], "replay_wall_s": round(wall, 2),
            "scheduler_s": round(sched_s, 3), "kernel_calls": rep.calls}
        print("# %s: %s" % (name, json.dumps(res[name])), file=sys.stderr, flush=True)
    ctb = res["ctb"]
    v = ctb["decode_GBps"]
    roofline = {"bound": "hbm", "achieved": v, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(v / PEAK_HBM_GBS, 4), "kernel": "decode_split_kernel<128, false, true, 4|8>",
                "traffic": None}
    extra = {"policies": res, "setup_s": round(setup_s, 1),
             "attention_speedup_ctb_vs_request_f1024": round(
                 res["request_f1024"]["attention_ms"] / ctb["attention_ms"], 3),
             "attention_speedup_ctb_vs_request_f512": round(
                 res["request_f512"]["attention_ms"] / ctb["attention_ms"], 3),
             "hit_rate_gain_vs_request_f1024": round(
                 ctb["kv_hit_rate"] / res["request_f1024"]["kv_hit_rate"], 3),
             "hit_rate_gain_vs_request_f512": round(
                 ctb["kv_hit_rate"] / res["request_f512"]["kv_hit_rate"], 3)}
    cpu = None
    if args.cpu_seconds > 0:
        from oracle import ctb as OC
        t0 = time.perf_counter()
        OC.simulate(tr, OC.Config(policy=0, pages_per_rank=CTB_POOL_PAGES,
                                  max_running=CTB_MAX_RUNNING))
        dt = time.perf_counter() - t0
        cpu = {"value": round(ctb["rounds"] / dt, 1), "unit": "scheduled rounds/s", "cores": 1,
               "kind": "oracle", "sample": "the CTB schedule of the whole trace (%d rounds), "
               "scheduling only, %.1f s" % (ctb["rounds"], dt)}
        extra["scheduler_rounds_per_s_native"] = round(ctb["rounds"] / max(ctb["scheduler_s"], 1e-9), 1)
    line = {
        "metric": METRIC, "value": v, "unit": "GB/s", "n_gpus": 1, "steps": 1, "warmup": 0,
        "ms_per_step": ctb["attention_ms"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": s.key, "trajectories": tr.num_tasks, "q_heads": s.num_q_heads,
                   "kv_heads": s.num_kv_heads, "head_dim": s.head_dim, "page_size": 16,
                   "pool_pages": CTB_POOL_PAGES, "max_running": CTB_MAX_RUNNING},
        "roofline": roofline, "cpu_baseline": cpu, "extra": extra}
    print(json.dumps(line), flush=True)
    return 0


def main():
    args = parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this library has no multi-GPU path (each GPU would "
              "run its own rank's tasks independently). Run with --gpus 1.", file=sys.stderr)
        return 2
    import torch
    import paper_2608_10402_amd as tide
    import workloads as W
    import workloads.traces as WT

    if args.workload in WT.TRACE_SPECS:
        tide.load()
        torch.cuda.set_device(0)
        return run_ctb(args, torch, tide)

    tide.load()  # fail loudly if the HIP library is missing
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    wl = W.make_workload(args.workload)
    s = wl.spec

    def up(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)

    t_setup = time.time()
    kv = tide.PagedKV(wl.num_pages, s.num_q_heads, s.num_kv_heads, s.head_dim, wl.block_table,
                      wl.sm_scale, device=dev)
    zeros = np.zeros(wl.num_tasks, np.int32)
    if wl.shared_lens is not None:
        # a group's prompt pages are written once, then each trajectory's own positions
        shared = np.repeat(wl.shared_lens, np.diff(wl.group_start)).astype(np.int32)
        first = np.zeros(wl.num_tasks, np.int32)
        first[wl.group_start[:-1]] = wl.shared_lens
        rng = [(0, int(n)) for n in first]
        kv.append(up(wl.packed("k", rng)), up(wl.packed("v", rng)), zeros, first)
        own = (wl.prefix_lens - shared).astype(np.int32)
        rng = [(int(a), int(a + n)) for a, n in zip(shared, own)]
        kv.append(up(wl.packed("k", rng)), up(wl.packed("v", rng)), shared, own)
    elif wl.prefix_lens.sum() > 0:
        kv.append(up(wl.packed("k", wl.prefix_ranges())), up(wl.packed("v", wl.prefix_ranges())),
                  zeros, wl.prefix_lens)
    if wl.stale_lens is not None:
        # sliding-window prune: the pages still hold the pre-prune context past the prompt
        kv.append(up(wl.stale_packed("k")), up(wl.stale_packed("v")), wl.prefix_lens,
                  (wl.stale_lens - wl.prefix_lens).astype(np.int32))
    stages, keep = build_stages(wl, kv, dev, args, torch, up)
    torch.cuda.synchronize()
    setup_s = time.time() - t_setup
    stream = torch.cuda.current_stream()

    step_stages = [st for st in stages if st.in_step]

    def step():
        for st in step_stages:
            st.fn()

    for _ in range(args.warmup):
        step()
    # The comparison stages run once too, so that their first call's one-time costs (the
    # kernel's code load, a workspace allocation) stay out of their per-call timing.
    for st in stages:
        if not st.in_step:
            st.fn()
    torch.cuda.synchronize()
    # Whole-job timing: K steps, one event pair around them.
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = e0.elapsed_time(e1) / args.steps
    # Per-call cost of each stage: the stage repeated K times back to back under one
    # event pair (its work-list upload, its kernels and launch gaps included).  Timing
    # events placed between different stages inside a step attribute the time around a
    # kernel boundary imprecisely, so they are not used for the per-stage figures.
    # A stage that moves less than 1 GB could be served from the 256 MB MALL and the L2s
    # when repeated back to back, so it is timed call by call, with 512 MB of scratch
    # overwritten between calls (outside the events).  The other stages are also timed
    # call by call after their back-to-back run; the median and minimum of the per-call
    # times are reported beside the back-to-back mean, which the rates use.
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    for st in stages:
        if st.flops == 0 and st.bytes < 1e9:
            evs = []
            for r in range(args.steps):
                flush.fill_(r & 0xFF)
                ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                ea.record(stream)
                st.fn()
                eb.record(stream)
                evs.append((ea, eb))
            torch.cuda.synchronize()
            st.per_call = [a_.elapsed_time(b_) for a_, b_ in evs]
            st.times.append(sum(st.per_call) / args.steps)
            st.flushed = True
            continue
        ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ea.record(stream)
        for _ in range(args.steps):
            st.fn()
        eb.record(stream)
        torch.cuda.synchronize()
        st.times.append(ea.elapsed_time(eb) / args.steps)
        # the same calls one by one under their own events, for the median and the minimum
        evs = []
        for _ in range(args.steps):
            ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            ea.record(stream)
            st.fn()
            eb.record(stream)
            evs.append((ea, eb))
        torch.cuda.synchronize()
        st.per_call = [a_.elapsed_time(b_) for a_, b_ in evs]
    del flush
    ms = {st.name: float(np.mean(st.times)) for st in stages}

    def total(prefix):
        sel = [st for st in stages if st.name.startswith(prefix)]
        return (sum(np.mean(st.times) for st in sel), sum(st.flops for st in sel),
                sum(st.bytes for st in sel))

    extra = {"stage_ms": {k: round(v, 4) for k, v in ms.items()},
             "stage_ms_median_min": {st.name: [round(float(np.median(st.per_call)), 4),
                                               round(float(np.min(st.per_call)), 4)]
                                     for st in stages},
             "setup_s": round(setup_s, 1),
             "wall_ms_per_step": round(wall * 1e3 / args.steps, 3),
             "stages_timed_per_call_with_cache_flush": [st.name for st in stages
                                                        if getattr(st, "flushed", False)]}
    rooflines = {}
    if "fused_append_extend" in ms:
        extra["speedup_fused_vs_append_then_extend"] = round(
            (ms["append_new"] + ms["extend"]) / ms["fused_append_extend"], 3)
        extra["fused_extend_vs_separate_bitwise_equal"] = bool(torch.equal(
            keep["out_ext"].view(torch.int16), keep["out_fused_ext"].view(torch.int16)))
    if "extend" in ms:
        t, f = ms["extend"], extend_flops(wl)
        v = f / (t * 1e-3) / 1e12
        rooflines["extend"] = {"bound": "mfma", "achieved": round(v, 2), "peak": PEAK_BF16_TFLOPS,
                               "unit": "TFLOP/s", "frac": round(v / PEAK_BF16_TFLOPS, 4)}
        extra["extend_tokens_per_s"] = round(float(wl.extend_lens.sum()) / (t * 1e-3), 1)
        if args.one_task:
            extra["one_task_resume"] = one_task_resume(wl, kv, keep, args.steps, torch, stream)
    if "prefill" in ms:
        t, f, _ = total("prefill")
        v = f / (t * 1e-3) / 1e12
        rooflines["prefill"] = {"bound": "mfma", "achieved": round(v, 2), "peak": PEAK_BF16_TFLOPS,
                                "unit": "TFLOP/s", "frac": round(v / PEAK_BF16_TFLOPS, 4)}
        resume = ms["append_new"] + ms["extend"]
        recompute = ms["append_history"] + ms["prefill"]
        extra.update({
            "speedup_vs_reprefill": round(recompute / resume, 3),
            "speedup_vs_reprefill_attention_only": round(ms["prefill"] / ms["extend"], 3),
            "flop_ratio_prefill_over_extend": round(prefill_flops(wl) / extend_flops(wl), 3),
            "prefill_tokens_per_s": round(float(wl.seq_lens.sum()) / (ms["prefill"] * 1e-3), 1),
            "extend_vs_prefill_rows": extend_vs_prefill(wl, keep, torch),
        })
    if "fused_append_decode" in ms:
        extra["speedup_fused_vs_append_then_decode"] = round(
            (ms["append_new"] + ms["decode"]) / ms["fused_append_decode"], 3)
        extra["fused_vs_separate_bitwise_equal"] = bool(torch.equal(
            keep["out_dec"].view(torch.int16), keep["out_fused"].view(torch.int16)))
    if any(k.startswith("decode") for k in ms):
        t, _, b = total("decode")
        v = b / (t * 1e-3) / 1e9
        rooflines["decode"] = {"bound": "hbm", "achieved": round(v, 1), "peak": PEAK_HBM_GBS,
                               "unit": "GB/s", "frac": round(v / PEAK_HBM_GBS, 4)}
        n_dec = sum(1 for k in ms if k.startswith("decode"))
        extra["decode_tokens_per_s"] = round(n_dec * wl.num_tasks / (t * 1e-3), 1)
    if "shared_decode" in ms:
        t_s, t_p = ms["shared_decode"], ms["plain_decode"]
        st_s = [st for st in stages if st.name == "shared_decode"][0]
        st_p = [st for st in stages if st.name == "plain_decode"][0]
        v = st_s.bytes / (t_s * 1e-3) / 1e9
        rooflines["shared_decode"] = {"bound": "hbm", "achieved": round(v, 1), "peak": PEAK_HBM_GBS,
                                      "unit": "GB/s", "frac": round(v / PEAK_HBM_GBS, 4)}
        vp = st_p.bytes / (t_p * 1e-3) / 1e9
        rooflines["plain_decode"] = {"bound": "hbm", "achieved": round(vp, 1), "peak": PEAK_HBM_GBS,
                                     "unit": "GB/s", "frac": round(vp / PEAK_HBM_GBS, 4)}
        extra.update({
            "speedup_shared_vs_plain_decode": round(t_p / t_s, 3),
            # plain decode streams every page with the non-temporal hint, so the group's
            # shared prompt pages are re-read from HBM rather than L2
            "plain_decode_cache_policy": "non-temporal",
            "shared_decode_plain_equivalent_GBps": round(st_p.bytes / (t_s * 1e-3) / 1e9, 1),
            "decode_tokens_per_s": round(wl.num_tasks / (t_s * 1e-3), 1),
            "shared_vs_plain_max_abs_diff": float((keep["out_shared"].float() -
                                                   keep["out_plain"].float()).abs().max().item()),
        })
    if any(k.startswith("append") for k in ms):
        t, _, b = total("append")
        v = b / (t * 1e-3) / 1e9
        rooflines["append"] = {"bound": "hbm", "achieved": round(v, 1), "peak": PEAK_HBM_GBS,
                               "unit": "GB/s", "frac": round(v / PEAK_HBM_GBS, 4)}

    primary = ("extend" if "extend" in rooflines else
               "shared_decode" if "shared_decode" in rooflines else "decode")
    roofline = dict(rooflines[primary])
    roofline["kernel"] = kernel_label(wl, primary)
    roofline["traffic"] = counter_traffic(s.key, primary)
    for name, r in rooflines.items():  # HBM bytes per launch of each stage's kernel, where a summary exists
        r["traffic"] = counter_traffic(s.key, name)

    cpu = None
    if args.cpu_seconds > 0 and "extend" in ms:
        cpu, outs = cpu_baseline_extend(wl, args.cpu_seconds)
        got = keep["out_ext"].float().cpu().numpy()
        errs = [np.abs(got[b] - o) for b, o in outs]
        if errs:
            e = np.concatenate([x.ravel() for x in errs])
            extra["parity_sampled_rows"] = {"rows": int(sum(len(b) for b, _ in outs)),
                                            "max_abs_err": float(e.max()),
                                            "mean_abs_err": float(e.mean())}
        if s.decode_steps:
            extra["cpu_baseline_decode"] = cpu_baseline_decode(wl, args.cpu_seconds,
                                                               steps=s.decode_steps)
    elif args.cpu_seconds > 0 and ("decode" in ms or "shared_decode" in ms):
        cpu = cpu_baseline_decode(wl, args.cpu_seconds)

    line = {
        "metric": METRIC,
        "value": roofline["achieved"],
        "unit": roofline["unit"],
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": s.key, "tasks": wl.num_tasks, "q_heads": s.num_q_heads,
                   "kv_heads": s.num_kv_heads, "head_dim": s.head_dim, "page_size": s.page_size,
                   "extend_tokens": int(wl.extend_lens.sum()), "context_tokens": int(wl.seq_lens.sum()),
                   "pool_pages": wl.num_pages, "lens_digest": wl.lens_digest()},
        "roofline": roofline,
        "rooflines": rooflines,
        "cpu_baseline": cpu,
        "extra": extra,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
