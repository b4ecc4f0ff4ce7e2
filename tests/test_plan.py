"""Host checks of the extend / prefill work lists (no GPU).

plan_check.cpp links the planner (plan.cpp, plain C++) and verifies, for each call it
reads, what the kernels assume of the uploaded work list: every row block covered once,
split chunks partitioning each block's key tiles, partial slots in bounds and written
once, merge descriptors naming exactly a row's chunks, workspace regions in order.  The
calls here cover the automatic choice and both forced plans over random and edge shapes.
"""
import os
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_10402_amd", "csrc")
OP_EXTEND, OP_PREFILL = 2, 4


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("plan") / "plan_check")
    subprocess.run(["g++", "-O2", "-std=c++17", "-Wall", "-Werror", "-I", CSRC, "-I",
                    os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "plan_check.cpp"),
                    os.path.join(CSRC, "plan.cpp"), "-o", exe], check=True)
    return exe


def _line(op, hq, hkv, d, prefix, extend):
    return "%d %d %d %d %d %s" % (op, hq, hkv, d, len(prefix),
                                  " ".join("%d %d" % (p, e) for p, e in zip(prefix, extend)))


def _run(exe, lines, mode=None):
    env = dict(os.environ)
    env.pop("TIDE_EXTEND_SPLIT", None)
    if mode is not None:
        env["TIDE_EXTEND_SPLIT"] = mode
    r = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True,
                       env=env)
    out = r.stdout.strip().split("\n")
    assert r.returncode == 0 and all(o.startswith("ok") for o in out), r.stdout[-2000:]
    assert len(out) == len(lines)
    return [o.split() for o in out]


def _random_calls(seed, n):
    rng = np.random.default_rng(seed)
    heads = [(28, 4), (32, 8), (8, 8), (16, 1), (12, 4), (32, 2), (64, 8)]
    lines = []
    for _ in range(n):
        hq, hkv = heads[rng.integers(len(heads))]
        d = int(rng.choice([64, 128]))
        ntask = int(rng.choice([1, 1, 2, 3, 4, 8, 17]))
        scale = int(rng.choice([10, 300, 3000, 20000]))
        prefix = rng.integers(0, scale, size=ntask)
        extend = rng.integers(0, max(2, scale // 4), size=ntask)
        extend[rng.random(ntask) < 0.2] = 0
        op = OP_EXTEND if rng.random() < 0.7 else OP_PREFILL
        if op == OP_PREFILL:
            prefix = np.zeros_like(prefix)
            extend = np.maximum(extend, 0)
        lines.append(_line(op, hq, hkv, d, prefix, extend))
    return lines


@pytest.mark.parametrize("mode", [None, "0", "1"])
def test_random_plans_are_valid(checker, mode):
    _run(checker, _random_calls(11, 150), mode)


def test_edge_plans_are_valid(checker):
    lines = [
        _line(OP_EXTEND, 28, 4, 128, [0], [1]),
        _line(OP_EXTEND, 28, 4, 128, [63], [1]),
        _line(OP_EXTEND, 28, 4, 128, [64 * 8 - 1], [1]),   # last key of a chunk grid line
        _line(OP_EXTEND, 16, 1, 128, [100000], [16]),       # one item, many chunks
        _line(OP_EXTEND, 8, 8, 64, [0, 0, 0], [0, 0, 5]),
        _line(OP_PREFILL, 28, 4, 128, [0], [65536]),
        _line(OP_EXTEND, 32, 32, 64, [2_000_000], [3]),     # capped chunk count
    ]
    for mode in (None, "0", "1"):
        _run(checker, lines, mode)


def test_split_choice(checker):
    """Few long items are split; a full batch and tiny calls keep the plain plan."""
    few = _line(OP_EXTEND, 28, 4, 128, [6000], [380])
    two = _line(OP_EXTEND, 28, 4, 128, [12000, 11000], [800, 700])
    rng = np.random.default_rng(3)
    many = _line(OP_EXTEND, 28, 4, 128, rng.integers(8000, 16000, 64), rng.integers(600, 1000, 64))
    tiny = _line(OP_EXTEND, 8, 8, 128, [16, 0], [1, 3])
    auto = _run(checker, [few, two, many, tiny])
    assert [a[1] for a in auto] == ["1", "1", "0", "0"]
    est_plain, est = float(auto[0][5]), float(auto[0][6])
    assert est < 0.6 * est_plain  # a one-task call leaves most CUs idle without the split
    plain = _run(checker, [few, two, many, tiny], "0")
    assert all(p[1] == "0" for p in plain)
    # the split plan's workspace adds the fp32 partials
    assert int(auto[0][4]) > int(plain[0][4])
    assert auto[2][2:5] == plain[2][2:5]


OP_DECODE, OP_SHARED = 3, 100


def _decode_line(hq, hkv, d, kv, splits=0):
    return "%d %d %d %d %d %d %s" % (OP_DECODE, hq, hkv, d, len(kv), splits,
                                     " ".join(str(int(x)) for x in kv))


def _shared_line(hq, hkv, d, kv, group_start, shared, splits=0):
    return "%d %d %d %d %d %d %d %s %s %s" % (
        OP_SHARED, hq, hkv, d, len(kv), splits, len(shared),
        " ".join(str(int(x)) for x in group_start), " ".join(str(int(x)) for x in shared),
        " ".join(str(int(x)) for x in kv))


def test_decode_plans_are_valid(checker):
    """Plain decode work lists: every (task, kv head) chunked exactly once in split order,
    full chunks before the shorter last ones (longest first), the merge mode as the rule
    says, counters zeroed in the upload, partial buffers sized for every slot."""
    rng = np.random.default_rng(5)
    heads = [(28, 4), (32, 8), (8, 8), (16, 1), (64, 8), (12, 4)]
    lines = []
    for i in range(120):
        hq, hkv = heads[rng.integers(len(heads))]
        d = int(rng.choice([64, 128]))
        n = int(rng.choice([1, 2, 7, 64, 256, 600]))
        scale = int(rng.choice([40, 1000, 8000, 60000]))
        kv = rng.integers(1, scale, size=n)
        splits = int(rng.choice([0, 0, 1, 2, 3, 7, 64]))
        lines.append(_decode_line(hq, hkv, d, kv, splits))
    lines += [
        _decode_line(28, 4, 128, [1]),                    # a lone first token
        _decode_line(32, 8, 128, [32, 33, 64, 4064, 4065]),
        _decode_line(16, 1, 64, [2_000_000]),             # chunk at its cap
        _decode_line(32, 8, 128, [16384] * 256),          # every chunk full
        _decode_line(32, 8, 128, [5] * 2048),             # one split each: direct writes
        _decode_line(8, 8, 64, [100, 3000], splits=100),  # more splits asked than keys
    ]
    out = _run(checker, lines)
    folds = [int(o[4]) for o in out]
    assert 0 in folds and 1 in folds  # both merge modes are exercised


def _decode_items(kv, hkv, c):
    return int(np.sum(-(-np.asarray(kv, dtype=np.int64) // c))) * hkv


def _expected_auto_chunk(kv, hkv):
    """The automatic decode chunk restated: for R rounds of 2048 waves (at most 8 values of
    R), the shortest chunk (a multiple of 32 in [512, 16384]) whose items fit, scored
    R * (1200 + chunk); if the best leaves fewer than 4 chunks per (task, kv head), or the
    shortest chunk already does, sum(kv) * Hkv / 4096 instead."""
    units = len(kv) * hkv

    def item_rule():
        c = -(-int(np.sum(kv)) * hkv // 4096)
        return min(max(-(-c // 32) * 32, 512), 16384)

    if _decode_items(kv, hkv, 512) < 4 * units:
        return item_rule()
    best, best_score = 16384, None
    r0 = max(1, -(-_decode_items(kv, hkv, 16384) // 2048))
    for r in range(r0, r0 + 8):
        if best_score is not None and r * (1200 + 512) >= best_score:
            break
        c = next(c for c in range(512, 16385, 32) if _decode_items(kv, hkv, c) <= 2048 * r)
        if best_score is None or r * (1200 + c) < best_score:
            best, best_score = c, r * (1200 + c)
        if c == 512:
            break
    return item_rule() if _decode_items(kv, hkv, best) < 4 * units else best


def test_decode_auto_chunk_rule(checker):
    """The planner's automatic decode chunk is the round rule (or, with fewer than 4 chunks
    per unit, the item-count rule), on the bench workloads' shapes and random ones."""
    rng = np.random.default_rng(11)
    cases = []
    for hq, hkv, n, lo, hi in [(28, 4, 64, 2048, 16384), (32, 8, 256, 1024, 32768),
                               (64, 8, 32, 33000, 99000), (32, 8, 32, 5000, 28000),
                               (28, 4, 16, 2000, 16000), (32, 8, 512, 256, 4000),
                               (16, 2, 200, 800, 12000), (64, 8, 8, 30000, 120000),
                               (28, 4, 1, 10, 100), (32, 8, 2048, 100, 400),
                               (32, 8, 20000, 1000, 9000)]:
        cases.append((hq, hkv, rng.integers(lo, hi, size=n)))
    out = _run(checker, [_decode_line(hq, hkv, 128, kv) for hq, hkv, kv in cases])
    for (hq, hkv, kv), o in zip(cases, out):
        assert int(o[2]) == _expected_auto_chunk(kv, hkv), (hq, hkv, len(kv))


def test_shared_decode_plans_are_valid(checker):
    """Shared-prefix decode work lists: per task and kv head the prompt chunks of its
    group and its own chunks give each split id once and tile [0, kv) in order; prompt
    items stay inside one group and 16 MFMA columns."""
    rng = np.random.default_rng(6)
    lines = []
    for i in range(80):
        hq, hkv = [(32, 8), (28, 4), (16, 1), (64, 8), (8, 8)][rng.integers(5)]
        d = int(rng.choice([64, 128]))
        ng = int(rng.choice([1, 2, 5, 16]))
        sizes = rng.integers(1, 9, size=ng)
        gs = np.concatenate([[0], np.cumsum(sizes)])
        shared = 16 * rng.integers(0, int(rng.choice([2, 60, 500])), size=ng)
        kv = np.concatenate([s + rng.integers(1, int(rng.choice([2, 300, 5000])), size=k)
                             for s, k in zip(shared, sizes)])
        splits = int(rng.choice([0, 0, 1, 4, 32]))
        lines.append(_shared_line(hq, hkv, d, kv, gs, shared, splits))
    lines += [
        _shared_line(32, 8, 128, [17, 17], [0, 2], [16]),          # one key past the prompt
        _shared_line(16, 1, 128, [1, 1, 1], [0, 3], [0]),          # no prompt at all
        _shared_line(8, 8, 64, [100001] * 4, [0, 4], [100000 // 16 * 16]),
    ]
    _run(checker, lines)
