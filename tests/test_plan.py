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
