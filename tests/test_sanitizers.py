"""AddressSanitizer + UndefinedBehaviorSanitizer runs of the host code (CPU only).

The host planner with its checker (csrc/plan.cpp + tests/plan_check.cpp, over extend,
prefill, decode and shared-decode calls), the task-batching scheduler (csrc/ctb.cpp,
driven by tests/ctb_fuzz.cpp over random traces under both policies and invalid
arguments) and the oracle's C code (oracle/oracle.c, driven by tests/oracle_fuzz.c
including its error paths) are compiled with g++ / gcc and
-fsanitize=address,undefined -fno-sanitize-recover=all, so the first invalid access,
overflow or leak ends the program with a report.  No GPU code is involved.
"""
import os
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_10402_amd", "csrc")
INC = os.path.join(ROOT, "include")
TESTS = os.path.join(ROOT, "tests")
SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
       "-fno-sanitize-recover=all"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1")


def _build(tmp, name, cmd):
    exe = str(tmp / name)
    r = subprocess.run(cmd + ["-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return exe


def _run(exe, stdin=None):
    r = subprocess.run([exe], input=stdin, capture_output=True, text=True, env=ENV, timeout=600)
    report = r.stderr[-4000:]
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, report
    assert "ERROR: LeakSanitizer" not in r.stderr, report
    assert r.returncode == 0, (r.stdout[-2000:], report)
    return r.stdout


@pytest.fixture(scope="module")
def tmp(tmp_path_factory):
    probe = tmp_path_factory.mktemp("san")
    src = probe / "probe.c"
    src.write_text("int main(void) { return 0; }\n")
    r = subprocess.run(["gcc", *SAN, str(src), "-o", str(probe / "probe")], capture_output=True)
    if r.returncode != 0:
        pytest.skip("the sanitizer runtimes are not installed")
    return probe


def test_planner_under_sanitizers(tmp):
    exe = _build(tmp, "plan_check", ["g++", "-std=c++17", *SAN, "-I", CSRC, "-I", INC,
                                     os.path.join(TESTS, "plan_check.cpp"),
                                     os.path.join(CSRC, "plan.cpp")])
    rng = np.random.default_rng(21)
    lines = []
    for i in range(60):  # extend / prefill
        n = int(rng.integers(1, 9))
        p = rng.integers(0, 5000, size=n)
        e = rng.integers(0, 1500, size=n)
        op = 2 if i % 3 else 4
        lines.append("%d 28 4 128 %d %s" % (op, n, " ".join("%d %d" % x for x in zip(p, e))))
    for i in range(60):  # decode
        n = int(rng.integers(1, 300))
        kv = rng.integers(1, 20000, size=n)
        lines.append("3 32 8 %d %d %d %s" % (int(rng.choice([64, 128])), n,
                                             int(rng.choice([0, 1, 3, 50])),
                                             " ".join(map(str, kv))))
    for i in range(40):  # shared-prefix decode
        ng = int(rng.integers(1, 6))
        sizes = rng.integers(1, 9, size=ng)
        gs = np.concatenate([[0], np.cumsum(sizes)])
        sh = 16 * rng.integers(0, 100, size=ng)
        kv = np.concatenate([s + rng.integers(1, 3000, size=k) for s, k in zip(sh, sizes)])
        lines.append("100 32 8 128 %d %d %d %s %s %s" % (
            len(kv), int(rng.choice([0, 4])), ng, " ".join(map(str, gs)), " ".join(map(str, sh)),
            " ".join(map(str, kv))))
    out = _run(exe, "\n".join(lines) + "\n").strip().split("\n")
    assert len(out) == len(lines) and all(o.startswith("ok") for o in out)


def test_scheduler_under_sanitizers(tmp):
    exe = _build(tmp, "ctb_fuzz", ["g++", "-std=c++17", *SAN, "-I", CSRC, "-I", INC,
                                   os.path.join(TESTS, "ctb_fuzz.cpp"),
                                   os.path.join(CSRC, "ctb.cpp")])
    assert _run(exe).strip().endswith("ok")


def test_oracle_under_sanitizers(tmp):
    exe = _build(tmp, "oracle_fuzz", ["gcc", *SAN, "-fopenmp", os.path.join(TESTS, "oracle_fuzz.c"),
                                      os.path.join(ROOT, "oracle", "oracle.c"), "-lm"])
    assert _run(exe).strip().endswith("ok")
