"""Code-generation checks of the gfx950 kernels (CPU only: hipcc cross-compiles).

Every attention kernel keeps its K/V tiles in flight with hand-counted vmcnt waits, and
its inner loops use the whole register file.  A value the compiler spills inside such a
loop costs a scratch (vector-memory) access, and each reload forces a wait for every
older vector-memory operation, i.e. for every K/V prefetch in flight.  The LSE extend
variant once ran 2.6x slower than the plain one for exactly this reason.  These tests
compile each kernel source to assembly with the library's own flags and check that no
loop of any kernel contains a scratch access.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_10402_amd", "csrc")
INC = os.path.join(ROOT, "include")

SOURCES = ["attn_extend.hip", "attn_extend_append.hip", "attn_decode.hip", "kv_append.hip"]


def _hipcc():
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        pytest.skip("hipcc not available")
    return path


def _asm(tmp_path, src):
    out = str(tmp_path / (src + ".s"))
    cmd = [_hipcc(), "--offload-arch=gfx950", "-O3", "-std=c++17", "-I", INC, "-I", CSRC,
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "--cuda-device-only",
           "-S", os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-3000:]
    return open(out).read().split("\n")


def loops_with_scratch(lines):
    """[(kernel, loop label, scratch accesses inside the loop)] for every loop of every
    kernel: a loop runs from its header label (marked 'Loop Header' by the compiler) to
    the last branch back to it."""
    kernels = [(m.group(1), i) for i, l in enumerate(lines)
               for m in [re.match(r"^(_Z\S+):", l)] if m]
    out = []
    for j, (name, start) in enumerate(kernels):
        end = kernels[j + 1][1] if j + 1 < len(kernels) else len(lines)
        body = lines[start:end]
        for k, l in enumerate(body):
            if "Loop Header" not in l:
                continue
            label = l.split(":")[0]
            back = [q for q, x in enumerate(body)
                    if re.search(r"\ts_(c)?branch\S*\s+" + re.escape(label) + r"\s*$", x)]
            if not back:
                continue
            n = sum(1 for x in body[k:max(back) + 1] if "scratch_" in x)
            out.append((name, label, n))
    return out


def test_loop_finder_sees_a_planted_spill():
    """The scanner itself: a loop with a scratch access is reported, one without is not."""
    text = """_Zkern:
.LBB0_1:                                ; =>This Inner Loop Header: Depth=1
\tv_add_f32_e32 v0, v1, v0
\tscratch_load_dword v2, off, off offset:4
\ts_cbranch_scc1 .LBB0_1
.LBB0_2:                                ; =>This Inner Loop Header: Depth=1
\tv_add_f32_e32 v0, v1, v0
\ts_cbranch_scc1 .LBB0_2
\tscratch_store_dword off, v2, off
\ts_endpgm"""
    assert loops_with_scratch(text.split("\n")) == [("_Zkern", ".LBB0_1", 1), ("_Zkern", ".LBB0_2", 0)]


@pytest.mark.parametrize("src", SOURCES)
def test_no_scratch_access_inside_loops(tmp_path, src):
    found = loops_with_scratch(_asm(tmp_path, src))
    assert found, "no loops found in %s: the scanner no longer matches the assembly" % src
    bad = [(k, l, n) for k, l, n in found if n]
    assert not bad, "scratch accesses inside loops: %s" % bad
