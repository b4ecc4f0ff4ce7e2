"""Compile the HIP sources in csrc/ into paper_2608_10402_amd/libtide.so for gfx950.

    python -m paper_2608_10402_amd.build

Every call recompiles (a build check must not trust stale objects).  Kernels are
compiled with packed-fp32 instructions disabled, so fp32 arithmetic stays scalar.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG, "_build")
LIB_PATH = os.path.join(PKG, "libtide.so")

HIP_SOURCES = ["tide_api.hip", "attn_extend.hip", "attn_extend_append.hip", "attn_decode.hip",
               "kv_append.hip"]
CXX_SOURCES = ["plan.cpp", "ctb.cpp"]
ARCH = "gfx950"


def _hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the HIP library cannot be built")
    return path


def _common_flags():
    return ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-I", INCLUDE, "-I", CSRC]


def _compile_hip(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [_hipcc(), "--offload-arch=" + ARCH, *_common_flags(),
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-c", os.path.join(CSRC, src), "-o", obj]
    _run(cmd)
    return obj


def _compile_cxx(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = ["g++", *_common_flags(), "-Wall", "-Wextra", "-c", os.path.join(CSRC, src), "-o", obj]
    _run(cmd)
    return obj


def _run(cmd):
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # the host pass of hipcc does not know the packed-fp32 feature; that note is harmless
    out = "\n".join(l for l in res.stdout.splitlines() if "not a recognized feature" not in l)
    if res.returncode != 0:
        raise RuntimeError("command failed (%d): %s\n%s" % (res.returncode, " ".join(cmd), out))
    if out.strip():
        sys.stderr.write(out + "\n")


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs = min(8, len(HIP_SOURCES) + len(CXX_SOURCES))
    with concurrent.futures.ThreadPoolExecutor(jobs) as ex:
        futs = [ex.submit(_compile_hip, s) for s in HIP_SOURCES]
        futs += [ex.submit(_compile_cxx, s) for s in CXX_SOURCES]
        objs = [f.result() for f in futs]
    tmp = LIB_PATH + ".tmp%d" % os.getpid()
    _run([_hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB_PATH)
    if verbose:
        print("built", LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
