"""fp64 CPU oracle of the paged-KV resume-attention path (TideRL, arXiv 2608.10402).

TEST INFRASTRUCTURE.  Only tests/, __graft_entry__.smoke() and bench.py's CPU
baseline may import this package.  It shares no code with the HIP library: the
arithmetic lives in oracle.c (plain C, fp64, OpenMP) and this module only marshals
numpy arrays into it.

Functions:
  new_pools      canary-filled host images of the K and V page pools
  kv_append      the append step: new tokens' K/V into their (page, slot)
  attention      attention for selected packed query rows (all rows by default)
  extend         every extend row (prefix_lens, extend_lens)
  decode         one query per task over kv_lens (== extend with E = 1)
  prefill        full causal attention over seq_lens (== extend with P = 0)

Pool layout (the library's documented one, restated independently in oracle.c):
  K and V [num_pages][Hkv][16][d], bf16 bits as uint16.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")
CANARY = 0x7FC0  # a bf16 quiet NaN: what an untouched pool slot holds
PAGE = 16

_lock = threading.Lock()
_libs: dict = {}


def build(force: bool = True, source: str = SOURCE, out: str = LIB_PATH) -> str:
    """Compile oracle.c with gcc (plain -O2: no reassociation of fp64 sums)."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", source, "-o", tmp, "-lm"],
                       check=True)
        os.replace(tmp, out)
    return out


def load(path: str = LIB_PATH):
    with _lock:
        lib = _libs.get(path)
        if lib is None:
            if path == LIB_PATH and not os.path.exists(path):
                build(force=False)
            lib = ctypes.CDLL(path)
            vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
            lib.oracle_kv_append.argtypes = [vp, vp, vp, vp, i64, vp, i32, i32, vp, vp, i32, i32]
            lib.oracle_kv_append.restype = ctypes.c_int
            lib.oracle_attention.argtypes = [vp, i64, vp, vp, vp, i64, vp, i32, i32, vp, vp, i32,
                                             i32, i32, ctypes.c_double, vp, vp, i32]
            lib.oracle_attention.restype = ctypes.c_int
            _libs[path] = lib
    return lib


def threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data


def new_pools(num_pages: int, num_kv_heads: int, head_dim: int):
    k = np.full((num_pages, num_kv_heads, PAGE, head_dim), CANARY, dtype=np.uint16)
    v = np.full((num_pages, num_kv_heads, PAGE, head_dim), CANARY, dtype=np.uint16)
    return k, v


def kv_append(k_new, v_new, k_pool, v_pool, block_table, prefix_lens, extend_lens, lib=None):
    """Write new K/V rows ([rows][Hkv][d] uint16) into the pool images in place."""
    lib = lib or load()
    num_pages, hkv, _, d = k_pool.shape
    assert k_pool.flags.c_contiguous and v_pool.flags.c_contiguous
    assert k_pool.dtype == np.uint16 and v_pool.dtype == np.uint16
    kn, kn_p = _c(k_new, np.uint16)
    vn, vn_p = _c(v_new, np.uint16)
    bt, bt_p = _c(block_table, np.int32)
    pl, pl_p = _c(prefix_lens, np.int32)
    el, el_p = _c(extend_lens, np.int32)
    assert kn.shape == (int(el.sum()), hkv, d) and vn.shape == kn.shape
    rc = lib.oracle_kv_append(kn_p, vn_p, k_pool.ctypes.data, v_pool.ctypes.data, num_pages,
                              bt_p, bt.shape[1], bt.shape[0], pl_p, el_p, hkv, d)
    if rc != 0:
        raise ValueError("oracle_kv_append failed: %d" % rc)


def attention(q_sel, sel_rows, k_pool, v_pool, block_table, prefix_lens, extend_lens,
              num_q_heads: int, scale: float, lib=None, nthreads: int | None = None):
    """fp64 output [n][Hq][d] and lse [n][Hq] of the selected packed query rows."""
    lib = lib or load()
    num_pages, hkv, _, d = k_pool.shape
    q, q_p = _c(q_sel, np.uint16)
    rows, rows_p = _c(sel_rows, np.int64)
    n = int(rows.size)
    assert q.shape == (n, num_q_heads, d)
    bt, bt_p = _c(block_table, np.int32)
    pl, pl_p = _c(prefix_lens, np.int32)
    el, el_p = _c(extend_lens, np.int32)
    out = np.zeros((n, num_q_heads, d), dtype=np.float64)
    lse = np.zeros((n, num_q_heads), dtype=np.float64)
    rc = lib.oracle_attention(q_p, n, rows_p, k_pool.ctypes.data, v_pool.ctypes.data, num_pages,
                              bt_p, bt.shape[1], bt.shape[0], pl_p, el_p, num_q_heads, hkv, d,
                              float(scale), out.ctypes.data, lse.ctypes.data,
                              int(nthreads or threads()))
    if rc != 0:
        raise ValueError("oracle_attention failed: %d" % rc)
    return out, lse


def extend(q, k_pool, v_pool, block_table, prefix_lens, extend_lens, num_q_heads, scale,
           **kw):
    rows = np.arange(int(np.sum(extend_lens)), dtype=np.int64)
    return attention(q, rows, k_pool, v_pool, block_table, prefix_lens, extend_lens,
                     num_q_heads, scale, **kw)


def decode(q, k_pool, v_pool, block_table, kv_lens, num_q_heads, scale, **kw):
    kv = np.asarray(kv_lens, dtype=np.int32)
    return extend(q, k_pool, v_pool, block_table, kv - 1, np.ones_like(kv), num_q_heads, scale,
                  **kw)


def prefill(q, k_pool, v_pool, block_table, seq_lens, num_q_heads, scale, **kw):
    sl = np.asarray(seq_lens, dtype=np.int32)
    return extend(q, k_pool, v_pool, block_table, np.zeros_like(sl), sl, num_q_heads, scale,
                  **kw)
