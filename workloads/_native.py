"""Loader (and builder) of the counter-based normal generator in philox_normal.c."""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "philox_normal.c")
_LIB_PATH = os.path.join(_HERE, "libtidegen.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile philox_normal.c with gcc into workloads/libtidegen.so."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH):
                build(force=False)
            lib = ctypes.CDLL(_LIB_PATH)
            lib.tg_normal_bf16.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32,
                                           ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p,
                                           ctypes.c_int]
            lib.tg_normal_bf16.restype = None
            lib.tg_normal_f32.argtypes = lib.tg_normal_bf16.argtypes
            lib.tg_normal_f32.restype = None
            lib.tg_normal_bf16_segments.argtypes = [
                ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64, ctypes.c_void_p,
                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
            lib.tg_normal_bf16_segments.restype = None
            lib.tg_philox4x32_10.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
            lib.tg_philox4x32_10.restype = None
            _lib = lib
    return _lib


def host_threads() -> int:
    """Threads the generator may use: the CPUs this process may run on, at most 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def philox4x32_10(ctr, key) -> list:
    lib = _load()
    c = (ctypes.c_uint32 * 4)(*ctr)
    k = (ctypes.c_uint32 * 2)(*key)
    out = (ctypes.c_uint32 * 4)()
    lib.tg_philox4x32_10(c, k, out)
    return list(out)


def normal_bf16(seed: int, stream_a: int, stream_b: int, first: int, n: int,
                out: np.ndarray | None = None) -> np.ndarray:
    """bf16 bit patterns (uint16) of N(0,1) samples first .. first+n-1 of a stream."""
    lib = _load()
    if out is None:
        out = np.empty(n, dtype=np.uint16)
    assert out.dtype == np.uint16 and out.flags.c_contiguous and out.size == n
    lib.tg_normal_bf16(seed, stream_a, stream_b, first, n, out.ctypes.data, host_threads())
    return out


def normal_f32(seed: int, stream_a: int, stream_b: int, first: int, n: int) -> np.ndarray:
    lib = _load()
    out = np.empty(n, dtype=np.float32)
    lib.tg_normal_f32(seed, stream_a, stream_b, first, n, out.ctypes.data, host_threads())
    return out


def normal_bf16_segments(seed: int, stream_a: int, stream_b, first, length) -> np.ndarray:
    """Concatenation of normal_bf16(seed, stream_a, stream_b[i], first[i], length[i])."""
    lib = _load()
    sb = np.ascontiguousarray(stream_b, dtype=np.uint32)
    fi = np.ascontiguousarray(first, dtype=np.uint64)
    ln = np.ascontiguousarray(length, dtype=np.int64)
    assert sb.shape == fi.shape == ln.shape and (ln >= 0).all()
    out = np.empty(int(ln.sum()), dtype=np.uint16)
    lib.tg_normal_bf16_segments(seed, stream_a, sb.size, sb.ctypes.data, fi.ctypes.data,
                                ln.ctypes.data, out.ctypes.data, host_threads())
    return out
