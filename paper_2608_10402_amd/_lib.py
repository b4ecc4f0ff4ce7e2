"""ctypes binding of libtide.so: the entry points of include/tide.h under the same names.

Argument marshalling only -- every step of the computation runs in the HIP kernels.
Device buffers are torch tensors on a ROCm device (torch supplies memory and streams);
lengths are host arrays.  Missing library => ImportError; a non-zero status from the
library => TideError.  There is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtide.so")

TIDE_OK = 0
TIDE_ERR_INVALID_ARG = -1
TIDE_ERR_UNSUPPORTED = -2
TIDE_ERR_CAPACITY = -3
TIDE_ERR_HIP = -4
TIDE_ERR_PAGE_RANGE = -5

TIDE_OP_KV_APPEND = 1
TIDE_OP_EXTEND = 2
TIDE_OP_DECODE = 3
TIDE_OP_FULL_PREFILL = 4

# bytes of the static device scratch of tide_decode_attn_noalloc (TIDE_NOALLOC_SCRATCH_BYTES)
NOALLOC_SCRATCH_BYTES = 64 << 20

EXPORTED = ("tide_workspace_size", "tide_kv_append", "tide_extend_attn", "tide_decode_attn",
            "tide_full_prefill_attn", "tide_decode_attn_shared", "tide_workspace_size_shared",
            "tide_decode_append_attn", "tide_decode_attn_noalloc", "tide_extend_append_attn",
            "tide_plan_info_get", "tide_ctb_create", "tide_ctb_step", "tide_ctb_get_stats", "tide_ctb_destroy",
            "tide_status_string", "tide_shutdown")


class TideError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (where, status_string(status), status))


class tide_dims(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("sm_scale", ctypes.c_float)]


class tide_plan_info(ctypes.Structure):
    _fields_ = [("num_items", ctypes.c_int32), ("waves_per_group", ctypes.c_int32),
                ("split", ctypes.c_int32), ("max_splits", ctypes.c_int32),
                ("merge_in_kernel", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_size_t)]


def make_dims(num_q_heads: int, num_kv_heads: int, head_dim: int, sm_scale: float,
              page_size: int = 16) -> tide_dims:
    return tide_dims(num_q_heads, num_kv_heads, head_dim, page_size, sm_scale)


_lib = None


def load(path: str = LIB_PATH):
    """Load libtide.so (once).  Raises ImportError when it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError("libtide.so not found at %s; build it with "
                          "`python -m paper_2608_10402_amd.build`" % path)
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    dims_p = ctypes.POINTER(tide_dims)
    lib.tide_workspace_size.argtypes = [ctypes.c_int, i32, vp, vp, dims_p, i32,
                                        ctypes.POINTER(sz)]
    lib.tide_kv_append.argtypes = [vp, vp, vp, vp, i64, vp, i32, i32, vp, vp, dims_p, vp, sz, vp]
    lib.tide_extend_attn.argtypes = [vp, vp, vp, i64, vp, i32, i32, vp, vp, dims_p, vp, vp, vp,
                                     sz, vp]
    lib.tide_decode_attn.argtypes = [vp, vp, vp, i64, vp, i32, i32, vp, dims_p, i32, vp, vp, vp,
                                     sz, vp]
    lib.tide_full_prefill_attn.argtypes = [vp, vp, vp, i64, vp, i32, i32, vp, dims_p, vp, vp, vp,
                                           sz, vp]
    lib.tide_decode_append_attn.argtypes = [vp, vp, vp, vp, vp, i64, vp, i32, i32, vp, dims_p,
                                            i32, vp, vp, vp, sz, vp]
    lib.tide_extend_append_attn.argtypes = [vp, vp, vp, vp, vp, i64, vp, i32, i32, vp, vp, dims_p,
                                            vp, vp, vp, sz, vp]
    lib.tide_decode_attn_noalloc.argtypes = [vp, vp, vp, i64, vp, i32, i32, vp, dims_p, i32, vp,
                                             vp, vp]
    lib.tide_decode_attn_shared.argtypes = [vp, vp, vp, i64, vp, i32, i32, vp, i32, vp, vp, dims_p,
                                            i32, vp, vp, vp, sz, vp]
    lib.tide_workspace_size_shared.argtypes = [i32, vp, i32, vp, vp, dims_p, i32,
                                               ctypes.POINTER(sz)]
    lib.tide_plan_info_get.argtypes = [ctypes.c_int, i32, vp, vp, dims_p, i32,
                                       ctypes.POINTER(tide_plan_info)]
    lib.tide_ctb_create.argtypes = [vp, i32, vp, vp, i32, vp, vp, vp, vp, vp,
                                    ctypes.POINTER(vp)]
    lib.tide_ctb_step.argtypes = [vp, vp]
    lib.tide_ctb_get_stats.argtypes = [vp, vp]
    lib.tide_ctb_destroy.argtypes = [vp]
    for name in EXPORTED[:-2]:
        getattr(lib, name).restype = ctypes.c_int
    lib.tide_status_string.argtypes = [ctypes.c_int]
    lib.tide_status_string.restype = ctypes.c_char_p
    lib.tide_shutdown.argtypes = []
    lib.tide_shutdown.restype = None
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().tide_status_string(int(status)).decode()


# ---- marshalling helpers ------------------------------------------------------------------
def _dev(t, dtype, name, nullable=False):
    if t is None:
        if nullable:
            return None
        raise ValueError("%s is required" % name)
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must live on a ROCm device" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t.data_ptr() if t.numel() else None


def _host(a, name):
    if a is None:
        return None, None
    arr = np.ascontiguousarray(np.asarray(a), dtype=np.int32)
    if arr.ndim != 1:
        raise ValueError("%s must be 1-D" % name)
    return arr, arr.ctypes.data


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _check(status, where):
    if status != TIDE_OK:
        raise TideError(status, where)


def _ws(workspace):
    if workspace is None:
        return None, 0
    if not isinstance(workspace, torch.Tensor) or workspace.device.type != "cuda":
        raise ValueError("workspace must be a device tensor")
    return workspace.data_ptr(), workspace.numel() * workspace.element_size()


def _same_device(*tensors):
    """All device tensors of one call must live on one device (the pointers are handed to
    kernels launched on that device)."""
    devs = {t.device for t in tensors if isinstance(t, torch.Tensor)}
    if len(devs) > 1:
        raise ValueError("all tensors of a call must be on one device, got %s" % sorted(map(str, devs)))


def _rows(t, name, rows, heads, d):
    """t must be [rows][heads][d] (the library reads and writes exactly that many bytes).
    rows None: the lengths are invalid, which the library itself rejects before any device
    work."""
    if t is None or rows is None:
        return
    if tuple(t.shape) != (rows, heads, d):
        raise ValueError("%s must have shape (%d, %d, %d), got %s"
                         % (name, rows, heads, d, tuple(t.shape)))


def _lse(t, rows, heads):
    if t is not None and rows is not None and tuple(t.shape) != (rows, heads):
        raise ValueError("lse must have shape (%d, %d), got %s" % (rows, heads, tuple(t.shape)))


def _block_table(bt, num_tasks):
    if not isinstance(bt, torch.Tensor) or bt.dim() != 2:
        raise ValueError("block_table must be a 2-D tensor [num_tasks][bt_stride]")
    if bt.shape[0] < num_tasks or bt.shape[1] < 1:
        raise ValueError("block_table has %d rows for %d tasks" % (bt.shape[0], num_tasks))
    return int(bt.shape[1])


def _lens_total(lens):
    """Sum of a host length array (the row count the library will use), or None when a
    length is negative: the library returns TIDE_ERR_INVALID_ARG for that itself."""
    if lens is None or (lens < 0).any():
        return None
    return int(lens.astype(np.int64).sum())


def _pool_shape(k_pool, v_pool, dims):
    if k_pool.dim() != 4 or v_pool.dim() != 4:
        raise ValueError("pools must be 4-D")
    n, hkv, ps, d = k_pool.shape
    if (hkv, ps, d) != (dims.num_kv_heads, dims.page_size, dims.head_dim):
        raise ValueError("k_pool must be [num_pages][Hkv][page_size][d]")
    if tuple(v_pool.shape) != (n, hkv, ps, d):
        raise ValueError("v_pool must be [num_pages][Hkv][page_size][d]")
    return int(n)


# ---- entry points ---------------------------------------------------------------------------
def tide_workspace_size(op: int, lens_a, lens_b, dims: tide_dims, num_splits: int = 0) -> int:
    a, a_p = _host(lens_a, "lens_a")
    b, b_p = _host(lens_b, "lens_b")
    n = 0 if a is None else int(a.size)
    out = ctypes.c_size_t(0)
    _check(load().tide_workspace_size(op, n, a_p, b_p, ctypes.byref(dims), int(num_splits),
                                      ctypes.byref(out)), "tide_workspace_size")
    return int(out.value)


def tide_plan_info_get(op: int, lens_a, lens_b, dims: tide_dims, num_splits: int = 0) -> dict:
    """The launch a call with these lengths makes (items, waves per workgroup, ...)."""
    a, a_p = _host(lens_a, "lens_a")
    b, b_p = _host(lens_b, "lens_b")
    n = 0 if a is None else int(a.size)
    info = tide_plan_info()
    _check(load().tide_plan_info_get(op, n, a_p, b_p, ctypes.byref(dims), int(num_splits),
                                     ctypes.byref(info)), "tide_plan_info_get")
    return {name: getattr(info, name) for name, _ in tide_plan_info._fields_ if name != "reserved"}


def alloc_workspace(nbytes: int, device="cuda") -> torch.Tensor:
    return torch.empty(max(1, int(nbytes)), dtype=torch.uint8, device=device)


def tide_kv_append(k_new, v_new, k_pool, v_pool, block_table, prefix_lens, extend_lens,
                   dims: tide_dims, workspace, stream=None) -> None:
    num_pages = _pool_shape(k_pool, v_pool, dims)
    p, p_p = _host(prefix_lens, "prefix_lens")
    e, e_p = _host(extend_lens, "extend_lens")
    if p is None or e is None or p.size != e.size:
        raise ValueError("prefix_lens and extend_lens must have one entry per task")
    rows = _lens_total(e)
    _rows(k_new, "k_new", rows, dims.num_kv_heads, dims.head_dim)
    _rows(v_new, "v_new", rows, dims.num_kv_heads, dims.head_dim)
    _block_table(block_table, int(p.size))
    _same_device(k_new, v_new, k_pool, v_pool, block_table, workspace)
    ws, ws_n = _ws(workspace)
    _check(load().tide_kv_append(
        _dev(k_new, torch.bfloat16, "k_new"), _dev(v_new, torch.bfloat16, "v_new"),
        _dev(k_pool, torch.bfloat16, "k_pool"), _dev(v_pool, torch.bfloat16, "v_pool"),
        num_pages, _dev(block_table, torch.int32, "block_table"), int(block_table.shape[1]),
        int(p.size), p_p, e_p, ctypes.byref(dims), ws, ws_n, _stream(stream)), "tide_kv_append")


def tide_extend_attn(q, k_pool, v_pool, block_table, prefix_lens, extend_lens, dims: tide_dims,
                     out, lse=None, workspace=None, stream=None) -> None:
    num_pages = _pool_shape(k_pool, v_pool, dims)
    p, p_p = _host(prefix_lens, "prefix_lens")
    e, e_p = _host(extend_lens, "extend_lens")
    if p is None or e is None or p.size != e.size:
        raise ValueError("prefix_lens and extend_lens must have one entry per task")
    rows = _lens_total(e)
    _rows(q, "q", rows, dims.num_q_heads, dims.head_dim)
    _rows(out, "out", rows, dims.num_q_heads, dims.head_dim)
    _lse(lse, rows, dims.num_q_heads)
    _block_table(block_table, int(p.size))
    _same_device(q, k_pool, v_pool, block_table, out, lse, workspace)
    ws, ws_n = _ws(workspace)
    _check(load().tide_extend_attn(
        _dev(q, torch.bfloat16, "q"), _dev(k_pool, torch.bfloat16, "k_pool"),
        _dev(v_pool, torch.bfloat16, "v_pool"), num_pages,
        _dev(block_table, torch.int32, "block_table"), int(block_table.shape[1]), int(p.size),
        p_p, e_p, ctypes.byref(dims), _dev(out, torch.bfloat16, "out"),
        _dev(lse, torch.float32, "lse", nullable=True), ws, ws_n, _stream(stream)),
        "tide_extend_attn")


def _decode_checks(q, out, lse, block_table, kv, dims, *others):
    if kv is None:
        raise ValueError("kv_lens is required")
    n = int(kv.size)
    _rows(q, "q", n, dims.num_q_heads, dims.head_dim)
    _rows(out, "out", n, dims.num_q_heads, dims.head_dim)
    _lse(lse, n, dims.num_q_heads)
    _block_table(block_table, n)
    _same_device(q, out, lse, block_table, *others)


def tide_extend_append_attn(q, k_new, v_new, k_pool, v_pool, block_table, prefix_lens,
                            extend_lens, dims: tide_dims, out, lse=None, workspace=None,
                            stream=None) -> None:
    num_pages = _pool_shape(k_pool, v_pool, dims)
    p, p_p = _host(prefix_lens, "prefix_lens")
    e, e_p = _host(extend_lens, "extend_lens")
    if p is None or e is None or p.size != e.size:
        raise ValueError("prefix_lens and extend_lens must have one entry per task")
    rows = _lens_total(e)
    _rows(q, "q", rows, dims.num_q_heads, dims.head_dim)
    _rows(out, "out", rows, dims.num_q_heads, dims.head_dim)
    _rows(k_new, "k_new", rows, dims.num_kv_heads, dims.head_dim)
    _rows(v_new, "v_new", rows, dims.num_kv_heads, dims.head_dim)
    _lse(lse, rows, dims.num_q_heads)
    _block_table(block_table, int(p.size))
    _same_device(q, k_new, v_new, k_pool, v_pool, block_table, out, lse, workspace)
    ws, ws_n = _ws(workspace)
    _check(load().tide_extend_append_attn(
        _dev(q, torch.bfloat16, "q"), _dev(k_new, torch.bfloat16, "k_new"),
        _dev(v_new, torch.bfloat16, "v_new"), _dev(k_pool, torch.bfloat16, "k_pool"),
        _dev(v_pool, torch.bfloat16, "v_pool"), num_pages,
        _dev(block_table, torch.int32, "block_table"), int(block_table.shape[1]), int(p.size),
        p_p, e_p, ctypes.byref(dims), _dev(out, torch.bfloat16, "out"),
        _dev(lse, torch.float32, "lse", nullable=True), ws, ws_n, _stream(stream)),
        "tide_extend_append_attn")


def tide_decode_attn(q, k_pool, v_pool, block_table, kv_lens, dims: tide_dims, out, lse=None,
                     num_splits: int = 0, workspace=None, stream=None) -> None:
    num_pages = _pool_shape(k_pool, v_pool, dims)
    kv, kv_p = _host(kv_lens, "kv_lens")
    _decode_checks(q, out, lse, block_table, kv, dims, k_pool, v_pool, workspace)
    ws, ws_n = _ws(workspace)
    _check(load().tide_decode_attn(
        _dev(q, torch.bfloat16, "q"), _dev(k_pool, torch.bfloat16, "k_pool"),
        _dev(v_pool, torch.bfloat16, "v_pool"), num_pages,
        _dev(block_table, torch.int32, "block_table"), int(block_table.shape[1]), int(kv.size),
        kv_p, ctypes.byref(dims), int(num_splits), _dev(out, torch.bfloat16, "out"),
        _dev(lse, torch.float32, "lse", nullable=True), ws, ws_n, _stream(stream)),
        "tide_decode_attn")


def tide_decode_append_attn(q, k_new, v_new, k_pool, v_pool, block_table, kv_lens,
                            dims: tide_dims, out, lse=None, num_splits: int = 0,
                            workspace=None, stream=None) -> None:
    num_pages = _pool_shape(k_pool, v_pool, dims)
    kv, kv_p = _host(kv_lens, "kv_lens")
    _decode_checks(q, out, lse, block_table, kv, dims, k_pool, v_pool, k_new, v_new, workspace)
    _rows(k_new, "k_new", int(kv.size), dims.num_kv_heads, dims.head_dim)
    _rows(v_new, "v_new", int(kv.size), dims.num_kv_heads, dims.head_dim)
    ws, ws_n = _ws(workspace)
    _check(load().tide_decode_append_attn(
        _dev(q, torch.bfloat16, "q"), _dev(k_new, torch.bfloat16, "k_new"),
        _dev(v_new, torch.bfloat16, "v_new"), _dev(k_pool, torch.bfloat16, "k_pool"),
        _dev(v_pool, torch.bfloat16, "v_pool"), num_pages,
        _dev(block_table, torch.int32, "block_table"), int(block_table.shape[1]), int(kv.size),
        kv_p, ctypes.byref(dims), int(num_splits), _dev(out, torch.bfloat16, "out"),
        _dev(lse, torch.float32, "lse", nullable=True), ws, ws_n, _stream(stream)),
        "tide_decode_append_attn")


def tide_decode_attn_noalloc(q, k_pool, v_pool, block_table, kv_lens, dims: tide_dims, out,
                             lse=None, num_splits: int = 0, stream=None) -> None:
    """tide_decode_attn without a workspace: runs in the library's static device scratch
    (NOALLOC_SCRATCH_BYTES per GPU); calls that overlap on one GPU race."""
    num_pages = _pool_shape(k_pool, v_pool, dims)
    kv, kv_p = _host(kv_lens, "kv_lens")
    _decode_checks(q, out, lse, block_table, kv, dims, k_pool, v_pool)
    _check(load().tide_decode_attn_noalloc(
        _dev(q, torch.bfloat16, "q"), _dev(k_pool, torch.bfloat16, "k_pool"),
        _dev(v_pool, torch.bfloat16, "v_pool"), num_pages,
        _dev(block_table, torch.int32, "block_table"), int(block_table.shape[1]), int(kv.size),
        kv_p, ctypes.byref(dims), int(num_splits), _dev(out, torch.bfloat16, "out"),
        _dev(lse, torch.float32, "lse", nullable=True), _stream(stream)),
        "tide_decode_attn_noalloc")


def _groups(group_start, shared_lens):
    gs, gs_p = _host(group_start, "group_start")
    sh, sh_p = _host(shared_lens, "shared_lens")
    if gs is None or sh is None or gs.size != sh.size + 1:
        raise ValueError("group_start must have one entry more than shared_lens")
    return int(sh.size), gs, gs_p, sh, sh_p


def tide_workspace_size_shared(kv_lens, group_start, shared_lens, dims: tide_dims,
                               num_splits: int = 0) -> int:
    kv, kv_p = _host(kv_lens, "kv_lens")
    ng, gs, gs_p, sh, sh_p = _groups(group_start, shared_lens)
    out = ctypes.c_size_t(0)
    _check(load().tide_workspace_size_shared(int(kv.size), kv_p, ng, gs_p, sh_p,
                                             ctypes.byref(dims), int(num_splits),
                                             ctypes.byref(out)), "tide_workspace_size_shared")
    return int(out.value)


def tide_decode_attn_shared(q, k_pool, v_pool, block_table, kv_lens, group_start, shared_lens,
                            dims: tide_dims, out, lse=None, num_splits: int = 0, workspace=None,
                            stream=None) -> None:
    num_pages = _pool_shape(k_pool, v_pool, dims)
    kv, kv_p = _host(kv_lens, "kv_lens")
    ng, gs, gs_p, sh, sh_p = _groups(group_start, shared_lens)
    _decode_checks(q, out, lse, block_table, kv, dims, k_pool, v_pool, workspace)
    ws, ws_n = _ws(workspace)
    _check(load().tide_decode_attn_shared(
        _dev(q, torch.bfloat16, "q"), _dev(k_pool, torch.bfloat16, "k_pool"),
        _dev(v_pool, torch.bfloat16, "v_pool"), num_pages,
        _dev(block_table, torch.int32, "block_table"), int(block_table.shape[1]), int(kv.size),
        kv_p, ng, gs_p, sh_p, ctypes.byref(dims), int(num_splits),
        _dev(out, torch.bfloat16, "out"), _dev(lse, torch.float32, "lse", nullable=True), ws,
        ws_n, _stream(stream)), "tide_decode_attn_shared")


def tide_full_prefill_attn(q, k_pool, v_pool, block_table, seq_lens, dims: tide_dims, out,
                           lse=None, workspace=None, stream=None) -> None:
    num_pages = _pool_shape(k_pool, v_pool, dims)
    s, s_p = _host(seq_lens, "seq_lens")
    if s is None:
        raise ValueError("seq_lens is required")
    rows = _lens_total(s)
    _rows(q, "q", rows, dims.num_q_heads, dims.head_dim)
    _rows(out, "out", rows, dims.num_q_heads, dims.head_dim)
    _lse(lse, rows, dims.num_q_heads)
    _block_table(block_table, int(s.size))
    _same_device(q, k_pool, v_pool, block_table, out, lse, workspace)
    ws, ws_n = _ws(workspace)
    _check(load().tide_full_prefill_attn(
        _dev(q, torch.bfloat16, "q"), _dev(k_pool, torch.bfloat16, "k_pool"),
        _dev(v_pool, torch.bfloat16, "v_pool"), num_pages,
        _dev(block_table, torch.int32, "block_table"), int(block_table.shape[1]), int(s.size),
        s_p, ctypes.byref(dims), _dev(out, torch.bfloat16, "out"),
        _dev(lse, torch.float32, "lse", nullable=True), ws, ws_n, _stream(stream)),
        "tide_full_prefill_attn")


def tide_shutdown() -> None:
    load().tide_shutdown()
