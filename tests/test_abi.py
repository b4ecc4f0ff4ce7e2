"""The C ABI on the CPU: libtide.so loads, exports exactly what include/tide.h declares,
and rejects bad arguments with the documented status codes before touching a GPU.

No call here launches work: every call fails validation (or is a no-op) on the host.
"""
import ctypes
import math
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2608_10402_amd as tide
from paper_2608_10402_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("tide.h", "tide_ctb.h")]


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    return sorted(set(re.findall(r"TIDE_API\s+[\w\s\*]+?\b(tide_\w+)\s*\(", text)))


def exported_functions():
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], check=True,
                         capture_output=True, text=True).stdout
    return sorted(l.split()[-1] for l in out.splitlines() if " T " in l)


def test_library_exports_exactly_the_header():
    lib = tide.load()
    decl = declared_functions()
    assert decl == sorted(_lib.EXPORTED)
    assert exported_functions() == decl
    for name in decl:
        assert hasattr(lib, name)


def test_header_compiles_as_c():
    src = ('#include "tide.h"\n#include "tide_ctb.h"\nint main(void) { tide_dims d = {8, 2, 64, 16, '
           '0.125f}; tide_ctb_config c = {0, 1, 64, 1024, 8, 8, 0, 100}; (void)d; (void)c; '
           'return 0; }\n')
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                        "-x", "c", "-", "-fsyntax-only"], input=src, text=True, capture_output=True)
    assert r.returncode == 0, r.stderr


def test_status_strings():
    for code in (0, -1, -2, -3, -4, -5):
        assert tide.status_string(code) and tide.status_string(code) != "unknown status"
    assert tide.status_string(42) == "unknown status"


def _ws(op, a, b, dims, splits=0):
    lib = tide.load()
    arr_a = None if a is None else np.ascontiguousarray(a, np.int32)
    arr_b = None if b is None else np.ascontiguousarray(b, np.int32)
    n = 0 if arr_a is None else arr_a.size
    out = ctypes.c_size_t(0)
    rc = lib.tide_workspace_size(op, n, None if arr_a is None else arr_a.ctypes.data,
                                 None if arr_b is None else arr_b.ctypes.data,
                                 ctypes.byref(dims) if dims is not None else None, splits,
                                 ctypes.byref(out))
    return rc, out.value


GOOD = _lib.make_dims(28, 4, 128, 1 / math.sqrt(128))


@pytest.mark.parametrize("dims,code", [
    (_lib.make_dims(8, 2, 96, 0.1), tide.TIDE_ERR_UNSUPPORTED),      # head_dim 96
    (_lib.make_dims(8, 3, 64, 0.1), tide.TIDE_ERR_UNSUPPORTED),      # 8 % 3 != 0
    (_lib.make_dims(34, 2, 64, 0.1), tide.TIDE_ERR_UNSUPPORTED),     # group 17 > 16
    (_lib.make_dims(65537, 65537, 64, 0.1), tide.TIDE_ERR_UNSUPPORTED),  # Hkv > 65536
    (_lib.make_dims(8, 2, 64, 0.1, page_size=32), tide.TIDE_ERR_UNSUPPORTED),
    (_lib.make_dims(0, 2, 64, 0.1), tide.TIDE_ERR_INVALID_ARG),
    (_lib.make_dims(8, 2, 64, 0.0), tide.TIDE_ERR_INVALID_ARG),
    (_lib.make_dims(8, 2, 64, float("nan")), tide.TIDE_ERR_INVALID_ARG),
    (_lib.make_dims(8, 2, 64, float("inf")), tide.TIDE_ERR_INVALID_ARG),
    (None, tide.TIDE_ERR_INVALID_ARG),
])
def test_dims_validation(dims, code):
    rc, _ = _ws(tide.TIDE_OP_EXTEND, [10], [5], dims)
    assert rc == code


def test_length_validation():
    assert _ws(tide.TIDE_OP_EXTEND, [10, -1], [5, 5], GOOD)[0] == tide.TIDE_ERR_INVALID_ARG
    assert _ws(tide.TIDE_OP_EXTEND, [10], [-5], GOOD)[0] == tide.TIDE_ERR_INVALID_ARG
    assert _ws(tide.TIDE_OP_EXTEND, [10], None, GOOD)[0] == tide.TIDE_ERR_INVALID_ARG
    assert _ws(tide.TIDE_OP_DECODE, [10, 0], None, GOOD)[0] == tide.TIDE_ERR_INVALID_ARG
    assert _ws(tide.TIDE_OP_DECODE, [10], None, GOOD, splits=-1)[0] == tide.TIDE_ERR_INVALID_ARG
    assert _ws(tide.TIDE_OP_EXTEND, [2**31 - 10], [100], GOOD)[0] == tide.TIDE_ERR_INVALID_ARG
    assert _ws(99, [1], [1], GOOD)[0] == tide.TIDE_ERR_INVALID_ARG


def test_workspace_sizes_are_consistent(monkeypatch):
    monkeypatch.setenv("TIDE_EXTEND_SPLIT", "0")  # the plain plan: no partials
    rc, a = _ws(tide.TIDE_OP_EXTEND, [100, 2000], [10, 300], GOOD)
    assert rc == 0 and a > 0
    rc, b = _ws(tide.TIDE_OP_EXTEND, [100, 2000], [10, 3000], GOOD)
    assert rc == 0 and b >= a  # more rows, more work items
    monkeypatch.setenv("TIDE_EXTEND_SPLIT", "1")  # the split plan adds fp32 partials
    rc, a1 = _ws(tide.TIDE_OP_EXTEND, [100, 2000], [10, 300], GOOD)
    assert rc == 0 and a1 > a
    monkeypatch.delenv("TIDE_EXTEND_SPLIT")
    rc, a2 = _ws(tide.TIDE_OP_EXTEND, [100, 2000], [10, 300], GOOD)
    assert rc == 0 and a2 in (a, a1)
    rc, p = _ws(tide.TIDE_OP_FULL_PREFILL, [110, 2300], None, GOOD)
    assert rc == 0 and p > 0
    rc, d1 = _ws(tide.TIDE_OP_DECODE, [5000, 9000], None, GOOD, splits=1)
    rc2, d8 = _ws(tide.TIDE_OP_DECODE, [5000, 9000], None, GOOD, splits=8)
    assert rc == 0 and rc2 == 0 and d8 > d1  # partials grow with the split count
    rc, z = _ws(tide.TIDE_OP_EXTEND, [], [], GOOD)
    assert rc == 0 and z > 0  # header only


def _call_extend(**over):
    lib = tide.load()
    args = dict(q=1, k=1, v=1, pages=10, bt=1, stride=4, n=1, p=[3], e=[2], dims=GOOD, out=1,
                lse=None, ws=1, ws_bytes=1 << 20)
    args.update(over)
    p = np.ascontiguousarray(args["p"], np.int32)
    e = np.ascontiguousarray(args["e"], np.int32)
    return lib.tide_extend_attn(args["q"], args["k"], args["v"], args["pages"], args["bt"],
                                args["stride"], args["n"], p.ctypes.data, e.ctypes.data,
                                ctypes.byref(args["dims"]) if args["dims"] else None, args["out"],
                                args["lse"], args["ws"], args["ws_bytes"], None)


def test_entry_point_validation_without_gpu():
    # each of these fails (or is a no-op) before any HIP call
    assert _call_extend(n=0) == tide.TIDE_OK                              # no tasks: no-op
    assert _call_extend(e=[0]) == tide.TIDE_OK                            # no rows: no-op
    assert _call_extend(n=-1) == tide.TIDE_ERR_INVALID_ARG
    assert _call_extend(q=None) == tide.TIDE_ERR_INVALID_ARG
    assert _call_extend(out=None) == tide.TIDE_ERR_INVALID_ARG
    assert _call_extend(ws=None) == tide.TIDE_ERR_INVALID_ARG
    assert _call_extend(pages=0) == tide.TIDE_ERR_INVALID_ARG
    assert _call_extend(stride=0) == tide.TIDE_ERR_INVALID_ARG
    assert _call_extend(p=[60], e=[10]) == tide.TIDE_ERR_CAPACITY          # 70 tokens > 4 pages
    assert _call_extend(ws_bytes=16) == tide.TIDE_ERR_CAPACITY
    assert _call_extend(dims=_lib.make_dims(8, 2, 80, 0.1)) == tide.TIDE_ERR_UNSUPPORTED
    assert _call_extend(p=[-1]) == tide.TIDE_ERR_INVALID_ARG


def test_other_entry_points_validation_without_gpu():
    lib = tide.load()
    one = np.array([1], np.int32)
    bad = np.array([0], np.int32)
    d = ctypes.byref(GOOD)
    assert lib.tide_decode_attn(1, 1, 1, 10, 1, 4, 1, bad.ctypes.data, d, 0, 1, None, 1, 1 << 20,
                                None) == tide.TIDE_ERR_INVALID_ARG       # kv_len 0
    assert lib.tide_decode_attn(1, 1, 1, 10, 1, 4, 0, None, d, 0, 1, None, 1, 0,
                                None) == tide.TIDE_OK                     # no tasks
    assert lib.tide_decode_attn(1, 1, 1, 10, 1, 4, 1, one.ctypes.data, d, -2, 1, None, 1, 1 << 20,
                                None) == tide.TIDE_ERR_INVALID_ARG       # negative splits
    assert lib.tide_full_prefill_attn(1, 1, 1, 10, 1, 4, 1, np.array([65], np.int32).ctypes.data,
                                      d, 1, None, 1, 1 << 20, None) == tide.TIDE_ERR_CAPACITY
    assert lib.tide_kv_append(None, 1, 1, 1, 10, 1, 4, 1, one.ctypes.data, one.ctypes.data, d, 1,
                              1 << 20, None) == tide.TIDE_ERR_INVALID_ARG
    assert lib.tide_kv_append(1, 1, 1, 1, 10, 1, 4, 1, one.ctypes.data, bad.ctypes.data, d, 1,
                              1 << 20, None) == tide.TIDE_OK              # nothing to append


def test_fused_decode_append_validation_without_gpu():
    lib = tide.load()
    one = np.array([1], np.int32)
    bad = np.array([0], np.int32)
    d = ctypes.byref(GOOD)
    f = lib.tide_decode_append_attn
    # (q, k_new, v_new, k_pool, v_pool, num_pages, bt, bt_stride, n, kv_lens, dims, splits,
    #  out, lse, ws, ws_bytes, stream)
    assert f(1, 1, 1, 1, 1, 10, 1, 4, 1, bad.ctypes.data, d, 0, 1, None, 1, 1 << 20,
             None) == tide.TIDE_ERR_INVALID_ARG                            # kv_len 0
    assert f(1, None, 1, 1, 1, 10, 1, 4, 1, one.ctypes.data, d, 0, 1, None, 1, 1 << 20,
             None) == tide.TIDE_ERR_INVALID_ARG                            # no k_new
    assert f(1, 1, None, 1, 1, 10, 1, 4, 1, one.ctypes.data, d, 0, 1, None, 1, 1 << 20,
             None) == tide.TIDE_ERR_INVALID_ARG                            # no v_new
    assert f(1, 1, 1, 1, 1, 10, 1, 4, 0, None, d, 0, 1, None, 1, 0, None) == tide.TIDE_OK
    assert f(1, 1, 1, 1, 1, 10, 1, 4, 1, np.array([65], np.int32).ctypes.data, d, 0, 1, None, 1,
             1 << 20, None) == tide.TIDE_ERR_CAPACITY                       # 5 pages > 4
    assert f(1, 1, 1, 1, 1, 10, 1, 4, 1, one.ctypes.data, d, 0, 1, None, 1, 16,
             None) == tide.TIDE_ERR_CAPACITY                                # workspace too small


def test_binding_rejects_host_tensors():
    import torch
    q = torch.zeros(4, 8, 64, dtype=torch.bfloat16)
    with pytest.raises((ValueError, TypeError)):
        tide.tide_extend_attn(q, q, q, q, [1], [1], _lib.make_dims(8, 2, 64, 0.1), q)


# ---- shared-prefix decode -------------------------------------------------------------------
def _ws_shared(kv, gs, sh, dims, splits=0):
    return _lib.tide_workspace_size_shared(kv, gs, sh, dims, splits)


def test_shared_decode_validation():
    dims = tide.make_dims(32, 8, 128, 1.0 / math.sqrt(128))
    kv = [100, 120, 80, 300]
    ok = _ws_shared(kv, [0, 2, 3, 4], [64, 48, 0], dims)
    assert ok > 0
    bad_tables = [
        ([1, 2, 3, 4], [64, 48, 0]),   # does not start at 0
        ([0, 2, 3, 3], [64, 48, 0]),   # empty group / does not end at num_tasks
        ([0, 3, 2, 4], [64, 48, 0]),   # not increasing
        ([0, 2, 3, 4], [60, 48, 0]),   # shared length not a page multiple
        ([0, 2, 3, 4], [112, 48, 0]),  # shared beyond kv_len - 1 of task 0 (100)
        ([0, 2, 3, 4], [64, 80, 0]),   # shared == kv_len of task 2: the decoded token is its own
        ([0, 2, 3, 4], [64, -16, 0]),  # negative
    ]
    for gs, sh in bad_tables:
        with pytest.raises(tide.TideError) as e:
            _ws_shared(kv, gs, sh, dims)
        assert e.value.status == tide.TIDE_ERR_INVALID_ARG, (gs, sh)
    with pytest.raises(ValueError):
        _ws_shared(kv, [0, 4], [0, 0], dims)  # group_start must be one longer than shared_lens


def test_shared_decode_workspace_covers_splits():
    """With nothing shared, the shared-prefix plan has the plain decode's split count, so
    its workspace is the plain one plus the larger work items."""
    dims = tide.make_dims(32, 8, 128, 1.0 / math.sqrt(128))
    rng = np.random.default_rng(5)
    kv = rng.integers(1, 5000, size=37)
    rc, plain = _ws(tide.TIDE_OP_DECODE, kv, None, dims)
    assert rc == tide.TIDE_OK
    shared0 = _ws_shared(kv, np.arange(38), np.zeros(37, np.int32), dims)
    assert shared0 >= plain
    # a shared prefix adds at most one split per task
    gs = [0, 10, 20, 37]
    sh = [min(kv[0:10].min() - 1, 1024) // 16 * 16, min(kv[10:20].min() - 1, 512) // 16 * 16, 0]
    assert _ws_shared(kv, gs, sh, dims) > 0


def test_shared_decode_rejects_before_gpu():
    """Argument errors are reported without any device work (this runs on the CPU)."""
    lib = tide.load()
    dims = tide.make_dims(32, 8, 128, 1.0 / math.sqrt(128))
    kv = np.array([40, 50], np.int32)
    gs = np.array([0, 2], np.int32)
    sh = np.array([48], np.int32)  # 48 > 40 - 1
    rc = lib.tide_decode_attn_shared(None, None, None, 10, None, 4, 2, kv.ctypes.data, 1,
                                     gs.ctypes.data, sh.ctypes.data, ctypes.byref(dims), 0, None,
                                     None, None, 0, None)
    assert rc == tide.TIDE_ERR_INVALID_ARG
    rc = lib.tide_decode_attn_shared(None, None, None, 10, None, 4, 0, None, 0, None, None,
                                     ctypes.byref(dims), 0, None, None, None, 0, None)
    assert rc == tide.TIDE_OK  # no tasks: nothing to do


# ---- decode without allocation ---------------------------------------------------------------
def test_noalloc_decode_validation_without_gpu():
    """tide_decode_attn_noalloc rejects bad arguments, and plans larger than its static
    scratch, before any device work."""
    lib = tide.load()
    f = lib.tide_decode_attn_noalloc
    d = ctypes.byref(GOOD)
    one = np.array([1], np.int32)
    bad = np.array([0], np.int32)
    # (q, k_pool, v_pool, num_pages, bt, bt_stride, n, kv_lens, dims, splits, out, lse, stream)
    assert f(1, 1, 1, 10, 1, 4, 1, bad.ctypes.data, d, 0, 1, None, None) == tide.TIDE_ERR_INVALID_ARG
    assert f(1, 1, 1, 10, 1, 4, 0, None, d, 0, 1, None, None) == tide.TIDE_OK
    assert f(None, 1, 1, 10, 1, 4, 1, one.ctypes.data, d, 0, 1, None, None) == tide.TIDE_ERR_INVALID_ARG
    assert f(1, 1, 1, 10, 1, 4, 1, one.ctypes.data, d, -1, 1, None, None) == tide.TIDE_ERR_INVALID_ARG
    assert f(1, 1, 1, 10, 1, 4, 1, np.array([65], np.int32).ctypes.data, d, 0, 1, None,
             None) == tide.TIDE_ERR_CAPACITY                                # 5 pages > 4
    # a plan whose partials exceed the static scratch
    big = np.full(4096, 32768, np.int32)
    rc, need = _ws(tide.TIDE_OP_DECODE, big, None, GOOD, splits=64)
    assert rc == tide.TIDE_OK and need > _lib.NOALLOC_SCRATCH_BYTES
    assert f(1, 1, 1, 10, 1, 2048, 4096, big.ctypes.data, d, 64, 1, None,
             None) == tide.TIDE_ERR_CAPACITY


def test_noalloc_scratch_size_matches_header():
    text = open(HEADERS[0]).read()
    m = re.search(r"#define TIDE_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == _lib.NOALLOC_SCRATCH_BYTES


# ---- binding: shapes are checked before the C call --------------------------------------------
def test_binding_checks_row_counts_before_the_call():
    """The C ABI takes no buffer sizes, so the binding checks every tensor against the host
    lengths first; a mismatch is a ValueError naming the tensor, never a device access.
    (Host tensors of the right shape would be rejected next, for not being on a device.)"""
    import torch
    dims = _lib.make_dims(8, 2, 64, 0.125)
    kp = torch.zeros(10, 2, 16, 64, dtype=torch.bfloat16)
    vp = torch.zeros(10, 2, 16, 64, dtype=torch.bfloat16)
    bt = torch.zeros(2, 4, dtype=torch.int32)
    q = torch.zeros(7, 8, 64, dtype=torch.bfloat16)    # 3 + 4 rows
    with pytest.raises(ValueError, match="q must have shape"):
        tide.tide_extend_attn(q[:6], kp, vp, bt, [5, 9], [3, 4], dims, q)
    with pytest.raises(ValueError, match="out must have shape"):
        tide.tide_extend_attn(q, kp, vp, bt, [5, 9], [3, 4], dims, q[:5])
    with pytest.raises(ValueError, match="lse must have shape"):
        tide.tide_extend_attn(q, kp, vp, bt, [5, 9], [3, 4], dims, q,
                              lse=torch.zeros(7, 4, dtype=torch.float32))
    with pytest.raises(ValueError, match="block_table has 1 rows"):
        tide.tide_extend_attn(q, kp, vp, bt[:1], [5, 9], [3, 4], dims, q)
    with pytest.raises(ValueError, match="q must have shape"):
        tide.tide_full_prefill_attn(q, kp, vp, bt, [3, 5], dims, q)
    kn = torch.zeros(7, 2, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="v_new must have shape"):
        tide.tide_kv_append(kn, kn[:, :1], kp, vp, bt, [5, 9], [3, 4], dims, None)
    with pytest.raises(ValueError, match="one entry per task"):
        tide.tide_kv_append(kn, kn, kp, vp, bt, [5, 9, 1], [3, 4], dims, None)
    qd = torch.zeros(2, 8, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="q must have shape"):
        tide.tide_decode_attn(qd[:1], kp, vp, bt, [6, 10], dims, qd)
    with pytest.raises(ValueError, match="k_new must have shape"):
        tide.tide_decode_append_attn(qd, kn, kn[:2], kp, vp, bt, [6, 10], dims, qd)
    with pytest.raises(ValueError, match="out must have shape"):
        tide.tide_decode_attn_noalloc(qd, kp, vp, bt, [6, 10], dims, qd[:, :4])
    with pytest.raises(ValueError, match="block_table has 2 rows"):
        tide.tide_decode_attn_shared(torch.zeros(3, 8, 64, dtype=torch.bfloat16), kp, vp, bt,
                                     [6, 10, 7], [0, 3], [0], dims,
                                     torch.zeros(3, 8, 64, dtype=torch.bfloat16))


def test_plan_info_matches_workspace_size_and_launch_rules():
    """tide_plan_info_get reports the same workspace as tide_workspace_size, 8-wave decode
    workgroups from 2,048 items on (4 below), and the in-kernel merge at <= 4 splits per
    task on average (no GPU needed: planning is host code)."""
    import paper_2608_10402_amd as tide
    dims = tide.make_dims(32, 8, 128, 0.088)
    for kv, waves in (([100] * 8, 4), ([5000] * 256, 8)):
        kv = np.asarray(kv, np.int32)
        info = tide.tide_plan_info_get(tide.TIDE_OP_DECODE, kv, None, dims)
        assert info["workspace_bytes"] == tide.tide_workspace_size(tide.TIDE_OP_DECODE, kv, None, dims)
        assert info["waves_per_group"] == waves
        assert info["merge_in_kernel"] == int(info["num_items"] <= 4 * kv.size * 8)
    one = tide.tide_plan_info_get(tide.TIDE_OP_DECODE, np.asarray([64] * 4, np.int32), None, dims,
                                  num_splits=1)
    many = tide.tide_plan_info_get(tide.TIDE_OP_DECODE, np.asarray([9000] * 4, np.int32), None,
                                   dims, num_splits=40)
    assert one["max_splits"] == 1 and one["merge_in_kernel"] == 1
    # 40 splits asked: chunks of ceil(9000 / 40) keys rounded up to 32 -> 256 -> 36 splits
    assert many["max_splits"] == 36 and many["merge_in_kernel"] == 0
    p, e = np.asarray([1000, 20], np.int32), np.asarray([300, 5], np.int32)
    info = tide.tide_plan_info_get(tide.TIDE_OP_EXTEND, p, e, dims)
    assert info["workspace_bytes"] == tide.tide_workspace_size(tide.TIDE_OP_EXTEND, p, e, dims)
    assert info["waves_per_group"] == 8 and info["num_items"] > 0
    with pytest.raises(tide.TideError):
        tide.tide_plan_info_get(tide.TIDE_OP_DECODE, np.asarray([0], np.int32), None, dims)
