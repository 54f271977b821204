"""Thin Python binding of liblora.so (the C ABI in include/lora.h).

Argument marshalling only: every step of the computation runs in the HIP
library.  Device buffers are passed as integer addresses or as objects with a
``data_ptr()`` method (torch tensors); streams as integer ``hipStream_t``
handles or objects with a ``cuda_stream`` attribute.  Failures raise
``LoraError`` carrying the library's code and message.  There is no fallback:
if the library is not built, loading it raises.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

import numpy as np

from . import build as _build

LORA_F16 = 0
LORA_BF16 = 1

LORA_OK = 0
LORA_E_ARG = -1
LORA_E_SHAPE = -2
LORA_E_RANK = -3
LORA_E_INDEX = -4
LORA_E_ALIGN = -5
LORA_E_NOMEM = -6
LORA_E_HIP = -7
LORA_E_WORKSPACE = -8
LORA_E_OVERLAP = -9
LORA_E_SYNC = -10
LORA_E_CAPTURE = -11
LORA_E_STALE = -12

# Every function the header declares (checked by the tests).
EXPORTS = (
    "lora_register_adapters", "lora_release_adapters", "lora_workspace_bytes", "lora_shrink",
    "lora_expand", "lora_apply_fused", "lora_plan_create", "lora_plan_apply", "lora_plan_destroy",
    "lora_plan_shrink", "lora_plan_expand", "lora_plan_status", "lora_plan_set_spin_limit",
    "lora_plan_bytes", "lora_plan_create_reserved", "lora_plan_update", "lora_apply_fused_static",
    "lora_plan_create_multi", "lora_plan_apply_multi",
    "lora_base_workspace_bytes", "lora_base_apply", "lora_base_plan_create", "lora_base_plan_apply",
    "lora_base_plan_destroy",
    "lora_group_rows", "lora_plan_inspect", "lora_base_inspect", "lora_last_error", "lora_abi_version",
)


class LoraError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"liblora error {code}: {message}")
        self.code = code
        self.message = message


class _Batch(C.Structure):
    _fields_ = [
        ("n_rows", C.c_int32),
        ("n_segments", C.c_int32),
        ("seg_offset", C.POINTER(C.c_int32)),
        ("seg_adapter", C.POINTER(C.c_int32)),
    ]


class Batch:
    """A step's batch: segments (offset, adapter); keeps its arrays alive."""

    def __init__(self, seg_offset, seg_adapter, n_rows: Optional[int] = None):
        self.seg_offset = np.ascontiguousarray(seg_offset, dtype=np.int32)
        self.seg_adapter = np.ascontiguousarray(seg_adapter, dtype=np.int32)
        if self.seg_offset.size == 0:
            self.seg_offset = np.zeros(1, dtype=np.int32)
        self.n_rows = int(self.seg_offset[-1]) if n_rows is None else int(n_rows)
        self._c = _Batch(self.n_rows, int(self.seg_adapter.shape[0]),
                         self.seg_offset.ctypes.data_as(C.POINTER(C.c_int32)),
                         self.seg_adapter.ctypes.data_as(C.POINTER(C.c_int32)))

    @property
    def c(self):
        return C.byref(self._c)


_lib = None


def load():
    """Load the in-tree liblora.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    path = _build.lib_path()
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run __graft_entry__.build() first")
    lib = C.CDLL(path)
    vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    i32p = C.POINTER(C.c_int32)
    f32p = C.POINTER(C.c_float)
    sig = {
        "lora_register_adapters": [C.POINTER(vp), C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                                   C.POINTER(vp), C.POINTER(vp), i32p, f32p, vp],
        "lora_release_adapters": [vp],
        "lora_workspace_bytes": [vp, C.POINTER(_Batch), C.POINTER(sz)],
        "lora_shrink": [vp, C.POINTER(_Batch), vp, i64, vp, i64, vp, sz, vp],
        "lora_expand": [vp, C.POINTER(_Batch), vp, i64, vp, i64, vp, sz, vp],
        "lora_apply_fused": [vp, C.POINTER(_Batch), vp, i64, vp, i64, vp, sz, vp],
        "lora_apply_fused_static": [vp, C.POINTER(_Batch), vp, i64, vp, i64, vp],
        "lora_base_workspace_bytes": [vp, C.POINTER(_Batch), C.POINTER(sz)],
        "lora_base_apply": [vp, C.POINTER(_Batch), vp, i64, vp, i64, vp, i64, vp, sz, vp],
        "lora_base_plan_create": [C.POINTER(vp), vp, C.POINTER(_Batch), vp],
        "lora_base_plan_apply": [vp, vp, vp, i64, vp, i64, vp, i64, vp],
        "lora_base_plan_destroy": [vp],
        "lora_plan_create": [C.POINTER(vp), vp, C.POINTER(_Batch), vp],
        "lora_plan_bytes": [vp, C.POINTER(_Batch), C.POINTER(sz)],
        "lora_plan_create_reserved": [C.POINTER(vp), vp, C.POINTER(_Batch), sz, vp],
        "lora_plan_update": [vp, vp, C.POINTER(_Batch), vp],
        "lora_plan_apply": [vp, vp, vp, i64, vp, i64, vp],
        "lora_plan_create_multi": [C.POINTER(vp), i32, C.POINTER(vp), C.POINTER(_Batch), vp],
        "lora_plan_apply_multi": [vp, C.POINTER(vp), vp, i64, C.POINTER(vp), C.POINTER(i64), vp],
        "lora_plan_destroy": [vp],
        "lora_plan_shrink": [vp, vp, vp, i64, vp],
        "lora_plan_expand": [vp, vp, vp, i64, vp],
        "lora_plan_status": [vp, vp],
        "lora_plan_set_spin_limit": [vp, i32],
        "lora_group_rows": [C.POINTER(_Batch), i32, i32p, i32p, i32p, i32p],
        "lora_plan_inspect": [C.POINTER(_Batch), i32, i32, i32, i32p, i32, vp, i32, i32p],
        "lora_base_inspect": [C.POINTER(_Batch), i32, i32, i32, i32p, i32, i32, vp],
        "lora_last_error": [],
        "lora_abi_version": [],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = C.c_int
    lib.lora_last_error.restype = C.c_char_p
    _lib = lib
    return lib


def _addr(p) -> int:
    if p is None:
        return 0
    if hasattr(p, "data_ptr"):
        return int(p.data_ptr())
    return int(p)


def _stream(s) -> int:
    if s is None:
        return 0
    if hasattr(s, "cuda_stream"):
        return int(s.cuda_stream)
    return int(s)


def _check(rc: int):
    if rc != LORA_OK:
        raise LoraError(rc, lora_last_error())


def lora_last_error() -> str:
    return load().lora_last_error().decode()


def lora_abi_version() -> int:
    return int(load().lora_abi_version())


def lora_register_adapters(device: int, h_in: int, h_out: int, dtype: int, A_ptrs: Sequence,
                           B_ptrs: Sequence, ranks: Sequence[int], scales: Sequence[float],
                           stream=None) -> int:
    n = len(ranks)
    A = (C.c_void_p * max(1, n))(*[_addr(p) for p in A_ptrs])
    B = (C.c_void_p * max(1, n))(*[_addr(p) for p in B_ptrs])
    r = np.ascontiguousarray(ranks, dtype=np.int32)
    s = np.ascontiguousarray(scales, dtype=np.float32)
    out = C.c_void_p()
    _check(load().lora_register_adapters(C.byref(out), device, h_in, h_out, dtype, n, A, B,
                                         r.ctypes.data_as(C.POINTER(C.c_int32)),
                                         s.ctypes.data_as(C.POINTER(C.c_float)), _stream(stream)))
    return out.value


def lora_release_adapters(table: int) -> None:
    _check(load().lora_release_adapters(table))


def lora_workspace_bytes(table: int, batch: Batch) -> int:
    out = C.c_size_t()
    _check(load().lora_workspace_bytes(table, batch.c, C.byref(out)))
    return int(out.value)


def lora_shrink(table: int, batch: Batch, x, ldx: int, v, ldv: int, ws, ws_bytes: int,
                stream=None) -> None:
    _check(load().lora_shrink(table, batch.c, _addr(x), ldx, _addr(v), ldv, _addr(ws), ws_bytes,
                              _stream(stream)))


def lora_expand(table: int, batch: Batch, v, ldv: int, y, ldy: int, ws, ws_bytes: int,
                stream=None) -> None:
    _check(load().lora_expand(table, batch.c, _addr(v), ldv, _addr(y), ldy, _addr(ws), ws_bytes,
                              _stream(stream)))


def lora_apply_fused(table: int, batch: Batch, x, ldx: int, y, ldy: int, ws, ws_bytes: int,
                     stream=None) -> None:
    _check(load().lora_apply_fused(table, batch.c, _addr(x), ldx, _addr(y), ldy, _addr(ws),
                                   ws_bytes, _stream(stream)))


def lora_apply_fused_static(table: int, batch: Batch, x, ldx: int, y, ldy: int, stream=None) -> None:
    """lora_apply_fused with the library's static scratch instead of a workspace."""
    _check(load().lora_apply_fused_static(table, batch.c, _addr(x), ldx, _addr(y), ldy, _stream(stream)))


def lora_base_workspace_bytes(table: int, batch: Batch) -> int:
    out = C.c_size_t()
    _check(load().lora_base_workspace_bytes(table, batch.c, C.byref(out)))
    return int(out.value)


def lora_base_apply(table: int, batch: Batch, x, ldx: int, wt, ldw: int, y, ldy: int, ws, ws_bytes: int,
                    stream=None) -> None:
    """y = round(x . W + s_g (x . A_g) . B_g); ``wt`` is W transposed, [h_out, ldw]."""
    _check(load().lora_base_apply(table, batch.c, _addr(x), ldx, _addr(wt), ldw, _addr(y), ldy, _addr(ws),
                                  ws_bytes, _stream(stream)))


def lora_base_plan_create(table: int, batch: Batch, stream=None) -> int:
    out = C.c_void_p()
    _check(load().lora_base_plan_create(C.byref(out), table, batch.c, _stream(stream)))
    return int(out.value or 0)


def lora_base_plan_apply(plan: int, table, x, ldx: int, wt, ldw: int, y, ldy: int, stream=None) -> None:
    _check(load().lora_base_plan_apply(plan, table or 0, _addr(x), ldx, _addr(wt), ldw, _addr(y), ldy,
                                       _stream(stream)))


def lora_base_plan_destroy(plan: int) -> None:
    _check(load().lora_base_plan_destroy(plan))


def lora_plan_create(table: int, batch: Batch, stream=None) -> int:
    out = C.c_void_p()
    _check(load().lora_plan_create(C.byref(out), table, batch.c, _stream(stream)))
    return out.value


def lora_plan_bytes(table: int, batch: Batch) -> int:
    out = C.c_size_t()
    _check(load().lora_plan_bytes(table, batch.c, C.byref(out)))
    return int(out.value)


def lora_plan_create_reserved(table: int, batch: Batch, min_bytes: int, stream=None) -> int:
    out = C.c_void_p()
    _check(load().lora_plan_create_reserved(C.byref(out), table, batch.c, int(min_bytes), _stream(stream)))
    return out.value


def lora_plan_update(plan: int, table, batch: Batch, stream=None) -> None:
    """Re-plan ``batch`` into the plan's memory (``table`` None = the plan's table)."""
    _check(load().lora_plan_update(plan, table or None, batch.c, _stream(stream)))


def lora_plan_apply(plan: int, table, x, ldx: int, y, ldy: int, stream=None) -> None:
    """``table`` None = the table the plan was made with."""
    _check(load().lora_plan_apply(plan, table or None, _addr(x), ldx, _addr(y), ldy, _stream(stream)))


def lora_plan_create_multi(tables, batch: Batch, stream=None) -> int:
    """One plan for projections that share x (their tables, in order)."""
    n = len(tables)
    T = (C.c_void_p * max(1, n))(*[int(t) for t in tables])
    out = C.c_void_p()
    _check(load().lora_plan_create_multi(C.byref(out), n, T, batch.c, _stream(stream)))
    return int(out.value or 0)


def lora_plan_apply_multi(plan: int, tables, x, ldx: int, ys, ldys, stream=None) -> None:
    """Every projection of a plan from lora_plan_create_multi, in one launch."""
    n = len(ys)
    T = (C.c_void_p * max(1, n))(*[int(t or 0) for t in tables])
    Y = (C.c_void_p * max(1, n))(*[_addr(y) for y in ys])
    LD = (C.c_int64 * max(1, n))(*[int(v) for v in ldys])
    _check(load().lora_plan_apply_multi(plan, T, _addr(x), ldx, Y, LD, _stream(stream)))


def lora_plan_shrink(plan: int, table, x, ldx: int, stream=None) -> None:
    _check(load().lora_plan_shrink(plan, table or None, _addr(x), ldx, _stream(stream)))


def lora_plan_expand(plan: int, table, y, ldy: int, stream=None) -> None:
    _check(load().lora_plan_expand(plan, table or None, _addr(y), ldy, _stream(stream)))


def lora_plan_destroy(plan: int) -> None:
    _check(load().lora_plan_destroy(plan))


def lora_plan_status(plan: int, stream=None) -> None:
    """Raise LoraError(LORA_E_SYNC) if a step launch of the plan gave up waiting."""
    _check(load().lora_plan_status(plan, _stream(stream)))


def lora_plan_set_spin_limit(plan: int, polls: int) -> None:
    _check(load().lora_plan_set_spin_limit(plan, int(polls)))


def lora_group_rows(batch: Batch, n_adapters: int):
    """(perm, group_off, group_adapter) of the library's host-side grouping."""
    T = max(1, batch.n_rows)
    perm = np.zeros(T, dtype=np.int32)
    goff = np.zeros(T + 1, dtype=np.int32)
    gad = np.zeros(T, dtype=np.int32)
    G = C.c_int32()
    p = lambda a: a.ctypes.data_as(C.POINTER(C.c_int32))
    _check(load().lora_group_rows(batch.c, n_adapters, p(perm), p(goff), p(gad), C.byref(G)))
    g = int(G.value)
    return perm[:int(goff[g])].copy(), goff[:g + 1].copy(), gad[:g].copy()


# lora_item_info_t, field for field
ITEM_INFO = np.dtype([("kind", np.int32), ("row_block", np.int32), ("rank", np.int32),
                      ("nrows", np.int32), ("lo", np.int32), ("len", np.int32), ("sub", np.int32),
                      ("nsplit", np.int32), ("pstride", np.int32), ("grid_pos", np.int32)])


# lora_base_info_t, field for field
BASE_INFO = np.dtype([("tile", np.int32), ("n_mt", np.int32), ("n_nt", np.int32), ("n_whole", np.int32),
                      ("split", np.int32), ("chunk", np.int32), ("n_stages", np.int32), ("stage_k", np.int32),
                      ("per_xcd", np.int32), ("grid", np.int32), ("panel", np.int32), ("pad", np.int32),
                      ("workspace_bytes", np.uint64)])


def lora_base_inspect(batch: Batch, h_in: int, h_out: int, ranks: Sequence[int], n_cu: int, n_xcd: int) -> dict:
    """The fused base GEMM's schedule for this batch (host only), as a dict
    with the fields of lora_base_info_t."""
    r = np.ascontiguousarray(ranks, dtype=np.int32)
    out = np.zeros(1, dtype=BASE_INFO)
    _check(load().lora_base_inspect(batch.c, h_in, h_out, len(r), r.ctypes.data_as(C.POINTER(C.c_int32)), n_cu,
                                    n_xcd, out.ctypes.data))
    return {k: int(out[0][k]) for k in BASE_INFO.names if k != "pad"}


def lora_plan_inspect(batch: Batch, h_in: int, h_out: int, ranks: Sequence[int], n_xcd: int = 1):
    """The work items of a plan of this batch (host only), as a structured
    array with the fields of lora_item_info_t."""
    r = np.ascontiguousarray(ranks, dtype=np.int32)
    n = C.c_int32()
    rp = r.ctypes.data_as(C.POINTER(C.c_int32))
    _check(load().lora_plan_inspect(batch.c, h_in, h_out, len(r), rp, n_xcd, None, 0, C.byref(n)))
    out = np.zeros(max(1, int(n.value)), dtype=ITEM_INFO)
    _check(load().lora_plan_inspect(batch.c, h_in, h_out, len(r), rp, n_xcd, out.ctypes.data, len(out),
                                    C.byref(n)))
    return out[:int(n.value)]
