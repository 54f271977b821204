"""ctypes wrapper of the plain CPU oracle (oracle/lora_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product path.  Shares no code with
the HIP library; its only common ground with it is the seeded input module.

Every function here marshals numpy arrays into the C oracle and back; the
arithmetic itself is in lora_oracle.c (paper Section 2.1, Eq. 1; Section 2.2;
Section 2.3 C2 and Section 4.1 for the per-row adapter gather).
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "lora_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

F16, BF16 = 0, 1

_lib = None


def build(verbose: bool = False) -> str:
    """Compile liboracle.so with gcc: strict IEEE double, no FP contraction."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-Wextra", "-o", LIB + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB):
        build()
    lib = C.CDLL(LIB)
    i32p = C.POINTER(C.c_int32)
    u16p = C.POINTER(C.c_uint16)
    f64p = C.POINTER(C.c_double)
    f32p = C.POINTER(C.c_float)
    u16pp = C.POINTER(u16p)
    lib.oracle_round_one.restype = C.c_uint16
    lib.oracle_round_one.argtypes = [C.c_double, C.c_int]
    lib.oracle_widen.argtypes = [u16p, C.c_int, f64p, C.c_int64]
    lib.oracle_round.argtypes = [f64p, C.c_int, u16p, C.c_int64]
    lib.oracle_num_threads.restype = C.c_int
    lib.oracle_set_num_threads.restype = None
    lib.oracle_set_num_threads.argtypes = [C.c_int]
    lib.oracle_group_rows.restype = C.c_int32
    lib.oracle_group_rows.argtypes = [C.c_int32, C.c_int32, i32p, i32p, i32p, i32p, i32p]
    lib.oracle_lora_shrink.argtypes = [C.c_int32, C.c_int32, i32p, i32p, C.c_int32, C.c_int,
                                       u16p, C.c_int64, u16pp, i32p, f64p, C.c_int64]
    lib.oracle_lora_expand.argtypes = [C.c_int32, C.c_int32, i32p, i32p, C.c_int32, C.c_int,
                                       f32p, C.c_int64, u16pp, i32p, f32p, u16p, C.c_int64,
                                       f64p, C.c_int64]
    lib.oracle_lora_apply.restype = C.c_int
    lib.oracle_lora_apply.argtypes = [C.c_int32, C.c_int32, i32p, i32p, C.c_int32, C.c_int32,
                                      C.c_int, u16p, C.c_int64, u16pp, u16pp, i32p, f32p,
                                      C.c_int32, u16p, C.c_int64, f64p, C.c_int64]
    lib.oracle_lora_apply_row.restype = C.c_int
    lib.oracle_lora_apply_row.argtypes = [C.c_int32, C.c_int32, i32p, i32p, C.c_int32, C.c_int32,
                                          C.c_int, u16p, C.c_int64, u16pp, u16pp, i32p, f32p,
                                          u16p, C.c_int64, f64p]
    lib.oracle_base_lora_apply.restype = C.c_int
    lib.oracle_base_lora_apply.argtypes = [C.c_int32, C.c_int32, i32p, i32p, C.c_int32, C.c_int32,
                                           C.c_int, u16p, C.c_int64, u16p, C.c_int64, u16pp, u16pp,
                                           i32p, f32p, C.c_int32, f64p, C.c_int64]
    _lib = lib
    return lib


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(C.POINTER(ctype))


def _c16(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.uint16)


def _ptr_array(arrs: Sequence[np.ndarray]):
    """Array of uint16* pointing into the given (kept-alive) arrays."""
    keep = [_c16(a) for a in arrs]
    arr = (C.POINTER(C.c_uint16) * max(1, len(keep)))()
    for i, a in enumerate(keep):
        arr[i] = _ptr(a, C.c_uint16)
    return arr, keep


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads the following calls use (results do not depend on it)."""
    _load().oracle_set_num_threads(int(n))


def widen(bits: np.ndarray, dtype: int) -> np.ndarray:
    bits = _c16(bits)
    out = np.empty(bits.shape, dtype=np.float64)
    _load().oracle_widen(_ptr(bits, C.c_uint16), dtype, _ptr(out, C.c_double), bits.size)
    return out


def round_bits(vals: np.ndarray, dtype: int) -> np.ndarray:
    vals = np.ascontiguousarray(vals, dtype=np.float64)
    out = np.empty(vals.shape, dtype=np.uint16)
    _load().oracle_round(_ptr(vals, C.c_double), dtype, _ptr(out, C.c_uint16), vals.size)
    return out


def _segs(seg_offset, seg_adapter):
    so = np.ascontiguousarray(seg_offset, dtype=np.int32)
    sa = np.ascontiguousarray(seg_adapter, dtype=np.int32)
    assert so.shape[0] == sa.shape[0] + 1
    return so, sa


def group_rows(n_rows: int, seg_offset, seg_adapter):
    """(perm, group_off, group_adapter) of the stable first-appearance grouping."""
    so, sa = _segs(seg_offset, seg_adapter)
    perm = np.zeros(max(1, n_rows), dtype=np.int32)
    goff = np.zeros(max(1, n_rows) + 1, dtype=np.int32)
    gad = np.zeros(max(1, n_rows), dtype=np.int32)
    G = _load().oracle_group_rows(n_rows, sa.shape[0], _ptr(so, C.c_int32), _ptr(sa, C.c_int32),
                                  _ptr(perm, C.c_int32), _ptr(goff, C.c_int32),
                                  _ptr(gad, C.c_int32))
    n = int(goff[G])
    return perm[:n].copy(), goff[:G + 1].copy(), gad[:G].copy()


def lora_shrink(seg_offset, seg_adapter, x, A: Sequence[np.ndarray], ranks, dtype: int,
                ldv: Optional[int] = None) -> np.ndarray:
    """v[t, :r_g] = x[t] . A_g in double; rows without an adapter are NaN."""
    so, sa = _segs(seg_offset, seg_adapter)
    x = _c16(x)
    T, h_in = x.shape
    ranks = np.ascontiguousarray(ranks, dtype=np.int32)
    ldv = int(ldv or max(1, int(ranks.max()) if ranks.size else 1))
    v = np.full((T, ldv), np.nan, dtype=np.float64)
    Ap, keep = _ptr_array(A)
    _load().oracle_lora_shrink(T, sa.shape[0], _ptr(so, C.c_int32), _ptr(sa, C.c_int32), h_in,
                               dtype, _ptr(x, C.c_uint16), h_in, Ap, _ptr(ranks, C.c_int32),
                               _ptr(v, C.c_double), ldv)
    del keep
    return v


def lora_expand(seg_offset, seg_adapter, v: np.ndarray, B: Sequence[np.ndarray], ranks, scales,
                y: np.ndarray, dtype: int) -> np.ndarray:
    """out = y + s_g . v[t,:r_g] . B_g in double, from a float32 v."""
    so, sa = _segs(seg_offset, seg_adapter)
    v = np.ascontiguousarray(v, dtype=np.float32)
    y = _c16(y)
    T, h_out = y.shape
    ranks = np.ascontiguousarray(ranks, dtype=np.int32)
    scales = np.ascontiguousarray(scales, dtype=np.float32)
    out = np.empty((T, h_out), dtype=np.float64)
    Bp, keep = _ptr_array(B)
    _load().oracle_lora_expand(T, sa.shape[0], _ptr(so, C.c_int32), _ptr(sa, C.c_int32), h_out,
                               dtype, _ptr(v, C.c_float), v.shape[1], Bp, _ptr(ranks, C.c_int32),
                               _ptr(scales, C.c_float), _ptr(y, C.c_uint16), h_out,
                               _ptr(out, C.c_double), h_out)
    del keep
    return out


def lora_apply(seg_offset, seg_adapter, x, A, B, ranks, scales, y, dtype: int) -> np.ndarray:
    """out = y + s_g . (x . A_g) . B_g per row, in double (unrounded)."""
    so, sa = _segs(seg_offset, seg_adapter)
    x = _c16(x)
    y = _c16(y)
    T, h_in = x.shape
    h_out = y.shape[1]
    ranks = np.ascontiguousarray(ranks, dtype=np.int32)
    scales = np.ascontiguousarray(scales, dtype=np.float32)
    out = np.empty((T, h_out), dtype=np.float64)
    Ap, k1 = _ptr_array(A)
    Bp, k2 = _ptr_array(B)
    r_max = int(ranks.max()) if ranks.size else 1
    rc = _load().oracle_lora_apply(T, sa.shape[0], _ptr(so, C.c_int32), _ptr(sa, C.c_int32), h_in,
                                   h_out, dtype, _ptr(x, C.c_uint16), h_in, Ap, Bp,
                                   _ptr(ranks, C.c_int32), _ptr(scales, C.c_float), r_max,
                                   _ptr(y, C.c_uint16), h_out, _ptr(out, C.c_double), h_out)
    assert rc == 0
    del k1, k2
    return out


def lora_apply_rows(rows: Sequence[int], seg_offset, seg_adapter, x, A, B, ranks, scales, y,
                    dtype: int) -> np.ndarray:
    """Selected output rows only (sampled checks at full size)."""
    so, sa = _segs(seg_offset, seg_adapter)
    x = _c16(x)
    y = _c16(y)
    h_in = x.shape[1]
    h_out = y.shape[1]
    ranks = np.ascontiguousarray(ranks, dtype=np.int32)
    scales = np.ascontiguousarray(scales, dtype=np.float32)
    Ap, k1 = _ptr_array(A)
    Bp, k2 = _ptr_array(B)
    out = np.empty((len(rows), h_out), dtype=np.float64)
    lib = _load()
    for i, t in enumerate(rows):
        row = np.empty(h_out, dtype=np.float64)
        rc = lib.oracle_lora_apply_row(int(t), sa.shape[0], _ptr(so, C.c_int32),
                                       _ptr(sa, C.c_int32), h_in, h_out, dtype,
                                       _ptr(x, C.c_uint16), h_in, Ap, Bp, _ptr(ranks, C.c_int32),
                                       _ptr(scales, C.c_float), _ptr(y, C.c_uint16), h_out,
                                       _ptr(row, C.c_double))
        assert rc == 0
        out[i] = row
    del k1, k2
    return out


def base_lora_apply(seg_offset, seg_adapter, x, W, A, B, ranks, scales, dtype: int) -> np.ndarray:
    """out = x . W + s_g . (x . A_g) . B_g per row, in double (unrounded); W is
    [h_in, h_out] (the paper's H1 x H2 base weight)."""
    so, sa = _segs(seg_offset, seg_adapter)
    x = _c16(x)
    W = _c16(W)
    T, h_in = x.shape
    assert W.shape[0] == h_in, (W.shape, h_in)
    h_out = W.shape[1]
    ranks = np.ascontiguousarray(ranks, dtype=np.int32)
    scales = np.ascontiguousarray(scales, dtype=np.float32)
    out = np.empty((T, h_out), dtype=np.float64)
    Ap, k1 = _ptr_array(A)
    Bp, k2 = _ptr_array(B)
    r_max = int(ranks.max()) if ranks.size else 1
    rc = _load().oracle_base_lora_apply(T, sa.shape[0], _ptr(so, C.c_int32), _ptr(sa, C.c_int32), h_in,
                                        h_out, dtype, _ptr(x, C.c_uint16), h_in, _ptr(W, C.c_uint16), h_out,
                                        Ap, Bp, _ptr(ranks, C.c_int32), _ptr(scales, C.c_float), r_max,
                                        _ptr(out, C.c_double), h_out)
    del k1, k2
    if rc != 0:
        raise MemoryError("oracle_base_lora_apply")
    return out
