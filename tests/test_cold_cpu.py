"""Cold-start host code without a GPU: the CPU LoRA kernel (lora_cpu_delta)
against the oracle's unrounded delta, the same result for every split of the
rows over threads, and the host flag wait / test (lora_flag_wait,
lora_flag_test) on plain host memory.

Tolerance of the CPU delta: float32 sums of h_in products (x . A) and of r
products ((s v) . B) carry at most about (h_in + r) 2^-24 times
M = s sum_j (sum_k |x_k||A_kj|) |B_jn|; the check allows (h_in + r + 4) 2^-24 M."""
import ctypes as C
import os
import time

import numpy as np
import pytest

import oracle
from paper_2401_11240_amd import build as B
from paper_2401_11240_amd import workloads as W


@pytest.fixture(scope="module")
def CS():
    if not os.path.exists(B.lib_path()):
        B.build()
    from paper_2401_11240_amd import coldstart
    return coldstart


def one_adapter(seed, dtype, T, h_in, h_out, r):
    w = W.build_workload(name=f"cpu_{seed}", seed=seed, dtype=dtype, n_adapters=1, fixed_ranks=[r],
                         seg_adapter=[0], seg_lens=[T], projections=(("p", h_in, h_out, "x"),))
    return w


def cpu_delta(CS, w, tpt=0, threads=4, ld_delta=None):
    p = w.projections[0]
    x = np.ascontiguousarray(w.xs["x"])
    T, h_in = x.shape
    ld = ld_delta or p.h_out
    out = np.full((T, ld), np.nan, dtype=np.float32)
    A = np.ascontiguousarray(p.A[0])
    Bm = np.ascontiguousarray(p.B[0])
    CS.cpu_delta(x.ctypes.data, h_in, T, h_in, p.h_out, w.dtype, A.ctypes.data, Bm.ctypes.data, int(w.ranks[0]),
                 float(w.scales[0]), out.ctypes.data, ld, tpt, threads)
    return out[:, :p.h_out]


def reference(w):
    p = w.projections[0]
    T = w.n_rows
    zero = np.zeros((T, p.h_out), dtype=np.uint16)
    ref = oracle.lora_apply(w.seg_offset, w.seg_adapter, w.xs["x"], p.A, p.B, w.ranks, w.scales, zero, w.dtype)
    xa = np.abs(W.bits_to_f32(w.xs["x"], w.dtype).astype(np.float64))
    r = int(w.ranks[0])
    Aa = np.abs(W.bits_to_f32(p.A[0], w.dtype).astype(np.float64)).reshape(p.h_in, r)
    Ba = np.abs(W.bits_to_f32(p.B[0], w.dtype).astype(np.float64)).reshape(r, p.h_out)
    mag = float(w.scales[0]) * ((xa @ Aa) @ Ba)
    return ref, (p.h_in + r + 4) * 2.0 ** -24 * mag


@pytest.mark.parametrize("case", [(1, W.BF16, 37, 520, 264, 8), (2, W.F16, 130, 1032, 776, 64),
                                  (3, W.BF16, 1, 64, 8, 1), (4, W.F16, 300, 4096, 4096, 256)])
def test_cpu_delta_against_oracle(CS, case):
    seed, dt, T, h_in, h_out, r = case
    w = one_adapter(seed, dt, T, h_in, h_out, r)
    got = cpu_delta(CS, w)
    ref, bound = reference(w)
    err = np.abs(got.astype(np.float64) - ref)
    assert np.all(err <= bound), float(np.max(err / np.maximum(bound, 1e-300)))


def test_cpu_delta_same_for_every_thread_split(CS):
    w = one_adapter(5, W.BF16, 203, 512, 256, 32)
    base = cpu_delta(CS, w, tpt=0, threads=1)
    for tpt, thr in [(1, 16), (7, 3), (64, 16), (0, 5), (500, 8)]:
        got = cpu_delta(CS, w, tpt=tpt, threads=thr)
        assert np.array_equal(got, base), (tpt, thr)


def test_cpu_delta_leaves_padding_and_rejects_bad_arguments(CS):
    from paper_2401_11240_amd import lora as L
    w = one_adapter(6, W.F16, 9, 64, 16, 4)
    p = w.projections[0]
    x = np.ascontiguousarray(w.xs["x"])
    out = np.full((9, 24), 7.0, dtype=np.float32)
    CS.cpu_delta(x.ctypes.data, 64, 9, 64, 16, w.dtype, p.A[0].ctypes.data, p.B[0].ctypes.data, 4, 1.0,
                 out.ctypes.data, 24)
    assert np.all(out[:, 16:] == 7.0)
    for args, code in [((0, 64, 9, 64, 16, w.dtype, 0, 0, 4, 1.0, 0, 24), L.LORA_E_ARG),
                       ((x.ctypes.data, 64, 9, 64, 16, w.dtype, p.A[0].ctypes.data, p.B[0].ctypes.data, 0, 1.0,
                         out.ctypes.data, 24), L.LORA_E_RANK),
                       ((x.ctypes.data, 32, 9, 64, 16, w.dtype, p.A[0].ctypes.data, p.B[0].ctypes.data, 4, 1.0,
                         out.ctypes.data, 24), L.LORA_E_SHAPE),
                       ((x.ctypes.data, 64, 9, 64, 16, 5, p.A[0].ctypes.data, p.B[0].ctypes.data, 4, 1.0,
                         out.ctypes.data, 24), L.LORA_E_ARG)]:
        with pytest.raises(L.LoraError) as e:
            CS.cpu_delta(*args)
        assert e.value.code == code


def test_flag_wait_and_test_on_host_memory(CS):
    from paper_2401_11240_amd import lora as L
    f = np.zeros(2, dtype=np.uint32)
    a = f.ctypes.data
    assert not CS.flag_test(a, 1)
    f[0] = 5
    assert CS.flag_test(a, 5) and CS.flag_test(a, 3) and not CS.flag_test(a, 6)
    f[0] = 2
    assert CS.flag_test(a, 0xFFFFFFF0)          # sequence numbers wrap: 2 comes after 2^32 - 16
    t0 = time.perf_counter()
    with pytest.raises(L.LoraError) as e:
        CS.flag_wait(a, 9, timeout_ns=20_000_000)
    assert e.value.code == L.LORA_E_SYNC
    assert time.perf_counter() - t0 >= 0.015
    CS.flag_wait(a, 2, timeout_ns=0)
    with pytest.raises(L.LoraError):
        CS.flag_test(0, 1)
