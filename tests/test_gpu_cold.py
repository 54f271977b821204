"""Cold start on the GPU and its host (include/lora_coldstart.h):

  * the sync-free hand-off of x: the host sees the signal only with every
    byte of x in place (compared bit for bit), for several sizes in a row;
  * the asynchronous adapter load on a side stream: the device copy equals
    the host source once the signal is seen;
  * the merge kernel: y = round(y + delta) bit for bit against float32
    addition rounded to nearest-even on the host;
  * the CPU-assisted prompt over three layers in every mode (CPU until the
    load lands, all CPU, on-demand load, resident), each layer's output
    against the oracle's Eq. 1 (x W + s (x A) B) on every row.

Tolerance of a layer's rows that took the CPU path: the base projection is
rounded once on the GPU and again after the CPU delta is added, so they may
be off by half an ulp of x W plus half an ulp of the result, plus the float32
sums: h_in 2^-24 sum_k |x_k||W_kn| and (h_in + r + 4) 2^-24 M for the delta,
M = s sum_j (sum_k |x_k||A_kj|) |B_jn|.  Other rows: the base GEMM's bound
(tests/parity.py with the allowance of test_gpu_base.py)."""
import sys

import numpy as np
import pytest

import oracle
from paper_2401_11240_amd import workloads as W

from parity import compare, ulp

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():   # collected on CPU-only hosts, never run there
    pytest.skip("no GPU", allow_module_level=True)

from paper_2401_11240_amd import coldstart as CS  # noqa: E402
from paper_2401_11240_amd import device as D  # noqa: E402

DEV = torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def test_handoff_x_signal_follows_the_data():
    rng = np.random.default_rng(21)
    flags = CS.HostFlags(1)
    s = torch.cuda.Stream(DEV)
    try:
        for i, (T, h, ld) in enumerate([(300, 512, 520), (1, 8, 8), (0, 64, 64), (1024, 4096, 4096), (77, 264, 300)]):
            say(f"handoff {i}: rows {T} h {h} ldx {ld}")
            xs = rng.integers(0, 65536, size=(max(T, 1), ld), dtype=np.uint16)
            xd = D.to_device_bits(xs, DEV)
            host = torch.full((max(T, 1), h), -1, dtype=torch.int16, pin_memory=True)
            torch.cuda.synchronize()
            CS.handoff_x(xd, ld, T, h, host, h, flags.addr(0), i + 1, s)
            CS.flag_wait(flags.addr(0), i + 1, timeout_ns=10 ** 10)
            got = host.numpy().view(np.uint16)[:T]
            assert np.array_equal(got, xs[:T, :h])
            s.synchronize()
    finally:
        flags.free()


def test_adapter_load_async_on_a_side_stream():
    rng = np.random.default_rng(22)
    flags = CS.HostFlags(1)
    side = torch.cuda.Stream(DEV)
    try:
        n = 3 * 2 ** 20 + 24
        src = torch.from_numpy(rng.integers(-32768, 32767, size=n, dtype=np.int16)).pin_memory()
        dst = torch.zeros(n, dtype=torch.int16, device=DEV)
        torch.cuda.synchronize()
        CS.adapter_load_async(dst, src, 2 * n, flags.addr(0), 7, side)
        CS.flag_wait(flags.addr(0), 7, timeout_ns=10 ** 10)
        torch.cuda.current_stream(DEV).wait_stream(side)
        assert torch.equal(dst.cpu(), src)
    finally:
        flags.free()


@pytest.mark.parametrize("dtype", [W.BF16, W.F16])
def test_add_delta_bit_for_bit(dtype):
    rng = np.random.default_rng(23 + dtype)
    T, h, ldy, ldd = 123, 520, 528, 532
    y32 = rng.standard_normal((T, ldy)).astype(np.float32)
    yb = W.to_bits(y32, dtype)
    delta = (rng.standard_normal((T, ldd)) * 0.05).astype(np.float32)
    yd = D.to_device_bits(yb, DEV)
    dd = torch.from_numpy(delta).to(DEV)
    CS.add_delta(dd, ldd, yd, ldy, T, h, dtype, torch.cuda.current_stream(DEV))
    torch.cuda.synchronize()
    got = D.from_device_bits(yd)
    want = yb.copy()
    want[:, :h] = W.to_bits(W.bits_to_f32(yb[:, :h], dtype) + delta[:, :h], dtype)
    assert np.array_equal(got, want)


def layer_workloads(dtype, n_layers=3):
    # segments: a warm adapter, the cold one, rows without an adapter
    return [W.build_workload(name=f"cold_l{i}", seed=60 + i, dtype=dtype, n_adapters=2, fixed_ranks=[16, 64],
                             seg_adapter=[0, 1, -1], seg_lens=[200, 300, 50],
                             projections=(("p", 1024, 768, "x"),), base_weight=True) for i in range(n_layers)]


def check_layer(w, got_bits, path, cold_rows):
    p = w.projections[0]
    ref = oracle.base_lora_apply(w.seg_offset, w.seg_adapter, w.xs["x"], p.W, p.A, p.B, w.ranks, w.scales, w.dtype)
    xf = np.abs(W.bits_to_f32(w.xs["x"], w.dtype).astype(np.float64))
    Wf = W.bits_to_f32(p.W, w.dtype).astype(np.float64)
    xw_mag = xf @ np.abs(Wf)
    ra = w.row_adapter()
    # the delta's magnitude per row (0 for rows without an adapter)
    mag = np.zeros_like(ref)
    for g in (0, 1):
        rows = np.nonzero(ra == g)[0]
        r = int(w.ranks[g])
        Aa = np.abs(W.bits_to_f32(p.A[g], w.dtype).astype(np.float64)).reshape(p.h_in, r)
        Ba = np.abs(W.bits_to_f32(p.B[g], w.dtype).astype(np.float64)).reshape(r, p.h_out)
        mag[rows] = float(w.scales[g]) * ((xf[rows] @ Aa) @ Ba)
    lo, hi = cold_rows
    other = np.ones(w.n_rows, dtype=bool)
    if path == "cpu":
        other[lo:hi] = False
        got = W.bits_to_f32(got_bits[lo:hi], w.dtype).astype(np.float64)
        xw = W.bits_to_f32(w.xs["x"][lo:hi], w.dtype).astype(np.float64) @ Wf
        r = int(w.ranks[1])
        bound = (0.5 * ulp(ref[lo:hi], w.dtype) + 0.5 * ulp(xw, w.dtype) +
                 2.0 ** -24 * (p.h_in * xw_mag[lo:hi] + (p.h_in + r + 4) * mag[lo:hi]) * 1.01)
        err = np.abs(got - ref[lo:hi])
        assert np.all(np.isfinite(got))
        assert np.all(err <= bound), float(np.max(err / bound))
    allowance = p.h_in * 2.0 ** -10 * xw_mag[other] + mag[other]
    return compare(got_bits[other], ref[other], w.dtype, f"layer ({path})", mag=allowance)


@pytest.mark.parametrize("mode", ["cpu", "wait", "assist", "gpu"])
def test_cpu_assisted_prompt_every_layer_against_the_oracle(mode):
    dtype = W.BF16 if mode in ("cpu", "assist") else W.F16
    ws = layer_workloads(dtype)
    say(f"cold-start prompt, mode {mode}")
    P = CS.ColdStartPrompt(torch, ws, cold=1, dev=DEV, max_threads=8)
    s = torch.cuda.Stream(DEV)
    side = torch.cuda.Stream(DEV)
    try:
        if mode == "gpu":
            P.start_load(side)
            CS.flag_wait(P.flags.addr(0), P.seq_load)
            s.wait_event(P.load_event)
        res = P.run(s, mode=mode, side_stream=side)
        say(f"  paths {res.paths}, {res.ms:.2f} ms")
        if mode == "cpu":
            assert res.paths == ["cpu"] * len(ws)
        if mode in ("wait", "gpu"):
            assert res.paths == ["gpu"] * len(ws)
        for w, L_, path in zip(ws, P.layers, res.paths):
            got = D.from_device_bits(L_.dw.projections[0].y)
            st = check_layer(w, got, path, P.cold_rows)
            say("  ", path, st)
    finally:
        torch.cuda.synchronize()
        P.release()
