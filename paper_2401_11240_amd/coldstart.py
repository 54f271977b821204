"""Adapter cold start on one GPU and its host (include/lora_coldstart.h):
binding, and the CPU-assisted prompt driver of Section 4.1.

A prompt whose adapter is not on the GPU yet starts at once: the adapter's
factors are copied host -> device on a side stream (lora_adapter_load_async),
and until the copy's signal shows up, every layer runs the adapter's rows on
the CPU: the layer input is handed to the host without a host-side stream
synchronisation (lora_handoff_x, Section 4.2's asynchronous copy and signal),
the GPU computes the base projection of every row (a base plan of the batch
with the cold rows as rows without an adapter), the host cores compute x A B for the cold
rows (lora_cpu_delta, token slices over threads) while it runs, and the delta
is merged into y (lora_add_delta).  Once loaded, the GPU takes the adapter's
rows over (the fused base projection plus delta).  Marshalling and
orchestration only: every step of the arithmetic runs in liblora.so.
"""
from __future__ import annotations

import ctypes as C
import os
import time
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from . import lora as _lora

EXPORTS = ("lora_handoff_x", "lora_adapter_load_async", "lora_host_alloc", "lora_host_free", "lora_signal",
           "lora_flag_wait", "lora_flag_test", "lora_cpu_delta", "lora_add_delta")

_bound = None


def _lib():
    global _bound
    if _bound is not None:
        return _bound
    lib = _lora.load()
    vp, i32, i64, sz, u32 = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t, C.c_uint32
    u32p = C.POINTER(C.c_uint32)
    sig = {
        "lora_handoff_x": [vp, i64, i32, i32, vp, i64, vp, u32, vp],
        "lora_adapter_load_async": [vp, vp, sz, vp, u32, vp],
        "lora_host_alloc": [sz, C.POINTER(vp)],
        "lora_host_free": [vp],
        "lora_signal": [vp, u32, vp],
        "lora_flag_wait": [vp, u32, i64],
        "lora_flag_test": [vp, u32],
        "lora_cpu_delta": [vp, i64, i32, i32, i32, i32, vp, vp, i32, C.c_float, vp, i64, i32, i32],
        "lora_add_delta": [vp, i64, vp, i64, i32, i32, i32, vp],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = C.c_int
    _bound = lib
    return lib


_addr = _lora._addr
_stream = _lora._stream
_check = _lora._check


class HostFlags:
    """Pinned, coherent uint32 flags (lora_host_alloc), all starting at 0."""

    def __init__(self, n: int = 4):
        p = C.c_void_p()
        _check(_lib().lora_host_alloc(4 * n, C.byref(p)))
        self.ptr = int(p.value)
        self.n = n
        self.view = np.ctypeslib.as_array(C.cast(self.ptr, C.POINTER(C.c_uint32)), shape=(n,))
        self.view[:] = 0

    def addr(self, i: int) -> int:
        assert 0 <= i < self.n
        return self.ptr + 4 * i

    def free(self):
        if self.ptr:
            _check(_lib().lora_host_free(self.ptr))
            self.ptr = 0


def handoff_x(x, ldx: int, n_rows: int, h: int, host_x, ld_host: int, flag: int, value: int, stream=None) -> None:
    _check(_lib().lora_handoff_x(_addr(x), ldx, n_rows, h, _addr(host_x), ld_host, flag, value, _stream(stream)))


def adapter_load_async(dst, src_host, nbytes: int, flag: int, value: int, stream=None) -> None:
    _check(_lib().lora_adapter_load_async(_addr(dst), _addr(src_host), nbytes, flag, value, _stream(stream)))


def signal(flag: int, value: int, stream=None) -> None:
    _check(_lib().lora_signal(flag, value, _stream(stream)))


def flag_wait(flag: int, value: int, timeout_ns: int = 10 ** 10) -> None:
    _check(_lib().lora_flag_wait(flag, value, timeout_ns))


def flag_test(flag: int, value: int) -> bool:
    r = _lib().lora_flag_test(flag, value)
    if r < 0:
        raise _lora.LoraError(_lora.LORA_E_ARG, "lora_flag_test: NULL flag")
    return r == 1


def cpu_delta(x_host, ldx: int, n_rows: int, h_in: int, h_out: int, dtype: int, A_host, B_host, rank: int,
              scale: float, delta_host, ld_delta: int, tokens_per_thread: int = 0, max_threads: int = 16) -> None:
    _check(_lib().lora_cpu_delta(_addr(x_host), ldx, n_rows, h_in, h_out, dtype, _addr(A_host), _addr(B_host), rank,
                                 float(scale), _addr(delta_host), ld_delta, tokens_per_thread, max_threads))


def add_delta(delta, ld_delta: int, y, ldy: int, n_rows: int, h_out: int, dtype: int, stream=None) -> None:
    _check(_lib().lora_add_delta(_addr(delta), ld_delta, _addr(y), ldy, n_rows, h_out, dtype, _stream(stream)))


# ---------------------------------------------------------------------------
# CPU-assisted prompt over several layers
# ---------------------------------------------------------------------------

@dataclass
class Layer:
    """One adapted projection of one layer, resident on the device: the
    workload's x, y, W^T, adapter table (the cold adapter's device factors
    included, unfilled until loaded) and the base-projection workspace."""
    dw: object
    wt: object
    cold_A_dev: int = 0           # device address of the cold adapter's A in this layer
    cold_B_dev: int = 0
    cold_A_host: object = None    # pinned host copies (the load's source; the CPU path reads them)
    cold_B_host: object = None


@dataclass
class PromptResult:
    paths: List[str] = field(default_factory=list)     # "cpu" or "gpu" per layer
    ms: float = 0.0                                    # host wall time of the whole prompt
    load_seen_at_layer: int = -1


class ColdStartPrompt:
    """A prompt batch over n layers in which adapter `cold` starts on the host.

    `workloads` are seeded one-projection workloads with base weights, one per
    layer, sharing their segment structure.  The cold adapter's device factors
    are overwritten with NaN bit patterns until the load lands, so that any use
    of them before the switch shows in the output."""

    def __init__(self, torch, workloads, cold: int, dev, max_threads: int = 16, tokens_per_thread: int = 0):
        from . import device as D
        self.torch = torch
        self.dev = dev
        self.cold = cold
        self.max_threads = max_threads
        self.tokens_per_thread = tokens_per_thread
        self.ws = workloads
        w0 = workloads[0]
        self.dtype = w0.dtype
        self.rank = int(w0.ranks[cold])
        self.scale = float(w0.scales[cold])
        so, sa = w0.seg_offset, w0.seg_adapter
        segs = [(int(so[s]), int(so[s + 1])) for s in range(len(sa)) if int(sa[s]) == cold]
        if len(segs) != 1:
            raise ValueError("the cold adapter must own exactly one segment (one prompt) of the batch")
        self.cold_rows = segs[0]
        sa_cold = np.where(sa == cold, -1, sa).astype(np.int32)
        self.batch_cpu = _lora.Batch(so, sa_cold, w0.n_rows)
        self.layers: List[Layer] = []
        pin = dict(dtype=torch.int16, pin_memory=True)
        nan16 = 0x7E00 if self.dtype == 0 else 0x7FC0
        for w in workloads:
            dw = D.upload(w, dev)
            p = dw.projections[0]
            pr = w.projections[0]
            wt = D.to_device_bits(np.ascontiguousarray(pr.W.T), dev)
            A_h = torch.from_numpy(np.ascontiguousarray(pr.A[cold]).view(np.int16).ravel().copy()).pin_memory()
            B_h = torch.from_numpy(np.ascontiguousarray(pr.B[cold]).view(np.int16).ravel().copy()).pin_memory()
            # the device copies start as NaN: the GPU must not read them before the load
            a_off = (p.A_ptrs[cold] - p.A_buf.data_ptr()) // 2
            b_off = (p.B_ptrs[cold] - p.B_buf.data_ptr()) // 2
            p.A_buf[a_off:a_off + A_h.numel()].fill_(nan16)
            p.B_buf[b_off:b_off + B_h.numel()].fill_(nan16)
            self.layers.append(Layer(dw, wt, p.A_ptrs[cold], p.B_ptrs[cold], A_h, B_h))
        rows = max(1, self.cold_rows[1] - self.cold_rows[0])
        h_in = workloads[0].projections[0].h_in
        h_out = workloads[0].projections[0].h_out
        self.host_x = torch.empty((rows, h_in), **pin)
        self.host_delta = torch.empty((rows, h_out), dtype=torch.float32, pin_memory=True)
        self.dev_delta = torch.empty((rows, h_out), dtype=torch.float32, device=dev)
        # one base plan per batch form, shared by the layers (same shapes and ranks):
        # every adapter on the GPU, and the cold adapter's rows as rows without one
        t0 = self.layers[0].dw.projections[0].table
        self.plan_gpu = _lora.lora_base_plan_create(t0, self.layers[0].dw.batch)
        self.plan_cpu = _lora.lora_base_plan_create(t0, self.batch_cpu)
        self.flags = HostFlags(2)          # 0: the adapter load, 1: the hand-offs
        self.seq_x = 0
        self.seq_load = 0
        torch.cuda.synchronize()

    def release(self):
        self.torch.cuda.synchronize()
        _lora.lora_base_plan_destroy(self.plan_gpu)
        _lora.lora_base_plan_destroy(self.plan_cpu)
        for L_ in self.layers:
            L_.dw.release()
        self.flags.free()

    def start_load(self, side_stream, ballast=None):
        """Every layer's cold factors host -> device on side_stream; the flag
        reaches the returned value once all of them have landed.  ``ballast``
        (a pinned host tensor, a device tensor of the same bytes) is copied
        first: the rest of a whole adapter (the layers and projections this
        prompt does not run), so that the load takes as long as a real one."""
        self.load_bytes = sum(L_.cold_A_host.numel() * 2 + L_.cold_B_host.numel() * 2 for L_ in self.layers)
        self.load_started = time.perf_counter()
        if ballast is not None:
            src, dst = ballast
            self.load_bytes += src.numel() * src.element_size()
            self.seq_load += 1
            adapter_load_async(dst, src, src.numel() * src.element_size(), self.flags.addr(0), self.seq_load,
                               side_stream)
        for L_ in self.layers:
            self.seq_load += 1
            adapter_load_async(L_.cold_A_dev, L_.cold_A_host, L_.cold_A_host.numel() * 2, self.flags.addr(0),
                               self.seq_load, side_stream)
            self.seq_load += 1
            adapter_load_async(L_.cold_B_dev, L_.cold_B_host, L_.cold_B_host.numel() * 2, self.flags.addr(0),
                               self.seq_load, side_stream)
        ev = self.torch.cuda.Event()
        ev.record(side_stream)
        self.load_event = ev
        return self.seq_load

    def run(self, stream, mode: str = "assist", side_stream=None, ballast=None, cpu_layer_ms: float = None,
            load_gbps: float = None, gpu_layer_ms: float = None) -> PromptResult:
        """mode: "assist" (CPU until the load lands, then GPU), "cpu" (every
        layer on the CPU path), "gpu" (adapter already resident), "wait"
        (load, wait for it, then every layer on the GPU: on-demand loading).

        With a profile (cpu_layer_ms, the CPU path's time per layer, and
        load_gbps, the host -> device rate), "assist" starts a CPU layer only
        while the load's predicted remaining time exceeds it, and otherwise
        waits for the load: a CPU layer that would end after the adapter lands
        only delays the GPU's take-over.  With gpu_layer_ms too, it stays on
        the CPU for every remaining layer when that ends no later than
        waiting for the load and running them on the GPU."""
        torch = self.torch
        res = PromptResult()
        t0 = time.perf_counter()
        target = None
        if mode in ("assist", "wait"):
            target = self.start_load(side_stream, ballast)
            if mode == "wait":
                flag_wait(self.flags.addr(0), target)
                stream.wait_event(self.load_event)
        on_gpu = mode in ("gpu", "wait")
        for li, L_ in enumerate(self.layers):
            if not on_gpu and mode == "assist":
                landed = flag_test(self.flags.addr(0), target)
                if not landed and cpu_layer_ms and load_gbps:
                    left_ms = self.load_bytes / (load_gbps * 1e6) - (time.perf_counter() - self.load_started) * 1e3
                    remaining = len(self.layers) - li
                    stay = gpu_layer_ms is not None and \
                        remaining * cpu_layer_ms <= max(left_ms, 0.0) + remaining * gpu_layer_ms
                    if not stay and left_ms < cpu_layer_ms:
                        flag_wait(self.flags.addr(0), target)
                        landed = True
                if landed:
                    stream.wait_event(self.load_event)       # GPU-side order after the copies
                    on_gpu = True
                    res.load_seen_at_layer = li
            if on_gpu:
                self._layer_gpu(L_, stream)
                res.paths.append("gpu")
            else:
                self._layer_cpu(L_, stream)
                res.paths.append("cpu")
        torch.cuda.synchronize()
        res.ms = (time.perf_counter() - t0) * 1e3
        return res

    def _layer_gpu(self, L_, stream):
        p = L_.dw.projections[0]
        x = L_.dw.xs[p.x]
        _lora.lora_base_plan_apply(self.plan_gpu, p.table, x, x.shape[1], L_.wt, L_.wt.shape[1], p.y, p.y.shape[1],
                                   stream)

    def _layer_cpu(self, L_, stream):
        """Stream order per layer: hand-off of the cold rows' x and its signal,
        the base projection, the delta's upload, the merge.  The host waits
        for the hand-off's signal only, so the CPU computes the delta while the
        GPU runs the base projection; the next layer's signal comes after this
        layer's merge, which is what frees the host buffers for reuse."""
        p = L_.dw.projections[0]
        x = L_.dw.xs[p.x]
        h_in, h_out = x.shape[1], p.y.shape[1]
        lo, hi = self.cold_rows
        n = hi - lo
        self.seq_x += 1
        handoff_x(x.data_ptr() + 2 * lo * h_in, h_in, n, h_in, self.host_x, h_in, self.flags.addr(1), self.seq_x,
                  stream)
        _lora.lora_base_plan_apply(self.plan_cpu, p.table, x, h_in, L_.wt, L_.wt.shape[1], p.y, h_out, stream)
        flag_wait(self.flags.addr(1), self.seq_x)
        cpu_delta(self.host_x, h_in, n, h_in, h_out, self.dtype, L_.cold_A_host, L_.cold_B_host, self.rank,
                  self.scale, self.host_delta, h_out, self.tokens_per_thread, self.max_threads)
        with self.torch.cuda.stream(stream):
            self.dev_delta[:n].copy_(self.host_delta[:n], non_blocking=True)
        add_delta(self.dev_delta, h_out, p.y.data_ptr() + 2 * lo * h_out, h_out, n, h_out, self.dtype, stream)
