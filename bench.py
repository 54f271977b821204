#!/usr/bin/env python3
"""Throughput of the batched multi-adapter LoRA delta on one MI355X.

Headline: decode step of 64 tokens on a 4096->4096 projection, 32 adapters of
ranks {8,16,32,64}, Zipf(1.1) adapter popularity, fp16 (the batched
heterogeneous-rank decode of Sections 2.3 C2 / 4.1).  One step = one pass of
the whole delta (plan already resident; shrink then expand) over the step's
batch, which the plan runs as ONE kernel launch (lora_step_kernel: the shrink
work items, then the expand work items, in one grid); ``value`` is the step's
algorithmic HBM bytes per second.  The prompt
workload (16 segments of U[64,1024] tokens, bf16) is timed the same way and
reported as tokens/s.

Timing: every step uses the next of R device copies of {adapters, x, y,
plan}, with R times the footprint above 512 MiB so that neither the 256 MB
Infinity Cache nor the L2s hold the previous step's data.  Steps are captured
in HIP graphs (one kernel launch per node, no memset or copy nodes) and
replayed between HIP events on the capturing stream, so the step kernel's
average launch duration is the timed region over the launches in it.  The
two-launch form (the shrink kernel, then the expand kernel) is captured and
timed the same way and reported beside it.

Prints exactly one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, datasheet

# HBM traffic of one step launch of the headline workload, from two rocprofv3
# --pmc passes (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch) scaled by the
# same counters on a plain 256 MiB device copy in the same run (FETCH_SIZE
# reads 131,088.8 KiB for 262,144 KiB read: x 1.99980; WRITE_SIZE reads
# 262,144.0 KiB: x 1.0).  Valid only for the kernel sources it was taken on
# (hash of csrc/*); reported as null otherwise.
MEASURED_TRAFFIC = {
    "sources_sha256_16": "2e0c8a031a8f851b",
    "workload": "decode_q4096_t64_mixed_rank_f16",
    "fetch_kib": 6707.1, "fetch_scale": 262144.0 / 131093.7,
    "write_kib": 732.9, "write_scale": 1.0,
}
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16/fp16
METRIC = "LoRA-delta HBM GB/s (% peak) at decode b=64 mixed rank; prefill tokens/s"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--workload", default="decode_mixed")
    ap.add_argument("--prefill-workload", default="prefill")
    ap.add_argument("--prefill-steps", type=int, default=40)
    ap.add_argument("--extra", default="decode_r8,llama13b_layer,llama70b_mixed,llama70b_mixed_tp4",
                    help="further named workloads timed the same way (comma-separated; empty for none)")
    ap.add_argument("--extra-steps", type=int, default=40)
    ap.add_argument("--base", default="prefill_base,prefill_base_l1024",
                    help="fused base projection workloads (Eq. 1 whole) timed with lora_base_apply")
    ap.add_argument("--base-steps", type=int, default=20)
    ap.add_argument("--costmodel-steps", type=int, default=96,
                    help="decode launches timed per point of the cost-model sweep (0: skip the sweep)")
    ap.add_argument("--no-coldstart", action="store_true", help="skip the cold-start measurements")
    ap.add_argument("--rotate-mib", type=float, default=640.0)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--calibrate-copy-mib", type=float, default=0.0,
                    help="also run one plain device copy of this many MiB (a known-traffic kernel "
                         "for scaling hardware byte counters)")
    return ap.parse_args()


class Rotation:
    """R device copies of one workload (stand-ins for R layers: their own
    adapter tables, x and y) sharing one plan per projection, as a serving
    loop shares the step's plan across all layers."""

    def __init__(self, w, copies, dev, stream):
        from paper_2401_11240_amd import device as D
        from paper_2401_11240_amd import lora as L
        self.L = L
        self.copies = [D.upload(w, dev, stream=stream) for _ in range(copies)]
        first = self.copies[0]
        self.plans = {p.name: L.lora_plan_create(p.table, first.batch, stream) for p in first.projections}
        # projections that share an input: one plan of all of them, one launch
        self.groups = shared_input_groups(w)
        self.multi = {k: L.lora_plan_create_multi([first.projections[i].table for i in ix], first.batch, stream)
                      for k, ix in self.groups.items() if len(ix) > 1}

    def step(self, c, stream, phase="apply"):
        """One pass of the delta over every projection of copy c ("multi":
        the projections that share an input in one launch each)."""
        L = self.L
        dw = self.copies[c]
        if phase == "multi":
            for key, ix in self.groups.items():
                ps = [dw.projections[i] for i in ix]
                x = dw.xs[key[0]]
                if len(ps) == 1:
                    p = ps[0]
                    L.lora_plan_apply(self.plans[p.name], p.table, x, x.shape[1], p.y, p.y.shape[1], stream)
                else:
                    L.lora_plan_apply_multi(self.multi[key], [p.table for p in ps], x, x.shape[1],
                                            [p.y for p in ps], [p.y.shape[1] for p in ps], stream)
            return
        for p in dw.projections:
            x = dw.xs[p.x]
            plan = self.plans[p.name]
            if phase == "apply":
                L.lora_plan_apply(plan, p.table, x, x.shape[1], p.y, p.y.shape[1], stream)
            elif phase == "shrink":
                L.lora_plan_shrink(plan, p.table, x, x.shape[1], stream)
            elif phase == "expand":
                L.lora_plan_expand(plan, p.table, p.y, p.y.shape[1], stream)

    def check_status(self, stream):
        """Raise if a step launch of any plan gave up waiting (its y would be
        invalid, so its time must not count as throughput)."""
        for h in list(self.plans.values()) + list(self.multi.values()):
            self.L.lora_plan_status(h, stream)

    def release(self):
        for h in list(self.plans.values()) + list(self.multi.values()):
            self.L.lora_plan_destroy(h)
        for dw in self.copies:
            dw.release()


MAX_PROJ_PER_LAUNCH = 4


def shared_input_groups(w):
    """The launches of a step when the projections that share an input run
    together, at most MAX_PROJ_PER_LAUNCH in one launch: {(x, k): [index]}."""
    by_x = {}
    for i, p in enumerate(w.projections):
        by_x.setdefault(p.x, []).append(i)
    out = {}
    for x, ix in by_x.items():
        for k in range(0, len(ix), MAX_PROJ_PER_LAUNCH):
            out[(x, k)] = ix[k:k + MAX_PROJ_PER_LAUNCH]
    return out


def footprint_bytes(w):
    n = sum(x.nbytes for x in w.xs.values())
    for p in w.projections:
        n += sum(a.nbytes for a in p.A) + sum(b.nbytes for b in p.B) + p.y.nbytes
    return n


def time_graph(torch, rot, n_steps, warmup, phase):
    """Capture one graph of R steps (one per copy) plus a tail graph, replay
    them so exactly n_steps steps run, and return the elapsed milliseconds."""
    R = len(rot.copies)
    s = torch.cuda.Stream()
    graphs = {}
    for count in sorted({R, n_steps % R} - {0}):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(s):
            for c in range(count):          # eager pass on the capture stream first
                rot.step(c, s, phase)
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=s):
                for c in range(count):
                    rot.step(c, s, phase)
        graphs[count] = g
    torch.cuda.synchronize()
    full, tail = divmod(n_steps, R)
    with torch.cuda.stream(s):
        for _ in range(max(1, math.ceil(warmup / R))):
            graphs[R].replay()
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record(s)
        for _ in range(full):
            graphs[R].replay()
        if tail:
            graphs[tail].replay()
        end.record(s)
    end.synchronize()
    torch.cuda.synchronize()
    rot.check_status(s)
    return float(start.elapsed_time(end))


def measure(torch, w, dev, steps, warmup, rotate_mib, label):
    from paper_2401_11240_amd import workloads as W
    fp = footprint_bytes(w)
    R = max(2, min(256, math.ceil(rotate_mib * 2 ** 20 / fp)))
    log(f"[{label}] {w.name}: footprint {fp / 2**20:.1f} MiB, {R} rotated copies")
    s0 = torch.cuda.current_stream(dev)
    rot = Rotation(w, R, dev, s0)
    torch.cuda.synchronize()
    ms = time_graph(torch, rot, steps, warmup, "apply")
    log(f"[{label}] {steps} steps in {ms:.3f} ms")
    ms_multi = time_graph(torch, rot, steps, warmup, "multi") if rot.multi else None
    if ms_multi is not None:
        log(f"[{label}] projections sharing an input in one launch: {ms_multi:.3f} ms")
    ms_shrink = time_graph(torch, rot, steps, warmup, "shrink")
    ms_expand = time_graph(torch, rot, steps, warmup, "expand")
    log(f"[{label}] shrink-only {ms_shrink:.3f} ms, expand-only {ms_expand:.3f} ms")
    rot.release()
    del rot
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    ra = w.row_adapter()
    used = np.unique(ra[ra >= 0])
    n_act = int((ra >= 0).sum())
    e = 2
    shrink_b = expand_b = 0
    seen = set()
    for p in w.projections:
        shrink_b += sum(int(w.ranks[g]) * p.h_in for g in used) * e
        if p.x not in seen:
            seen.add(p.x)
            shrink_b += n_act * p.h_in * e
        expand_b += sum(int(w.ranks[g]) * p.h_out for g in used) * e + n_act * 2 * p.h_out * e
    total_b = W.algorithmic_bytes(w)
    assert total_b == shrink_b + expand_b
    flops = W.algorithmic_flops(w)
    n_proj = len(w.projections)
    return dict(
        steps=steps, R=R, ms=ms, ms_per_step=ms / steps, bytes_per_step=total_b,
        flops_per_step=flops, gbps=total_b * steps / (ms * 1e-3) / 1e9,
        tokens_per_s=n_act * steps / (ms * 1e-3), n_active=n_act, distinct=int(used.size),
        shrink=dict(bytes=shrink_b, us=ms_shrink * 1e3 / (steps * n_proj)),
        expand=dict(bytes=expand_b, us=ms_expand * 1e3 / (steps * n_proj)),
        n_proj=n_proj, ms_multi=ms_multi,
    )


def plan_update_cost(torch, w, dev, n=400):
    """Host time of re-planning a step (lora_plan_update: grouping, work
    list, staging copy, enqueue of the upload and the arming fill) and the
    device time of that upload, alternating between the workload's batch and
    a second batch of the same size drawn with another seed."""
    from paper_2401_11240_amd import device as D
    from paper_2401_11240_amd import lora as L
    from paper_2401_11240_amd import workloads as W
    s = torch.cuda.current_stream(dev)
    dw = D.upload(w, dev, stream=s)
    p = dw.projections[0]
    rng = np.random.default_rng(12345)
    sa2 = rng.choice(w.n_adapters, size=w.seg_adapter.size, p=W.zipf_probs(w.n_adapters)).astype(np.int32)
    batches = [dw.batch, L.Batch(w.seg_offset, sa2, w.n_rows)]
    need = max(L.lora_plan_bytes(p.table, b) for b in batches)
    plan = L.lora_plan_create_reserved(p.table, batches[0], need, s)
    torch.cuda.synchronize()
    for i in range(20):
        L.lora_plan_update(plan, None, batches[i % 2], s)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(n):
        L.lora_plan_update(plan, None, batches[i % 2], s)
    host = (time.perf_counter() - t0) / n
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(s)
    for i in range(n):
        L.lora_plan_update(plan, None, batches[i % 2], s)
    ev1.record(s)
    ev1.synchronize()
    dev_us = ev0.elapsed_time(ev1) * 1e3 / n
    L.lora_plan_status(plan, s)
    L.lora_plan_destroy(plan)
    dw.release()
    return dict(plan_us=round(host * 1e6, 2), upload_and_arm_device_us=round(dev_us, 2),
                plan_bytes=need)


def measure_base(torch, name, dev, steps, rotate_mib):
    """Eq. 1 whole on R rotated copies of {x, W, adapters, y}: one base plan
    for the batch (lora_base_plan_create), and per step lora_base_plan_apply
    (the shrink into float32 v, its reduction, the MFMA GEMM with the delta in
    its epilogue, the reduction of split tiles), captured in a HIP graph and
    replayed between HIP events; the eager per-call form (lora_base_apply,
    which plans and uploads its work list every call) is timed beside it."""
    from paper_2401_11240_amd import device as D
    from paper_2401_11240_amd import lora as L
    from paper_2401_11240_amd import workloads as W
    w = W.BASE_NAMED[name]()
    p0 = w.projections[0]
    fp = footprint_bytes(w) + p0.W.nbytes
    R = max(2, min(16, math.ceil(rotate_mib * 2 ** 20 / fp)))
    log(f"[base] {w.name}: footprint {fp / 2**20:.1f} MiB, {R} rotated copies")
    s = torch.cuda.Stream(dev)
    copies = []
    for _ in range(R):
        dw = D.upload(w, dev, stream=s)
        wt = D.to_device_bits(np.ascontiguousarray(p0.W.T), dev)
        p = dw.projections[0]
        n = L.lora_base_workspace_bytes(p.table, dw.batch)
        ws = torch.empty(n, dtype=torch.uint8, device=dev)
        copies.append((dw, wt, ws, n))
    torch.cuda.synchronize()
    plan = L.lora_base_plan_create(copies[0][0].projections[0].table, copies[0][0].batch, s)

    def planned(c):
        dw, wt, _, _ = copies[c]
        p = dw.projections[0]
        x = dw.xs[p.x]
        L.lora_base_plan_apply(plan, p.table, x, x.shape[1], wt, wt.shape[1], p.y, p.y.shape[1], s)

    def eager(c):
        dw, wt, ws, n = copies[c]
        p = dw.projections[0]
        x = dw.xs[p.x]
        L.lora_base_apply(p.table, dw.batch, x, x.shape[1], wt, wt.shape[1], p.y, p.y.shape[1], ws, n, s)

    with torch.cuda.stream(s):
        for c in range(R):
            planned(c)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for c in range(R):
            planned(c)
    reps = max(1, math.ceil(steps / R))
    with torch.cuda.stream(s):
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(reps):
            g.replay()
        e1.record(s)
    e1.synchronize()
    ms = e0.elapsed_time(e1) / (reps * R)
    for i in range(R):
        eager(i)
    torch.cuda.synchronize()
    e0.record(s)
    for i in range(steps):
        eager(i % R)
    e1.record(s)
    e1.synchronize()
    ms_eager = e0.elapsed_time(e1) / steps
    del g
    L.lora_base_plan_destroy(plan)
    for dw, *_ in copies:
        dw.release()
    del copies
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    M, K, N = w.n_rows, p0.h_in, p0.h_out
    base_flops = 2 * M * K * N
    flops = base_flops + W.algorithmic_flops(w)
    tf = flops / (ms * 1e-3) / 1e12
    return {
        "workload": w.name, "tokens": M, "h_in": K, "h_out": N, "ms_per_step": ms,
        "tokens_per_s": round(M / (ms * 1e-3), 1), "TFLOPs": round(tf, 2),
        "pct_mfma_peak": round(100.0 * tf / MFMA_BF16_PEAK_TFLOPS, 2),
        "eager_ms_per_call": ms_eager,
        "algorithmic_flops_per_step": flops, "rotated_copies": R,
        "timing": "HIP graph replays of lora_base_plan_apply between HIP events (shrink into v, its reduction, "
                  "the fused GEMM, the split tiles' reduction)",
    }


def measure_coldstart(torch, dev, layers: int = 8, tokens: int = 1024, reps: int = 3):
    """Cold start (Sections 2.3 C1, 4.1, 4.2) on this GPU and its host:
    the sync-free hand-off of one layer's x (how long the launching thread is
    held, against a copy followed by a stream synchronisation); the load of a
    whole rank-64 adapter of a 7B-class model (32 layers x q, k, v, o at
    4096 -> 4096: 128 MiB) host -> device on a side stream, and the decode
    step's latency while it runs; a one-prompt batch of `tokens` tokens whose
    adapter is cold, over `layers` layers, with the load in flight (CPU
    assistance), waiting for it (on-demand loading), on the CPU only, and with
    the adapter resident."""
    from paper_2401_11240_amd import coldstart as CS
    from paper_2401_11240_amd import device as D
    from paper_2401_11240_amd import lora as L
    from paper_2401_11240_amd import workloads as W
    out = {}
    s = torch.cuda.Stream(dev)
    side = torch.cuda.Stream(dev)
    flags = CS.HostFlags(2)
    # hand-off of x [tokens, 4096] bf16
    h = 4096
    x = torch.randint(-30000, 30000, (tokens, h), dtype=torch.int16, device=dev)
    hx = torch.empty((tokens, h), dtype=torch.int16, pin_memory=True)
    torch.cuda.synchronize()
    held, lat, native = [], [], []
    for i in range(20):
        t0 = time.perf_counter()
        CS.handoff_x(x, h, tokens, h, hx, h, flags.addr(0), i + 1, s)
        t1 = time.perf_counter()
        CS.flag_wait(flags.addr(0), i + 1)
        t2 = time.perf_counter()
        held.append(t1 - t0)
        lat.append(t2 - t0)
        s.synchronize()
        t0 = time.perf_counter()
        with torch.cuda.stream(s):
            hx.copy_(x, non_blocking=True)
        s.synchronize()
        native.append(time.perf_counter() - t0)
    nb = tokens * h * 2
    out["handoff"] = {
        "bytes": nb,
        "host_held_us": round(1e6 * float(np.median(held)), 2),
        "signal_seen_us": round(1e6 * float(np.median(lat)), 2),
        "GBps": round(nb / float(np.median(lat)) / 1e9, 2),
        "native_copy_and_sync_host_held_us": round(1e6 * float(np.median(native)), 2),
    }
    del x, hx
    # a whole adapter's load on a side stream, and decode steps beside it
    nbytes = 32 * 4 * 64 * (4096 + 4096) * 2
    src = torch.empty(nbytes // 2, dtype=torch.int16).pin_memory()
    dst = torch.empty(nbytes // 2, dtype=torch.int16, device=dev)
    wd = W.NAMED["decode_mixed"]()
    dw = D.upload(wd, dev)
    p = dw.projections[0]
    plan = L.lora_plan_create(p.table, dw.batch, s)
    xd = dw.xs[p.x]
    n_dec = 200
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        L.lora_plan_apply(plan, p.table, xd, xd.shape[1], p.y, p.y.shape[1], s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        for _ in range(n_dec):
            L.lora_plan_apply(plan, p.table, xd, xd.shape[1], p.y, p.y.shape[1], s)
    with torch.cuda.stream(s):
        g.replay()
    torch.cuda.synchronize()

    def decode_us():
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(s):
            e0.record(s)
            g.replay()
            e1.record(s)
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e3 / n_dec

    alone = [decode_us() for _ in range(3)]
    loads, beside = [], []
    seq = 100
    for _ in range(3):
        seq += 1
        t0 = time.perf_counter()
        CS.adapter_load_async(dst, src, nbytes, flags.addr(1), seq, side)
        beside.append(decode_us())
        CS.flag_wait(flags.addr(1), seq)
        loads.append(time.perf_counter() - t0)
        torch.cuda.synchronize()
    L.lora_plan_status(plan, s)
    L.lora_plan_destroy(plan)
    dw.release()
    del g
    out["adapter_load"] = {
        "bytes": nbytes,
        "ms": round(1e3 * float(np.median(loads)), 3),
        "GBps": round(nbytes / float(np.median(loads)) / 1e9, 2),
        "decode_step_us_alone": round(float(np.median(alone)), 3),
        "decode_step_us_during_load": round(float(np.median(beside)), 3),
    }
    # a cold prompt over `layers` layers, at two prompt lengths
    rest = nbytes - layers * 64 * (4096 + 4096) * 2
    ballast = (src[: rest // 2], dst[: rest // 2])
    out["cold_prompt"] = {}
    for toks in (tokens, 128):
        ws = [W.build_workload(name=f"cold_prompt_l{i}", seed=200 + i, dtype=W.BF16, n_adapters=1,
                               fixed_ranks=[64], seg_adapter=[0], seg_lens=[toks],
                               projections=(("q_proj", 4096, 4096, "x"),), base_weight=True) for i in range(layers)]
        P = CS.ColdStartPrompt(torch, ws, cold=0, dev=dev, max_threads=16)
        res = {}
        for mode in ("gpu", "wait", "assist", "cpu", "assist_profiled"):
            ms, paths = [], None
            kw = {}
            if mode == "assist_profiled":
                # the profile: the CPU path's time per layer and the load's rate, both measured above
                kw = dict(cpu_layer_ms=res["cpu"]["ms"] / layers, load_gbps=out["adapter_load"]["GBps"],
                          gpu_layer_ms=res["gpu"]["ms"] / layers)
            for _ in range(reps):
                r = P.run(s, mode=mode.split("_")[0], side_stream=side, ballast=ballast, **kw)
                ms.append(r.ms)
                paths = r.paths
            res[mode] = {"ms": round(float(np.median(ms)), 3), "layers_on_cpu": paths.count("cpu")}
        P.release()
        out["cold_prompt"][f"tokens_{toks}"] = {"tokens": toks, "layers": layers, "rank": 64, "h": 4096,
                                                "dtype": "bf16", "load_bytes": nbytes, "cpu_threads": 16, **res}
    flags.free()
    del src, dst
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def sources_hash() -> str:
    import hashlib
    csrc = os.path.join(ROOT, "paper_2401_11240_amd", "csrc")
    h = hashlib.sha256()
    # the sources the step kernel and its planner are built from
    for f in ("lora_api.hip", "lora_internal.h", "lora_kernels.hip", "lora_device.h"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload_name):
    """HBM bytes per step launch from the counters, if they describe these sources."""
    m = MEASURED_TRAFFIC
    if m["workload"] != workload_name or m["sources_sha256_16"] != sources_hash():
        return None
    return int(round((m["fetch_kib"] * m["fetch_scale"] + m["write_kib"] * m["write_scale"]) * 1024))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, seconds):
    """The oracle as it stands, timed on full headline steps: with its OpenMP
    threads (rows spread over them), then with one thread, each for about
    half of ``seconds``."""
    import oracle
    from paper_2401_11240_amd import workloads as W

    def run(budget):
        reps = 0
        t0 = time.perf_counter()
        while True:
            for p in w.projections:
                oracle.lora_apply(w.seg_offset, w.seg_adapter, w.xs[p.x], p.A, p.B, w.ranks, w.scales,
                                  p.y, w.dtype)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget:
                return reps, el

    threads = oracle.num_threads()
    reps, el = run(seconds / 2)
    oracle.set_num_threads(1)
    reps1, el1 = run(seconds / 2)
    oracle.set_num_threads(threads)
    b = W.algorithmic_bytes(w)
    return dict(value=b * reps / el / 1e9, unit="GB/s", cores=threads, kind="oracle",
                sample=f"{reps} full steps of {w.name} (fp64 C oracle, OpenMP over rows, {threads} threads) "
                       f"in {el:.1f} s; {reps1} steps with 1 thread in {el1:.1f} s",
                ms_per_step=el * 1e3 / reps,
                one_thread={"value": b * reps1 / el1 / 1e9, "ms_per_step": el1 * 1e3 / reps1},
                affinity_cores=len(os.sched_getaffinity(0)), cpu_model=cpu_model())


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus > 1 or world > 1:
        if int(os.environ.get("RANK", "0")) == 0:
            log("bench.py measures one GPU only: the delta is data-parallel per GPU and this "
                "build runs no multi-GPU path; run with --gpus 1.")
        sys.exit(2)

    import torch
    from paper_2401_11240_amd import build as B
    from paper_2401_11240_amd import workloads as W
    if not os.path.exists(B.lib_path()):
        B.build()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    w = W.NAMED[args.workload]()
    dec = measure(torch, w, dev, args.steps, args.warmup, args.rotate_mib, "decode")
    step_us = dec["ms_per_step"] * 1e3 / dec["n_proj"]          # one step launch per projection
    step_bytes = dec["bytes_per_step"] // dec["n_proj"]
    achieved = step_bytes / (step_us * 1e-6) / 1e9
    out = {
        "metric": METRIC,
        "value": round(dec["gbps"], 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dec["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": W.DTYPE_NAMES[w.dtype],
        "data": "synthetic (seeded Llama-shaped workload; no datasets or weights)",
        "config": {
            "workload": w.name,
            "h_in": w.projections[0].h_in,
            "h_out": w.projections[0].h_out,
            "tokens": w.n_rows,
            "adapters": w.n_adapters,
            "distinct_adapters": dec["distinct"],
            "ranks": sorted(set(int(r) for r in w.ranks)),
            "adapter_law": "Zipf(1.1)",
            "rotated_copies": dec["R"],
            "algorithmic_bytes_per_step": dec["bytes_per_step"],
            "timing": "HIP graph replays between HIP events",
            "plan": "one plan per step shared by the rotated layer tables",
        },
        "pct_hbm_peak": round(100.0 * dec["gbps"] / HBM_PEAK_GBPS, 2),
        "roofline": {
            "kernel": "lora_step_kernel",
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": measured_traffic(w.name),
            "avg_launch_us": round(step_us, 3),
            "algorithmic_bytes_per_launch": step_bytes,
        },
        "two_launch": {
            "shrink_kernel_us": round(dec["shrink"]["us"], 3),
            "shrink_bytes": dec["shrink"]["bytes"] // dec["n_proj"],
            "expand_kernel_us": round(dec["expand"]["us"], 3),
            "expand_bytes": dec["expand"]["bytes"] // dec["n_proj"],
        },
    }
    log("[plan] re-planning cost")
    out["replan"] = plan_update_cost(torch, w, dev)
    out["replan"]["launches_sharing_one_plan"] = "every adapted projection of every layer with the same ranks"
    if not args.no_prefill:
        wp = W.NAMED[args.prefill_workload]()
        pre = measure(torch, wp, dev, args.prefill_steps, max(4, args.prefill_steps // 10),
                      args.rotate_mib, "prefill")
        out["prefill"] = {
            "workload": wp.name,
            "tokens_per_s": round(pre["tokens_per_s"], 1),
            "tokens_per_step": pre["n_active"],
            "ms_per_step": pre["ms_per_step"],
            "GBps": round(pre["gbps"], 2),
            "pct_hbm_peak": round(100.0 * pre["gbps"] / HBM_PEAK_GBPS, 2),
            "TFLOPs": round(pre["flops_per_step"] / (pre["ms_per_step"] * 1e-3) / 1e12, 3),
            "step_kernel_us": round(pre["ms_per_step"] * 1e3 / pre["n_proj"], 2),
            "two_launch_shrink_us": round(pre["shrink"]["us"], 2),
            "two_launch_expand_us": round(pre["expand"]["us"], 2),
            "algorithmic_bytes_per_step": pre["bytes_per_step"],
            "rotated_copies": pre["R"],
        }
    bases = [e for e in args.base.split(",") if e]
    if bases:
        out["base_fused"] = {}
    for name in bases:
        out["base_fused"][name] = measure_base(torch, name, dev, args.base_steps, args.rotate_mib)
    extras = [e for e in args.extra.split(",") if e]
    if extras:
        out["more"] = {}
    for name in extras:
        wx = W.NAMED[name]()
        mx = measure(torch, wx, dev, args.extra_steps, max(4, args.extra_steps // 10),
                     args.rotate_mib, name)
        out["more"][wx.name] = {
            "ms_per_step": mx["ms_per_step"],
            "us_per_launch": round(mx["ms_per_step"] * 1e3 / mx["n_proj"], 3),
            "GBps": round(mx["gbps"], 2),
            "pct_hbm_peak": round(100.0 * mx["gbps"] / HBM_PEAK_GBPS, 2),
            "tokens_per_step": mx["n_active"],
            "tokens_per_s": round(mx["tokens_per_s"], 1),
            "TFLOPs": round(mx["flops_per_step"] / (mx["ms_per_step"] * 1e-3) / 1e12, 3),
            "launches_per_step": mx["n_proj"],
            **({} if mx["ms_multi"] is None else {
                "shared_input_one_launch": {
                    "ms_per_step": mx["ms_multi"] / mx["steps"],
                    "GBps": round(mx["bytes_per_step"] / (mx["ms_multi"] / mx["steps"] * 1e-3) / 1e9, 2),
                    "pct_hbm_peak": round(100.0 * mx["bytes_per_step"] / (mx["ms_multi"] / mx["steps"] * 1e-3)
                                          / 1e9 / HBM_PEAK_GBPS, 2),
                    "launches_per_step": len(shared_input_groups(wx)),
                    "how": "lora_plan_apply_multi: the projections that share x (q/k/v, gate/up) in one grid"}}),
            "distinct_adapters": mx["distinct"],
            "algorithmic_bytes_per_step": mx["bytes_per_step"],
            "rotated_copies": mx["R"],
        }
        del wx
    if args.costmodel_steps > 0:
        from paper_2401_11240_amd import costmodel as CM
        log("[costmodel] decode sweep over batch sizes x rank mixes")
        pts = CM.decode_sweep(torch, dev, steps=args.costmodel_steps)
        fits = CM.fit(pts)
        log("[costmodel] prompt sweep")
        ppts = CM.prefill_sweep(torch, dev)
        pfits = CM.fit_prefill(ppts)
        log("[costmodel] simulating the routing policies")
        sims = {}
        for kind in ("sum_rank", "padded"):
            pre_m, dec_m = CM.serving_models(fits, kind, prefill_fit=pfits)
            sims[kind] = CM.simulate_policies(pre_m, dec_m)
            sims[kind]["models_ms"] = {"decode": list(dec_m.as_tuple()), "prefill": list(pre_m.as_tuple())}
        out["cost_model"] = {
            "projection": f"{CM.H_IN}->{CM.H_OUT} f16 decode step launch, one adapter per request",
            "fit_us": fits,
            "prefill_fit_us": pfits,
            "prefill_points": [{k: (round(v, 3) if isinstance(v, float) else v) for k, v in p.items()} for p in ppts],
            "points": [{k: (round(v, 3) if isinstance(v, float) else v) for k, v in p.items()} for p in pts],
            "simulation": sims,
        }
    if not args.no_coldstart:
        log("[coldstart] hand-off, adapter load, cold prompt")
        out["coldstart"] = measure_coldstart(torch, dev)
    if args.calibrate_copy_mib > 0:
        n = int(args.calibrate_copy_mib * 2 ** 20)
        src = torch.ones(n // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["calibration_copy_bytes"] = {"read": n, "write": n}
        del src, dst
    if not args.no_cpu_baseline:
        log("[cpu] timing the oracle")
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
