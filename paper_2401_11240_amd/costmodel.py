"""Profiling-based performance models and scheduling (Section 5) for this
library's kernels.

``decode_sweep`` times the single-launch decode step (lora_plan_apply) over a
grid of batch sizes and rank mixes, every request with its own adapter;
``fit`` fits the two linear models of Section 5 to it through the library
(lora_perf_fit): the padded form, linear in |S| * max rank, and the
padding-free form, linear in the sum of ranks; ``simulate_policies`` then runs
the library's continuous-batching simulator with Algorithm 1 and the three
baselines, on a synthetic Poisson / Zipf trace, with decode and prompt models
built from the fit.  Marshalling and timing only: the kernels, the fit and the
simulation run in liblora.so.
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence

import numpy as np

from . import sched as S
from . import workloads as W

# The decode projection of the sweep: 4096 -> 4096, binary16 (the shape of the
# decode workloads of the benchmark).
H_IN = H_OUT = 4096
BATCH_SIZES = (1, 4, 16, 32, 64, 128)
RANK_MIXES = {
    "r8": lambda b: [8] * b,
    "r16": lambda b: [16] * b,
    "r32": lambda b: [32] * b,
    "r64": lambda b: [64] * b,
    "mixed": lambda b: [(8, 16, 32, 64)[i % 4] for i in range(b)],
    "one64": lambda b: [64] + [8] * (b - 1),
}


def sweep_points(batch_sizes: Sequence[int] = BATCH_SIZES, mixes: Sequence[str] = tuple(RANK_MIXES)) -> List[Dict]:
    pts = []
    for b in batch_sizes:
        for m in mixes:
            pts.append(dict(batch=b, mix=m, ranks=RANK_MIXES[m](b)))
    return pts


def _workload(ranks: Sequence[int], seed: int, lens: Sequence[int] = None):
    b = len(ranks)
    return W.build_workload(name=f"sweep_b{b}", seed=seed, dtype=W.F16, n_adapters=b, fixed_ranks=list(ranks),
                            seg_adapter=list(range(b)), seg_lens=list(lens) if lens else [1] * b,
                            projections=(("q_proj", H_IN, H_OUT, "x"),))


# Prompt batches of the prefill sweep: (segments, tokens per segment); every
# segment its own adapter, ranks cycling 8/16/32/64.
PREFILL_POINTS = [(s, n) for s in (1, 2, 4, 8, 16) for n in (64, 256, 1024)]


def time_decode(torch, ranks: Sequence[int], dev, steps: int = 200, rotate_mib: float = 256.0,
                max_copies: int = 48, seed: int = 0, lens: Sequence[int] = None) -> float:
    """Microseconds per step launch of one batch (every request its own
    adapter; one token each unless `lens` gives the segments' lengths), from
    HIP graph replays over rotated copies of adapters, x and y."""
    from . import device as D
    from . import lora as L
    w = _workload(ranks, seed, lens)
    fp = sum(x.nbytes for x in w.xs.values()) + sum(
        sum(a.nbytes for a in p.A) + sum(b.nbytes for b in p.B) + p.y.nbytes for p in w.projections)
    R = max(2, min(max_copies, math.ceil(rotate_mib * 2 ** 20 / fp)))
    s = torch.cuda.Stream(dev)
    copies = [D.upload(w, dev, stream=s) for _ in range(R)]
    p0 = copies[0].projections[0]
    plan = L.lora_plan_create(p0.table, copies[0].batch, s)

    def one(c):
        p = copies[c].projections[0]
        x = copies[c].xs[p.x]
        L.lora_plan_apply(plan, p.table, x, x.shape[1], p.y, p.y.shape[1], s)

    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        for c in range(R):
            one(c)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for c in range(R):
            one(c)
    reps = max(1, steps // R)
    with torch.cuda.stream(s):
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(reps):
            g.replay()
        e1.record(s)
    e1.synchronize()
    L.lora_plan_status(plan, s)
    us = e0.elapsed_time(e1) * 1e3 / (reps * R)
    L.lora_plan_destroy(plan)
    for c in copies:
        c.release()
    del g
    torch.cuda.synchronize()
    return float(us)


def decode_sweep(torch, dev, points: Sequence[Dict] = None, steps: int = 200) -> List[Dict]:
    out = []
    for i, pt in enumerate(points or sweep_points()):
        us = time_decode(torch, pt["ranks"], dev, steps=steps, seed=i)
        reqs = [(r, 1) for r in pt["ranks"]]
        out.append(dict(batch=pt["batch"], mix=pt["mix"], us=us,
                        padded=S.perf_feature(S.PADDED, reqs), sum_rank=S.perf_feature(S.SUM_RANK, reqs)))
    return out


def prefill_sweep(torch, dev, steps: int = 40) -> List[Dict]:
    """The step launch on prompt batches (PREFILL_POINTS), for the prompt
    model: microseconds against the batch's tokens and sum of ranks."""
    out = []
    for i, (nseg, n) in enumerate(PREFILL_POINTS):
        ranks = [(8, 16, 32, 64)[j % 4] for j in range(nseg)]
        us = time_decode(torch, ranks, dev, steps=steps, seed=100 + i, lens=[n] * nseg, max_copies=16)
        reqs = [(r, n) for r in ranks]
        out.append(dict(segments=nseg, tokens_per_segment=n, us=us, tokens=S.perf_feature(S.TOKENS, reqs),
                        sum_rank=S.perf_feature(S.SUM_RANK, reqs)))
    return out


def fit_prefill(points: Sequence[Dict]) -> Dict:
    """The prompt model (tokens) fitted to the prefill sweep (microseconds),
    beside the sum-of-ranks form for comparison."""
    t = [p["us"] for p in points]
    res = {}
    for name, kind in (("tokens", S.TOKENS), ("sum_rank", S.SUM_RANK)):
        m, r2 = S.perf_fit(kind, [p[name] for p in points], t)
        res[name] = dict(alpha_us=m.alpha, beta_us=m.beta, r2=r2)
    return res


def fit(points: Sequence[Dict]) -> Dict:
    """Both models of Section 5 fitted to the measured points (microseconds)."""
    t = [p["us"] for p in points]
    res = {}
    for name, kind in (("padded", S.PADDED), ("sum_rank", S.SUM_RANK)):
        m, r2 = S.perf_fit(kind, [p[name] for p in points], t)
        res[name] = dict(alpha_us=m.alpha, beta_us=m.beta, r2=r2)
    return res


def serving_models(fit_res: Dict, kind: str = "sum_rank", *, layers: int = 32, projections: int = 4,
                   base_decode_ms: float = 2.5, base_prefill_us_per_token: float = 15.0,
                   lora_prefill_us_per_token: float = 1.0, prefill_fit: Dict = None):
    """Iteration models of a 7B-class model whose every layer runs the fitted
    decode launch on `projections` projections: decode = base + layers *
    projections * (alpha feature(S) + beta), feature of the chosen fit;
    prompt = tokens times a base plus adapter cost per token (the adapter's
    share from the prompt fit when given).  The base terms are assumptions for
    the simulation (the paper profiles a whole serving stack); the adapter
    terms are measured here.  Milliseconds."""
    f = fit_res[kind]
    launches = layers * projections
    dec = S.model(S.SUM_RANK if kind == "sum_rank" else S.PADDED, launches * f["alpha_us"] / 1000.0,
                  base_decode_ms + launches * f["beta_us"] / 1000.0)
    if prefill_fit is not None:
        # the adapter's share of a prompt token, measured: the fitted slope per
        # launch times the launches of a step
        lora_prefill_us_per_token = launches * prefill_fit["tokens"]["alpha_us"]
    pre = S.model(S.TOKENS, (base_prefill_us_per_token + lora_prefill_us_per_token) / 1000.0, 0.0)
    return pre, dec


def simulate_policies(pre, dec, *, n_instances: int = 60, max_batch: int = 48, n_requests: int = 20000,
                      rps: float = 3000.0, seed: int = 7, slo_factor: float = 1.5, avg_resp_len: float = 136.0,
                      penalty: float = 1e6) -> Dict:
    """Every policy on one seeded Poisson / Zipf trace over 60 instances (the
    instance count of Section 7.4's simulation; the arrival rate is raised to
    load instances whose steps are milliseconds rather than tens of them).
    The time-per-token objective is slo_factor times the decode step of a
    half-full instance at the trace's mean rank."""
    trace = W.sim_trace(seed, n_requests, rps, n_adapters=256, output=(16, 256))
    mean_rank = float(np.mean([r["rank"] for r in trace]))
    ref = S.perf_eval(dec, [(int(round(mean_rank)), 1)] * (max_batch // 2))
    slo = slo_factor * ref
    out = dict(slo_ms=slo, n_instances=n_instances, rps=rps, n_requests=n_requests, max_batch=max_batch)
    for pol, name in S.POLICY_NAMES.items():
        res = S.sim_run(pre, dec, n_instances, max_batch, pol, avg_resp_len, slo, penalty, trace)
        out[name] = S.summarize(res, slo)
    return out
