"""Thin Python binding of the scheduler half of liblora.so (include/lora_sched.h):
Section 5's linear performance models, their fit, Algorithm 1's cost score
and the continuous-batching simulator.  Argument marshalling only; the
arithmetic runs in the library's C++ (host code, no GPU needed).
"""
from __future__ import annotations

import ctypes as C
from typing import Dict, List, Sequence, Tuple

import numpy as np

from . import lora as _lora

PADDED, SUM_RANK, TOKENS = 0, 1, 2
RANK_AWARE, MOST_IDLE, RANDOM, FIRST_FIT = 0, 1, 2, 3
POLICY_NAMES = {RANK_AWARE: "rank_aware", MOST_IDLE: "most_idle", RANDOM: "random", FIRST_FIT: "first_fit"}

# Every function include/lora_sched.h declares (checked by the tests).
EXPORTS = ("lora_perf_feature", "lora_perf_eval", "lora_perf_fit", "lora_sched_cost", "lora_sim_run")


class Req(C.Structure):
    _fields_ = [("rank", C.c_int32), ("tokens", C.c_int32)]


class PerfModel(C.Structure):
    _fields_ = [("kind", C.c_int32), ("pad", C.c_int32), ("alpha", C.c_double), ("beta", C.c_double)]

    def as_tuple(self) -> Tuple[int, float, float]:
        return (int(self.kind), float(self.alpha), float(self.beta))


class SimConfig(C.Structure):
    _fields_ = [("pre", PerfModel), ("dec", PerfModel), ("n_instances", C.c_int32), ("max_batch", C.c_int32),
                ("policy", C.c_int32), ("pad", C.c_int32), ("avg_resp_len", C.c_double), ("slo", C.c_double),
                ("penalty", C.c_double)]


class SimReq(C.Structure):
    _fields_ = [("arrival", C.c_double), ("rank", C.c_int32), ("prompt", C.c_int32), ("output", C.c_int32),
                ("pad", C.c_int32), ("u", C.c_double)]


class SimOut(C.Structure):
    _fields_ = [("instance", C.c_int32), ("pad", C.c_int32), ("first_token", C.c_double),
                ("finish", C.c_double), ("tpot", C.c_double)]


_bound = None


def _lib():
    global _bound
    if _bound is not None:
        return _bound
    lib = _lora.load()
    rp, mp = C.POINTER(Req), C.POINTER(PerfModel)
    dp = C.POINTER(C.c_double)
    lib.lora_perf_feature.argtypes = [C.c_int32, rp, C.c_int32]
    lib.lora_perf_feature.restype = C.c_double
    lib.lora_perf_eval.argtypes = [mp, rp, C.c_int32]
    lib.lora_perf_eval.restype = C.c_double
    lib.lora_perf_fit.argtypes = [C.c_int32, dp, dp, C.c_int32, mp, dp]
    lib.lora_perf_fit.restype = C.c_int
    lib.lora_sched_cost.argtypes = [mp, mp, rp, rp, C.c_int32, rp, C.c_int32, C.c_double, C.c_double, C.c_double]
    lib.lora_sched_cost.restype = C.c_double
    lib.lora_sim_run.argtypes = [C.POINTER(SimConfig), C.POINTER(SimReq), C.c_int32, C.POINTER(SimOut)]
    lib.lora_sim_run.restype = C.c_int
    _bound = lib
    return lib


def _reqs(pairs: Sequence[Tuple[int, int]]):
    arr = (Req * max(1, len(pairs)))()
    for i, (r, t) in enumerate(pairs):
        arr[i].rank, arr[i].tokens = int(r), int(t)
    return arr, len(pairs)


def model(kind: int, alpha: float, beta: float) -> PerfModel:
    return PerfModel(int(kind), 0, float(alpha), float(beta))


def perf_feature(kind: int, pairs: Sequence[Tuple[int, int]]) -> float:
    a, n = _reqs(pairs)
    return float(_lib().lora_perf_feature(int(kind), a, n))


def perf_eval(m: PerfModel, pairs: Sequence[Tuple[int, int]]) -> float:
    a, n = _reqs(pairs)
    return float(_lib().lora_perf_eval(C.byref(m), a, n))


def perf_fit(kind: int, f: Sequence[float], t: Sequence[float]) -> Tuple[PerfModel, float]:
    f = np.ascontiguousarray(f, dtype=np.float64)
    t = np.ascontiguousarray(t, dtype=np.float64)
    out = PerfModel()
    r2 = C.c_double()
    dp = C.POINTER(C.c_double)
    _lora._check(_lib().lora_perf_fit(int(kind), f.ctypes.data_as(dp), t.ctypes.data_as(dp), int(f.size),
                                      C.byref(out), C.byref(r2)))
    return out, float(r2.value)


def sched_cost(pre: PerfModel, dec: PerfModel, req: Tuple[int, int], running: Sequence[Tuple[int, int]],
               queue: Sequence[Tuple[int, int]], avg_resp_len: float, slo: float, penalty: float) -> float:
    r, _ = _reqs([req])
    ra, nr = _reqs(running)
    qa, nq = _reqs(queue)
    return float(_lib().lora_sched_cost(C.byref(pre), C.byref(dec), r, ra, nr, qa, nq, float(avg_resp_len),
                                        float(slo), float(penalty)))


def sim_run(pre: PerfModel, dec: PerfModel, n_instances: int, max_batch: int, policy: int, avg_resp_len: float,
            slo: float, penalty: float, reqs: Sequence[Dict]) -> List[Dict]:
    cfg = SimConfig(pre, dec, int(n_instances), int(max_batch), int(policy), 0, float(avg_resp_len), float(slo),
                    float(penalty))
    n = len(reqs)
    arr = (SimReq * max(1, n))()
    for i, q in enumerate(reqs):
        arr[i] = SimReq(float(q["arrival"]), int(q["rank"]), int(q["prompt"]), int(q["output"]), 0, float(q["u"]))
    out = (SimOut * max(1, n))()
    _lora._check(_lib().lora_sim_run(C.byref(cfg), arr, n, out))
    return [dict(instance=int(o.instance), first_token=float(o.first_token), finish=float(o.finish),
                 tpot=float(o.tpot)) for o in out[:n]]


def summarize(res: Sequence[Dict], slo: float) -> Dict:
    """SLO attainment (share of requests whose time per token meets slo) and
    time-per-token statistics of a simulation."""
    tp = np.array([r["tpot"] for r in res], dtype=np.float64)
    if tp.size == 0:
        return dict(slo_attainment=1.0, mean_tpot=0.0, p99_tpot=0.0)
    return dict(slo_attainment=float(np.mean(tp <= slo)), mean_tpot=float(tp.mean()),
                p99_tpot=float(np.percentile(tp, 99)))
