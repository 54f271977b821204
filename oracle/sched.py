"""Oracle of the rank-aware scheduler (Section 5): the linear performance
models, their least-squares fit, Algorithm 1's cost score, and a simulation of
instances under continuous batching.

TEST INFRASTRUCTURE ONLY: imported by the tests, never by the product path.
Plain Python over floats (IEEE double, every operation rounded on its own, no
fused multiply-add), written from the paper's definitions.  It shares no code
with the library's C++ scheduler; both take the same seeded request lists.

Readings of the paper taken here (the paper is silent on them):
  * a model of an empty batch gives 0 (no launch), not beta;
  * a prompt batch is modelled by its total prompt tokens (the paper names the
    prefill model but gives it no feature);
  * Algorithm 1's candidates are the instances with fewer than max_batch
    running + queued requests, every instance when none has room; ties go to
    the lower index;
  * an instance runs iterations back to back, a prefill of its whole queue
    whenever the queue is not empty, else one decode step of its running batch
    (Section 2.2's continuous batching); a request's time per token is the
    time from its first token to its last over its output tokens minus one.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

PADDED, SUM_RANK, TOKENS = 0, 1, 2
RANK_AWARE, MOST_IDLE, RANDOM, FIRST_FIT = 0, 1, 2, 3


def feature(kind: int, reqs: Sequence[Tuple[int, int]]) -> float:
    """Section 5, "Performance modeling": the batch quantity a model is linear
    in.  reqs are (rank, tokens) pairs.  PADDED: |S| times the largest rank
    (every adapter padded to it); SUM_RANK: the sum of the ranks; TOKENS: the
    sum of the tokens."""
    if len(reqs) == 0:
        return 0.0
    if kind == PADDED:
        return float(len(reqs) * max(r for r, _ in reqs))
    if kind == SUM_RANK:
        return float(sum(r for r, _ in reqs))
    if kind == TOKENS:
        return float(sum(t for _, t in reqs))
    raise ValueError(kind)


def perf(model: Tuple[int, float, float], reqs: Sequence[Tuple[int, int]]) -> float:
    """Perf(S) = alpha * feature(S) + beta (Section 5); 0 for the empty batch."""
    kind, alpha, beta = model
    if len(reqs) == 0:
        return 0.0
    return alpha * feature(kind, reqs) + beta


def fit(f: Sequence[float], t: Sequence[float]) -> Tuple[float, float, float]:
    """Ordinary least squares t ~ alpha f + beta: (alpha, beta, R^2)."""
    n = len(f)
    mf = sum(f) / n
    mt = sum(t) / n
    sff = sum((a - mf) * (a - mf) for a in f)
    sft = sum((a - mf) * (b - mt) for a, b in zip(f, t))
    stt = sum((b - mt) * (b - mt) for b in t)
    alpha = sft / sff
    beta = mt - alpha * mf
    ssr = sum((b - (alpha * a + beta)) ** 2 for a, b in zip(f, t))
    r2 = 1.0 - ssr / stt if stt > 0 else 1.0
    return alpha, beta, r2


def calc_cost(pre, dec, req: Tuple[int, int], running: Sequence[Tuple[int, int]],
              queue: Sequence[Tuple[int, int]], avg_resp_len: float, slo: float, penalty: float) -> float:
    """CalcCost of Algorithm 1: the extra prefill time of the queue, spread over
    the average response length, plus the extra time of every decode step,
    plus the penalty when the decode step would exceed the SLO.  Requests are
    (rank, prompt tokens); in decode steps each counts one token."""
    d_prefill = perf(pre, list(queue) + [req]) - perf(pre, list(queue))
    exists = [(r, 1) for r, _ in running] + [(r, 1) for r, _ in queue]
    with_req = exists + [(req[0], 1)]
    dec_with = perf(dec, with_req)
    d_decode = dec_with - perf(dec, exists)
    cost = d_prefill / avg_resp_len + d_decode
    if dec_with > slo:
        cost = cost + penalty
    return cost


def simulate(pre, dec, n_instances: int, max_batch: int, policy: int, avg_resp_len: float, slo: float,
             penalty: float, reqs: Sequence[dict]) -> List[dict]:
    """Routes every request of the trace (dicts with arrival, rank, prompt,
    output, u; arrivals non-decreasing) and plays each instance's iterations.
    Returns per request: instance, first_token, finish, tpot."""
    clock = [0.0] * n_instances
    running = [[] for _ in range(n_instances)]     # [request index, tokens still to produce]
    queued = [[] for _ in range(n_instances)]
    res = [dict(instance=-1, first_token=0.0, finish=0.0, tpot=0.0) for _ in reqs]

    def done(j, t):
        res[j]["finish"] = t
        o = reqs[j]["output"]
        res[j]["tpot"] = (t - res[j]["first_token"]) / float(o - 1) if o > 1 else 0.0

    def one_iteration(i):
        if queued[i]:
            clock[i] = clock[i] + perf(pre, [(reqs[j]["rank"], reqs[j]["prompt"]) for j in queued[i]])
            for j in queued[i]:
                res[j]["first_token"] = clock[i]
                if reqs[j]["output"] == 1:
                    done(j, clock[i])
                else:
                    running[i].append([j, reqs[j]["output"] - 1])
            queued[i] = []
        else:
            clock[i] = clock[i] + perf(dec, [(reqs[j]["rank"], 1) for j, _ in running[i]])
            still = []
            for j, left in running[i]:
                if left - 1 == 0:
                    done(j, clock[i])
                else:
                    still.append([j, left - 1])
            running[i] = still

    def run_until(i, t):
        while (running[i] or queued[i]) and clock[i] < t:
            one_iteration(i)

    def load(i):
        return len(running[i]) + len(queued[i])

    def least_loaded():
        best = 0
        for i in range(1, n_instances):
            if load(i) < load(best):
                best = i
        return best

    for j, rq in enumerate(reqs):
        for i in range(n_instances):
            run_until(i, rq["arrival"])
        if policy == MOST_IDLE:
            pick = least_loaded()
        elif policy == RANDOM:
            pick = min(max(int(math.floor(rq["u"] * n_instances)), 0), n_instances - 1)
        elif policy == FIRST_FIT:
            room = [i for i in range(n_instances) if load(i) < max_batch]
            pick = room[0] if room else least_loaded()
        else:
            room = [i for i in range(n_instances) if load(i) < max_batch]
            cands = room if room else list(range(n_instances))
            pick, best = -1, 0.0
            for i in cands:
                run_pairs = [(reqs[k]["rank"], reqs[k]["prompt"]) for k, _ in running[i]]
                q_pairs = [(reqs[k]["rank"], reqs[k]["prompt"]) for k in queued[i]]
                total = calc_cost(pre, dec, (rq["rank"], rq["prompt"]), run_pairs, q_pairs,
                                  avg_resp_len, slo, penalty) * float(load(i))
                if pick < 0 or total < best:
                    pick, best = i, total
        if not running[pick] and not queued[pick] and clock[pick] < rq["arrival"]:
            clock[pick] = rq["arrival"]
        queued[pick].append(j)
        res[j]["instance"] = pick
    for i in range(n_instances):
        run_until(i, math.inf)
    return res
