"""Section 5's scheduler: the oracle (oracle/sched.py) pinned by the paper's
toy example, closed forms and a library least-squares routine, then the
library's C++ (include/lora_sched.h) against the oracle, bit for bit where
the definitions fix the operation order.  Host code only: no GPU."""
import json
import math
import os

import numpy as np
import pytest

from oracle import sched as O
from paper_2401_11240_amd import build as B
from paper_2401_11240_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def S():
    if not os.path.exists(B.lib_path()):
        B.build()
    from paper_2401_11240_amd import sched
    return sched


def fig5():
    with open(os.path.join(ROOT, "tests", "golden", "fig5_schedule.json")) as f:
        return json.load(f)


def two_point_models(g, key, kind):
    """The linear model through the two latencies the example prints."""
    f = [O.feature(kind, [(i["rank"], 1)] * i["requests"]) for i in g["instances"]]
    t = [i[key] for i in g["instances"]]
    a, b, r2 = O.fit(f, t)
    return (kind, a, b), r2


# ---------------------------------------------------------------------------
# oracle pins
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("key,kind", [("bgmv_ms", O.PADDED), ("mbgmv_ms", O.SUM_RANK)])
def test_oracle_fig5_toy_example(key, kind):
    """Fit through the printed latencies, the models give them back; Algorithm
    1 then sends the new rank-64 request where the example says, and the
    instance it avoids would exceed the 36 ms SLO."""
    g = fig5()
    m, r2 = two_point_models(g, key, kind)
    assert r2 == pytest.approx(1.0, abs=1e-12)
    for inst in g["instances"]:
        assert O.perf(m, [(inst["rank"], 1)] * inst["requests"]) == pytest.approx(inst[key], abs=1e-9)
    req = (g["new_rank"], 128)
    pre = (O.TOKENS, 0.01, 1.0)
    costs = []
    for inst in g["instances"]:
        running = [(inst["rank"], 128)] * inst["requests"]
        c = O.calc_cost(pre, m, req, running, [], 100.0, g["slo_ms"], 1000.0)
        costs.append(c * inst["requests"])
    name = "bgmv" if kind == O.PADDED else "mbgmv"
    assert int(np.argmin(costs)) == g["choice"][name]
    for i in g["violates_if_sent_to"][name]:
        inst = g["instances"][i]
        assert O.perf(m, [(inst["rank"], 1)] * inst["requests"] + [(g["new_rank"], 1)]) > g["slo_ms"]
    if kind == O.SUM_RANK:
        # the chosen instance stays within the SLO under the padding-free model
        inst = g["instances"][g["choice"]["mbgmv"]]
        assert O.perf(m, [(inst["rank"], 1)] * inst["requests"] + [(g["new_rank"], 1)]) <= g["slo_ms"]


def test_oracle_features_by_hand():
    S_ = [(8, 3), (64, 1), (16, 5)]
    assert O.feature(O.PADDED, S_) == 3 * 64
    assert O.feature(O.SUM_RANK, S_) == 8 + 64 + 16
    assert O.feature(O.TOKENS, S_) == 9
    assert O.perf((O.SUM_RANK, 2.0, 5.0), []) == 0.0
    assert O.perf((O.SUM_RANK, 2.0, 5.0), S_) == 2.0 * 88 + 5.0


def test_oracle_fit_against_library_regression():
    """Exact data is recovered; noisy data agrees with scipy's linregress."""
    f = [1.0, 3.0, 5.0, 7.0, 12.0, 20.0]       # dyadic means and sums: every step exact
    a, b, r2 = O.fit(f, [0.25 * x + 3.0 for x in f])
    assert (a, b, r2) == (0.25, 3.0, 1.0)
    from scipy import stats
    rng = np.random.default_rng(3)
    x = rng.uniform(0, 100, 40)
    y = 0.7 * x + 12 + rng.normal(0, 5, 40)
    a, b, r2 = O.fit(list(x), list(y))
    ref = stats.linregress(x, y)
    assert a == pytest.approx(ref.slope, rel=1e-12)
    assert b == pytest.approx(ref.intercept, rel=1e-12)
    assert r2 == pytest.approx(ref.rvalue ** 2, rel=1e-12)


def test_oracle_calc_cost_by_hand():
    """Numbers worked out by hand: PrePerf = 0.5 tokens + 2, DecPerf = 0.1 sum
    of ranks + 20, running (8, 16), queue (32 with a 10-token prompt), new
    request of rank 64 with a 6-token prompt, average response 4 tokens.
    d_prefill = (0.5*16+2) - (0.5*10+2) = 3; d_decode = 0.1*64 = 6.4;
    cost = 3/4 + 6.4 = 7.15; DecPerf with it = 0.1*120 + 20 = 32."""
    pre, dec = (O.TOKENS, 0.5, 2.0), (O.SUM_RANK, 0.1, 20.0)
    c = O.calc_cost(pre, dec, (64, 6), [(8, 99), (16, 7)], [(32, 10)], 4.0, 40.0, 100.0)
    assert c == pytest.approx(7.15, abs=1e-12)
    c = O.calc_cost(pre, dec, (64, 6), [(8, 99), (16, 7)], [(32, 10)], 4.0, 31.9, 100.0)
    assert c == pytest.approx(107.15, abs=1e-12)
    # an empty instance: the whole prefill and decode cost of the request
    c = O.calc_cost(pre, dec, (64, 6), [], [], 4.0, 1e9, 0.0)
    assert c == pytest.approx((0.5 * 6 + 2) / 4 + (0.1 * 64 + 20), abs=1e-12)


def test_oracle_simulation_closed_forms():
    pre, dec = (O.TOKENS, 0.5, 2.0), (O.SUM_RANK, 0.25, 10.0)
    # one request: prefill, then output-1 decode steps of its own
    r = O.simulate(pre, dec, 1, 8, O.MOST_IDLE, 10.0, 1e9, 0.0,
                   [dict(arrival=5.0, rank=16, prompt=20, output=4, u=0.0)])[0]
    first = 5.0 + (0.5 * 20 + 2.0)
    assert r["first_token"] == first
    assert r["finish"] == first + 3 * (0.25 * 16 + 10.0)
    assert r["tpot"] == 0.25 * 16 + 10.0
    # a second request that arrives during the first one's prefill waits for
    # it, is prefilled alone, then decodes with it
    reqs = [dict(arrival=0.0, rank=8, prompt=8, output=3, u=0.0),
            dict(arrival=1.0, rank=32, prompt=4, output=2, u=0.0)]
    r = O.simulate(pre, dec, 1, 8, O.MOST_IDLE, 10.0, 1e9, 0.0, reqs)
    t1 = 0.0 + (0.5 * 8 + 2.0)             # 6: first token of request 0
    t2 = t1 + (0.5 * 4 + 2.0)              # 10: prefill of request 1 (queue first)
    t3 = t2 + (0.25 * 40 + 10.0)           # 30: decode step of both; request 1 done
    t4 = t3 + (0.25 * 8 + 10.0)            # 42: last token of request 0
    assert [r[0]["first_token"], r[1]["first_token"]] == [t1, t2]
    assert [r[0]["finish"], r[1]["finish"]] == [t4, t3]
    assert r[0]["tpot"] == (t4 - t1) / 2 and r[1]["tpot"] == t3 - t2
    # a one-token request finishes with its prefill
    r = O.simulate(pre, dec, 1, 8, O.MOST_IDLE, 10.0, 1e9, 0.0,
                   [dict(arrival=0.0, rank=8, prompt=2, output=1, u=0.0)])[0]
    assert r["finish"] == r["first_token"] == 3.0 and r["tpot"] == 0.0


def test_oracle_routing_policies_by_hand():
    pre, dec = (O.TOKENS, 0.0, 1.0), (O.SUM_RANK, 0.0, 1.0)
    # three simultaneous long requests on three instances
    reqs = [dict(arrival=0.0, rank=8, prompt=1, output=1000, u=u) for u in (0.9, 0.1, 0.5, 0.0)]
    inst = lambda p, mb=2: [r["instance"] for r in O.simulate(pre, dec, 3, mb, p, 10.0, 1e9, 0.0, reqs)]
    assert inst(O.MOST_IDLE) == [0, 1, 2, 0]
    assert inst(O.FIRST_FIT) == [0, 0, 1, 1]
    assert inst(O.FIRST_FIT, 1) == [0, 1, 2, 0]   # none has room: the most idle
    assert inst(O.RANDOM) == [2, 0, 1, 0]
    # Algorithm 1: an idle instance scores 0 and is taken first (with models
    # of positive slope; at slope 0 one more request costs a busy instance
    # nothing and ties go to the lower index)
    ra = [r["instance"] for r in O.simulate((O.TOKENS, 0.1, 1.0), (O.SUM_RANK, 0.1, 1.0), 3, 2, O.RANK_AWARE,
                                            10.0, 1e9, 0.0, reqs)]
    assert ra == [0, 1, 2, 0]
    assert inst(O.RANK_AWARE) == [0, 0, 1, 1]      # instance 0 full at max_batch 2: no longer a candidate


def test_oracle_rank_aware_separates_ranks_under_padding():
    """Under the padded model a rank-64 request joins the instance already at
    rank 64 rather than raising a rank-8 batch's padding (Section 2.3, C2)."""
    pre, dec = (O.TOKENS, 0.0, 1.0), (O.PADDED, 0.01, 1.0)
    reqs = ([dict(arrival=0.0, rank=8, prompt=1, output=10 ** 6, u=0.0)] * 4 +
            [dict(arrival=0.0, rank=64, prompt=1, output=10 ** 6, u=0.0)] * 2)
    reqs = [dict(r) for r in reqs]
    # first fill: instance 0 takes rank 8 work, instance 1 rank 64 work
    order = [dict(reqs[0]), dict(reqs[4]), dict(reqs[1]), dict(reqs[5]), dict(reqs[2])]
    order.append(dict(arrival=0.0, rank=64, prompt=1, output=10 ** 6, u=0.0))
    r = O.simulate(pre, dec, 2, 100, O.RANK_AWARE, 10.0, 1e9, 0.0, order)
    assert [x["instance"] for x in r] == [0, 1, 0, 1, 0, 1]


# ---------------------------------------------------------------------------
# library against the oracle
# ---------------------------------------------------------------------------

def random_batch(rng, n):
    return [(int(rng.choice([1, 8, 16, 32, 64, 256])), int(rng.integers(1, 600))) for _ in range(n)]


def test_features_and_models_bit_for_bit(S):
    rng = np.random.default_rng(11)
    for trial in range(200):
        b = random_batch(rng, int(rng.integers(0, 40)))
        for kind in (O.PADDED, O.SUM_RANK, O.TOKENS):
            assert S.perf_feature(kind, b) == O.feature(kind, b)
            a, c = float(rng.uniform(1e-4, 1e-1)), float(rng.uniform(0, 50))
            assert S.perf_eval(S.model(kind, a, c), b) == O.perf((kind, a, c), b)


def test_fit_matches_oracle(S):
    rng = np.random.default_rng(12)
    for trial in range(20):
        n = int(rng.integers(2, 60))
        f = rng.uniform(0, 1e4, n)
        t = 3e-3 * f + 7 + rng.normal(0, 1, n)
        m, r2 = S.perf_fit(O.SUM_RANK, f, t)
        a, b, r2o = O.fit(list(f), list(t))
        assert m.kind == O.SUM_RANK
        assert m.alpha == pytest.approx(a, rel=1e-12)
        assert m.beta == pytest.approx(b, rel=1e-12, abs=1e-12)
        assert r2 == pytest.approx(r2o, rel=1e-12, abs=1e-12)


def test_sched_cost_bit_for_bit(S):
    rng = np.random.default_rng(13)
    for trial in range(200):
        pre = (O.TOKENS, float(rng.uniform(0, 0.05)), float(rng.uniform(0, 5)))
        dec = (int(rng.integers(0, 2)), float(rng.uniform(0, 0.05)), float(rng.uniform(0, 30)))
        req = random_batch(rng, 1)[0]
        run, q = random_batch(rng, int(rng.integers(0, 30))), random_batch(rng, int(rng.integers(0, 5)))
        avg, slo, pen = float(rng.uniform(1, 300)), float(rng.uniform(10, 60)), float(rng.uniform(0, 1000))
        got = S.sched_cost(S.model(*pre), S.model(*dec), req, run, q, avg, slo, pen)
        assert got == O.calc_cost(pre, dec, req, run, q, avg, slo, pen)


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("policy", [0, 1, 2, 3])
def test_simulation_bit_for_bit(S, seed, policy):
    trace = W.sim_trace(seed, 300, rps=40.0, n_adapters=32)
    pre = (O.TOKENS, 0.02, 3.0)
    dec = (O.PADDED if seed % 2 else O.SUM_RANK, 0.004, 18.0)
    args = (8, 12, policy, 100.0, 30.0, 1000.0)
    got = S.sim_run(S.model(*pre), S.model(*dec), *args, trace)
    ref = O.simulate(pre, dec, *args, trace)
    for j, (a, b) in enumerate(zip(got, ref)):
        assert a == b, (j, a, b)
    assert all(r["finish"] >= r["first_token"] >= t["arrival"] for r, t in zip(got, trace))


def test_library_rejects_bad_arguments(S):
    from paper_2401_11240_amd import lora as L
    with pytest.raises(L.LoraError) as e:
        S.perf_fit(O.SUM_RANK, [1.0, 1.0, 1.0], [1.0, 2.0, 3.0])
    assert e.value.code == L.LORA_E_SHAPE
    with pytest.raises(L.LoraError) as e:
        S.perf_fit(O.SUM_RANK, [1.0], [1.0])
    assert e.value.code == L.LORA_E_ARG
    with pytest.raises(L.LoraError) as e:
        S.sim_run(S.model(2, 0.1, 1), S.model(1, 0.1, 1), 2, 4, 0, 10.0, 30.0, 0.0,
                  [dict(arrival=2.0, rank=8, prompt=4, output=3, u=0.1),
                   dict(arrival=1.0, rank=8, prompt=4, output=3, u=0.1)])
    assert e.value.code == L.LORA_E_ARG
    assert S.perf_feature(7, [(8, 1)]) == -1.0
    assert math.isnan(S.sched_cost(S.model(2, 0.1, 1), S.model(1, 0.1, 1), (8, 1), [], [], 0.0, 30.0, 0.0))
