"""Projections that share their input in one launch (lora_plan_create_multi,
lora_plan_apply_multi): every projection's y equals its own lora_plan_apply
launch bit for bit (whose results the full-size parity tests compare with the
oracle on every row), on the 13B-shaped layer (q, k, v on one input; gate
and up on another), on the 70B-shaped batch (q and gate, outputs of
different widths, on one input), on a decode-sized batch (the grid laid out
per XCD) and prompt-sized ones (projections of ragged and of different
widths), eagerly and from a
recorded graph replayed with eager work between replays; the rows are also
compared with the oracle on the small cases; malformed calls are refused
before anything runs."""
import sys

import numpy as np
import pytest

import oracle
from paper_2401_11240_amd import workloads as W

from parity import compare, magnitude

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():   # collected on CPU-only hosts, never run there
    pytest.skip("no GPU", allow_module_level=True)

from paper_2401_11240_amd import device as D  # noqa: E402
from paper_2401_11240_amd import lora as L  # noqa: E402

DEV = torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def groups(w):
    g = {}
    for i, p in enumerate(w.projections):
        g.setdefault((p.x,), []).append(i)
    return {k: v for k, v in g.items() if len(v) > 1}


def check_workload(w, graph_replays=2, against_oracle=False):
    dw = D.upload(w, DEV)
    s = torch.cuda.Stream(DEV)
    y0 = [p.y.clone() for p in dw.projections]
    plans = {}
    try:
        single = [L.lora_plan_create(p.table, dw.batch, s) for p in dw.projections]
        for h, p in zip(single, dw.projections):
            x = dw.xs[p.x]
            L.lora_plan_apply(h, p.table, x, x.shape[1], p.y, p.y.shape[1], s)
        torch.cuda.synchronize()
        ref = [D.from_device_bits(p.y) for p in dw.projections]
        for h in single:
            L.lora_plan_status(h, s)
            L.lora_plan_destroy(h)
        for key, ix in groups(w).items():
            ps = [dw.projections[i] for i in ix]
            plans[key] = L.lora_plan_create_multi([p.table for p in ps], dw.batch, s)
            say(f"  {w.name}: one launch for {[p.name for p in ps]}")

        def run():
            for key, ix in groups(w).items():
                ps = [dw.projections[i] for i in ix]
                x = dw.xs[key[0]]
                L.lora_plan_apply_multi(plans[key], [p.table for p in ps], x, x.shape[1], [p.y for p in ps],
                                        [p.y.shape[1] for p in ps], s)

        def reset():
            for p, y in zip(dw.projections, y0):
                p.y.copy_(y)
            torch.cuda.synchronize()

        def check(tag):
            for key, ix in groups(w).items():
                for i in ix:
                    got = D.from_device_bits(dw.projections[i].y)
                    assert np.array_equal(got, ref[i]), (tag, w.projections[i].name)

        reset()
        with torch.cuda.stream(s):
            run()
        torch.cuda.synchronize()
        check("eager")
        if against_oracle:
            for key, ix in groups(w).items():
                for i in ix:
                    p = w.projections[i]
                    o = oracle.lora_apply(w.seg_offset, w.seg_adapter, w.xs[p.x], p.A, p.B, w.ranks, w.scales, p.y,
                                          w.dtype)
                    compare(D.from_device_bits(dw.projections[i].y), o, w.dtype, p.name, mag=magnitude(w, p.name))
        g = torch.cuda.CUDAGraph()
        reset()
        with torch.cuda.graph(g, stream=s):
            run()
        for rep in range(graph_replays):
            reset()
            g.replay()
            torch.cuda.synchronize()
            check(f"replay {rep}")
        del g
        for h in plans.values():
            L.lora_plan_status(h, s)
    finally:
        torch.cuda.synchronize()
        for h in plans.values():
            L.lora_plan_destroy(h)
        dw.release()


def test_13b_layer_shared_inputs_in_one_launch():
    check_workload(W.NAMED["llama13b_layer"]())


def test_more_than_128_distinct_adapters_in_one_launch():
    # every projection's factor pointers come from its table (the launch's
    # pointer table is the projections' tables, not 128 kernel-argument slots)
    w = W.build_workload(name="multi_pool", seed=41, dtype=W.BF16, n_adapters=400, rank_set=[8, 16, 32, 64],
                         adapter_law="uniform", n_segments=202, seg_lens=[1] * 200 + [40, 70],
                         projections=(("q", 1024, 1024, "x"), ("gate", 1024, 2056, "x")))
    ra = w.row_adapter()
    assert np.unique(ra[ra >= 0]).size > 128
    check_workload(w, graph_replays=1, against_oracle=True)


def test_70b_batch_q_and_gate_in_one_launch():
    check_workload(W.NAMED["llama70b_mixed"](), graph_replays=1)


@pytest.mark.parametrize("kind", ["decode", "prompt", "widths"])
def test_small_batches_shared_input(kind):
    if kind == "decode":
        lens, sa = [1] * 40, [i % 7 for i in range(40)]
    else:
        lens, sa = [100, 37, 300, 5], [0, 3, 5, -1]
    if kind == "widths":   # output widths that differ: q, gate, up and a narrow k
        projs = (("q", 520, 264, "x"), ("gate", 520, 776, "x"), ("up", 520, 776, "x"), ("k", 520, 72, "x"))
    else:
        projs = (("q", 520, 264, "x"), ("k", 520, 264, "x"), ("v", 520, 264, "x"))
    w = W.build_workload(name=f"multi_{kind}", seed=31, dtype=W.F16 if kind == "decode" else W.BF16, n_adapters=7,
                         rank_set=[8, 16, 40, 64], seg_adapter=sa, seg_lens=lens, projections=projs)
    check_workload(w, against_oracle=True)


def test_multi_refuses_bad_calls():
    w = W.build_workload(name="multi_bad", seed=7, dtype=W.BF16, n_adapters=3, rank_set=[8, 16],
                         seg_adapter=[0, 2], seg_lens=[3, 4],
                         projections=(("q", 256, 128, "x"), ("k", 256, 128, "x"), ("o", 256, 64, "x")))
    dw = D.upload(w, DEV)
    q, k, o = dw.projections
    x = dw.xs["x"]
    s = torch.cuda.current_stream(DEV)
    try:
        with pytest.raises(L.LoraError) as e:
            L.lora_plan_create_multi([], dw.batch, s)
        assert e.value.code == L.LORA_E_ARG
        h = L.lora_plan_create_multi([q.table, o.table], dw.batch, s)
        try:
            with pytest.raises(L.LoraError) as e:  # a table of another output width in a projection's place
                L.lora_plan_apply_multi(h, [q.table, k.table], x, 256, [q.y, k.y], [128, 128], s)
            assert e.value.code == L.LORA_E_SHAPE
        finally:
            L.lora_plan_destroy(h)
        h = L.lora_plan_create_multi([q.table, k.table], dw.batch, s)
        try:
            with pytest.raises(L.LoraError) as e:  # outputs overlapping each other
                L.lora_plan_apply_multi(h, [q.table, k.table], x, 256, [q.y, q.y], [128, 128], s)
            assert e.value.code == L.LORA_E_OVERLAP
            with pytest.raises(L.LoraError) as e:  # a plan of several projections on the single call
                L.lora_plan_apply(h, q.table, x, 256, q.y, 128, s)
            assert e.value.code == L.LORA_E_ARG
        finally:
            L.lora_plan_destroy(h)
    finally:
        torch.cuda.synchronize()
        dw.release()
