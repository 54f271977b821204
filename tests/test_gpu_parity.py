"""HIP path vs the CPU oracle, element by element, through the C ABI.

Small cases compare every output; the five named Llama-shaped workloads run
at full size through the plan's step launch (the configuration the benchmark
times), are checked bit for bit against the two-launch form and, on every
row, against the oracle, plus properties that hold at any size.
"""
import os
import sys

import numpy as np
import pytest

import oracle
from paper_2401_11240_amd import workloads as W

from parity import compare, compare_v, magnitude

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


def stream():
    return torch.cuda.current_stream(DEV)


def workspace(table, batch):
    n = L.lora_workspace_bytes(table, batch)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=DEV), n


def run_fused(dw, name):
    p = dw.projection(name)
    x = dw.xs[p.x]
    y = p.y.clone()
    ws, n = workspace(p.table, dw.batch)
    L.lora_apply_fused(p.table, dw.batch, x, x.shape[1], y, y.shape[1], ws, n, stream())
    torch.cuda.synchronize()
    return D.from_device_bits(y)


def run_plan(dw, name):
    """The plan path (one step launch), as the benchmark runs it."""
    p = dw.projection(name)
    x = dw.xs[p.x]
    y = p.y.clone()
    plan = L.lora_plan_create(p.table, dw.batch, stream())
    try:
        L.lora_plan_apply(plan, None, x, x.shape[1], y, y.shape[1], stream())
        L.lora_plan_status(plan, stream())
    finally:
        L.lora_plan_destroy(plan)
    return D.from_device_bits(y)


def oracle_full(w, name):
    p = w.projection(name)
    return oracle.lora_apply(w.seg_offset, w.seg_adapter, w.xs[p.x], p.A, p.B, w.ranks, w.scales,
                             p.y, w.dtype)


def int_bits(rng, shape, lo, hi, dtype):
    return W.to_bits(rng.integers(lo, hi, shape).astype(np.float32), dtype)


def make_selector(seed, dtype, h_in, h_out, ranks, seg_lens, seg_adapter):
    """Selector adapters with integer x and y: every product and sum is exact,
    so the HIP result must equal the oracle bit for bit."""
    rng = np.random.default_rng(seed)
    T = int(np.sum(seg_lens))
    A, B = [], []
    for r in ranks:
        c = int(rng.integers(0, h_in - r + 1))
        e = int(rng.integers(0, h_out - r + 1))
        a = np.zeros((h_in, r), np.float32)
        b = np.zeros((r, h_out), np.float32)
        a[c + np.arange(r), np.arange(r)] = 1.0
        b[np.arange(r), e + np.arange(r)] = 1.0
        A.append(W.to_bits(a, dtype))
        B.append(W.to_bits(b, dtype))
    so = np.concatenate([[0], np.cumsum(seg_lens)]).astype(np.int32)
    w = W.Workload(name=f"selector{seed}", dtype=dtype, n_rows=T, seg_offset=so,
                   seg_adapter=np.asarray(seg_adapter, np.int32),
                   ranks=np.asarray(ranks, np.int32),
                   scales=np.array([2.0 ** int(rng.integers(-2, 3)) for _ in ranks], np.float32),
                   xs={"x": int_bits(rng, (T, h_in), -8, 9, dtype)},
                   projections=[W.Projection("p", h_in, h_out, "x", A, B,
                                             int_bits(rng, (T, h_out), -64, 65, dtype))])
    return w


# ---------------------------------------------------------------------------
# exact cases
# ---------------------------------------------------------------------------

def test_hand_worked_example_exact():
    import json
    with open(os.path.join(os.path.dirname(__file__), "golden", "tiny_delta.json")) as f:
        g = json.load(f)
    # h=2 is below the 16-byte row granule: embed the example in h=8 with zeros.
    dt = W.F16
    T = len(g["x"])
    x = np.zeros((T, 8), np.float32)
    x[:, :2] = g["x"]
    y = np.zeros((T, 8), np.float32)
    y[:, :2] = g["y"]
    A = []
    B = []
    for a, b in zip(g["A"], g["B"]):
        a = np.asarray(a, np.float32)
        b = np.asarray(b, np.float32)
        aa = np.zeros((8, a.shape[1]), np.float32)
        aa[:2] = a
        bb = np.zeros((b.shape[0], 8), np.float32)
        bb[:, :2] = b
        A.append(W.to_bits(aa, dt))
        B.append(W.to_bits(bb, dt))
    w = W.Workload("golden", dt, T, np.asarray(g["seg_offset"], np.int32),
                   np.asarray(g["seg_adapter"], np.int32), np.asarray(g["ranks"], np.int32),
                   np.asarray(g["scales"], np.float32), {"x": W.to_bits(x, dt)},
                   [W.Projection("p", 8, 8, "x", A, B, W.to_bits(y, dt))])
    dw = D.upload(w, DEV)
    out = run_fused(dw, "p")
    dw.release()
    got = W.bits_to_f32(out, dt)[:, :2]
    assert got.tolist() == g["out_expected"]
    assert np.all(W.bits_to_f32(out, dt)[:, 2:] == 0)


SELECTOR_CASES = [
    # (dtype, h_in, h_out, ranks, seg_lens, seg_adapter)
    (W.F16, 4096, 4096, [8, 8, 8, 8], [1] * 8, [0, 1, 2, 3, 0, 1, 2, 3]),
    (W.BF16, 4104, 1032, [8, 16, 32, 64, 128, 256], [1, 3, 1, 40, 1, 2, 5, 1],
     [0, 1, -1, 2, 3, 4, 5, 1]),
    (W.F16, 520, 2056, [3, 24, 1, 200, 255], [2, 1, 7, 1, 9], [0, 1, 2, 3, 4]),
    (W.BF16, 8192, 8200, [64, 16], [300, 1, 1, 77], [0, 1, -1, 0]),
    # prompt-sized blocks through LDS at every A row width (1, 3, 4, 6, 16
    # and 24 chunks), blocks of two and four subtiles, a last pass of 40 K
    # and a last column tile of 16 columns
    (W.BF16, 1064, 1040, [8, 24, 32, 48, 128, 192], [20, 70, 130, 33, 17, 64], [0, 1, 2, 3, 4, 5]),
]


@pytest.mark.parametrize("case", range(len(SELECTOR_CASES)))
def test_selector_adapters_bit_exact(case):
    dtype, h_in, h_out, ranks, lens, sa = SELECTOR_CASES[case]
    say(f"selector case {case}: h_in={h_in} h_out={h_out} ranks={ranks}")
    w = make_selector(500 + case, dtype, h_in, h_out, ranks, lens, sa)
    dw = D.upload(w, DEV)
    got = run_fused(dw, "p")
    ref = oracle.round_bits(oracle_full(w, "p"), dtype)
    assert np.array_equal(got, ref)
    # the shrink alone: v[t, j] = x[t, c_g + j] exactly
    p = dw.projection("p")
    r_max = max(ranks)
    ldv = (r_max + 3) // 4 * 4
    v = torch.full((w.n_rows, ldv), float("nan"), dtype=torch.float32, device=DEV)
    ws, n = workspace(p.table, dw.batch)
    x = dw.xs["x"]
    L.lora_shrink(p.table, dw.batch, x, x.shape[1], v, ldv, ws, n, stream())
    torch.cuda.synchronize()
    vg = v.cpu().numpy()
    vr = oracle.lora_shrink(w.seg_offset, w.seg_adapter, w.xs["x"], w.projections[0].A, w.ranks,
                            dtype, ldv=ldv)
    ra = w.row_adapter()
    for t in range(w.n_rows):
        g = ra[t]
        if g < 0:
            assert np.all(np.isnan(vg[t]))
        else:
            assert np.array_equal(vg[t, :ranks[g]], vr[t, :ranks[g]].astype(np.float32))
            assert np.all(np.isnan(vg[t, ranks[g]:]))
    dw.release()


# ---------------------------------------------------------------------------
# random inputs, several tiles and ragged tails
# ---------------------------------------------------------------------------

RANDOM_CASES = [
    # seed, dtype, h_in, h_out, n_adapters, rank_set, seg_lens, adapter law
    (1, W.F16, 4096, 4096, 6, [8, 16, 32, 64], [1] * 24, "zipf"),
    (2, W.BF16, 1032, 2056, 5, [8, 16, 32, 64, 128, 256], [1, 1, 1, 70, 1, 9, 1, 130, 1], "uniform"),
    (3, W.F16, 776, 520, 4, [3, 40, 96, 1], [1, 5, 1, 2, 1, 33], "uniform"),
    (4, W.BF16, 5120, 13824, 8, [8, 16, 32, 64], [1] * 20, "zipf"),
    (5, W.BF16, 13824, 5120, 8, [8, 16, 32, 64], [1] * 20, "zipf"),
    (6, W.F16, 1064, 1040, 6, [8, 24, 32, 48, 128, 192], [20, 70, 1, 130, 33, 17, 64, 3], "uniform"),
]


def random_workload(case):
    seed, dtype, h_in, h_out, n_ad, rank_set, lens, law = case
    rng = np.random.default_rng(seed)
    if law == "zipf":
        sa = rng.choice(n_ad, size=len(lens), p=W.zipf_probs(n_ad)).astype(np.int32)
    else:
        sa = rng.integers(-1, n_ad, size=len(lens)).astype(np.int32)
    return W.small_random(seed, dtype=dtype, h_in=h_in, h_out=h_out, n_adapters=n_ad,
                          rank_set=rank_set, seg_lens=lens, seg_adapter=sa)


@pytest.mark.parametrize("case", range(len(RANDOM_CASES)))
def test_random_parity_fused_shrink_expand(case):
    c = RANDOM_CASES[case]
    say(f"random case {case}: {c[:6]}")
    w = random_workload(c)
    dw = D.upload(w, DEV)
    p = dw.projection("proj")
    got = run_fused(dw, "proj")
    ref = oracle_full(w, "proj")
    st = compare(got, ref, w.dtype, f"random case {case}")
    say("  fused", st)
    # rows without an adapter are bit-identical to the input
    none = w.row_adapter() < 0
    assert np.array_equal(got[none], w.projections[0].y[none])

    # shrink alone vs the oracle's shrink
    ldv = (int(w.ranks.max()) + 3) // 4 * 4
    v = torch.zeros((w.n_rows, ldv), dtype=torch.float32, device=DEV)
    ws, n = workspace(p.table, dw.batch)
    x = dw.xs["x"]
    L.lora_shrink(p.table, dw.batch, x, x.shape[1], v, ldv, ws, n, stream())
    torch.cuda.synchronize()
    vg = v.cpu().numpy()
    vr = np.nan_to_num(oracle.lora_shrink(w.seg_offset, w.seg_adapter, w.xs["x"],
                                          w.projections[0].A, w.ranks, w.dtype, ldv=ldv))
    mask = np.zeros_like(vr, dtype=bool)
    ra = w.row_adapter()
    for t in range(w.n_rows):
        if ra[t] >= 0:
            mask[t, :w.ranks[ra[t]]] = True
    compare_v(np.where(mask, vg, 0.0), np.where(mask, vr, 0.0), f"shrink case {case}")

    # expand alone from a float32 v drawn by the generator's RNG
    rng = np.random.default_rng(900 + case)
    v_in = rng.standard_normal((w.n_rows, ldv)).astype(np.float32)
    y = p.y.clone()
    vt = torch.from_numpy(v_in).to(DEV)
    L.lora_expand(p.table, dw.batch, vt, ldv, y, y.shape[1], ws, n, stream())
    torch.cuda.synchronize()
    ref_e = oracle.lora_expand(w.seg_offset, w.seg_adapter, v_in, w.projections[0].B, w.ranks,
                               w.scales, w.projections[0].y, w.dtype)
    compare(D.from_device_bits(y), ref_e, w.dtype, f"expand case {case}")

    # fused == shrink then expand through the boundary, bit for bit
    y2 = p.y.clone()
    L.lora_expand(p.table, dw.batch, v, ldv, y2, y2.shape[1], ws, n, stream())
    torch.cuda.synchronize()
    assert np.array_equal(D.from_device_bits(y2), got)
    # the one-launch step == the separate launches, bit for bit
    assert np.array_equal(run_plan(dw, "proj"), got)
    dw.release()


def test_plan_reuse_and_determinism():
    w = random_workload(RANDOM_CASES[1])
    dw = D.upload(w, DEV)
    p = dw.projection("proj")
    x = dw.xs["x"]
    ref = run_fused(dw, "proj")
    again = run_fused(dw, "proj")
    assert np.array_equal(ref, again)
    plan = L.lora_plan_create(p.table, dw.batch, stream())
    try:
        for rep in range(3):   # the split-K counters must re-arm between launches
            y = p.y.clone()
            L.lora_plan_apply(plan, None, x, x.shape[1], y, y.shape[1], stream())
            torch.cuda.synchronize()
            assert np.array_equal(D.from_device_bits(y), ref), rep
        L.lora_plan_status(plan, stream())
    finally:
        L.lora_plan_destroy(plan)
    dw.release()


def test_step_launch_graph_replays():
    """The step launch captured in a HIP graph: every replay re-arms the row
    block counters and gives the eager two-launch result bit for bit."""
    w = random_workload(RANDOM_CASES[1])
    dw = D.upload(w, DEV)
    p = dw.projection("proj")
    x = dw.xs["x"]
    ref = run_fused(dw, "proj")
    plan = L.lora_plan_create(p.table, dw.batch, stream())
    try:
        y = p.y.clone()
        side = torch.cuda.Stream(DEV)
        side.wait_stream(torch.cuda.current_stream(DEV))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            with torch.cuda.graph(g, stream=side):
                L.lora_plan_apply(plan, None, x, x.shape[1], y, y.shape[1], side)
        torch.cuda.synchronize()
        for rep in range(4):
            y.copy_(p.y)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert np.array_equal(D.from_device_bits(y), ref), rep
            # eager work between the replays
            y2 = p.y.clone()
            L.lora_plan_apply(plan, None, x, x.shape[1], y2, y2.shape[1], stream())
            torch.cuda.synchronize()
            assert np.array_equal(D.from_device_bits(y2), ref), rep
        L.lora_plan_status(plan, stream())
        del g
    finally:
        L.lora_plan_destroy(plan)
    dw.release()


def test_step_launch_alternating_layers():
    """Consecutive step launches of one plan on different layers (tables and
    inputs): a partial value left over from the previous launch would give
    that layer's numbers, so every launch is checked against its own
    two-launch result, eagerly and inside one captured graph."""
    c = RANDOM_CASES[1]
    w1 = random_workload(c)
    w2 = W.build_workload(name="layer2", seed=78, dtype=w1.dtype, n_adapters=w1.n_adapters,
                          fixed_ranks=w1.ranks, seg_adapter=w1.seg_adapter,
                          seg_lens=np.diff(w1.seg_offset), projections=(("proj", c[2], c[3], "x"),))
    d1, d2 = D.upload(w1, DEV), D.upload(w2, DEV)
    ref = [run_fused(d1, "proj"), run_fused(d2, "proj")]
    layers = [(d1.projection("proj"), d1.xs["x"]), (d2.projection("proj"), d2.xs["x"])]
    plan = L.lora_plan_create(layers[0][0].table, d1.batch, stream())
    try:
        for rep in range(3):
            for i, (p, x) in enumerate(layers):
                y = p.y.clone()
                L.lora_plan_apply(plan, p.table, x, x.shape[1], y, y.shape[1], stream())
                torch.cuda.synchronize()
                assert np.array_equal(D.from_device_bits(y), ref[i]), (rep, i)
        ys = [p.y.clone() for p, _ in layers]
        side = torch.cuda.Stream(DEV)
        side.wait_stream(torch.cuda.current_stream(DEV))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            with torch.cuda.graph(g, stream=side):
                for k in range(4):   # layer 1, 2, 1, 2: the last two redo the first two on their output
                    p, x = layers[k % 2]
                    L.lora_plan_apply(plan, p.table, x, x.shape[1], ys[k % 2], ys[k % 2].shape[1], side)
        torch.cuda.synchronize()
        for rep in range(3):
            for i, (p, _) in enumerate(layers):
                ys[i].copy_(p.y)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for i, (p, x) in enumerate(layers):
                # twice applied: the second launch adds the delta once more onto the first result
                y = torch.from_numpy(ref[i].view(np.int16)).to(DEV)
                L.lora_plan_apply(plan, p.table, x, x.shape[1], y, y.shape[1], stream())
                torch.cuda.synchronize()
                assert np.array_equal(D.from_device_bits(ys[i]), D.from_device_bits(y)), (rep, i)
        L.lora_plan_status(plan, stream())
        del g
    finally:
        L.lora_plan_destroy(plan)
    d1.release()
    d2.release()


def test_step_wait_that_gives_up_is_reported_and_recovered():
    """A spin limit of zero (set from the host) makes every expand workgroup
    give up at once: the launch still ends, the status reports LORA_E_SYNC and
    resets the counters, and the next launch with the normal limit is exact."""
    w = random_workload(RANDOM_CASES[1])
    dw = D.upload(w, DEV)
    p = dw.projection("proj")
    x = dw.xs["x"]
    ref = run_fused(dw, "proj")
    plan = L.lora_plan_create(p.table, dw.batch, stream())
    try:
        L.lora_plan_set_spin_limit(plan, 0)
        y = p.y.clone()
        L.lora_plan_apply(plan, None, x, x.shape[1], y, y.shape[1], stream())
        torch.cuda.synchronize()
        gave_up = False
        try:
            L.lora_plan_status(plan, stream())
        except L.LoraError as e:
            assert e.code == L.LORA_E_SYNC
            gave_up = True
        say(f"  spin limit 0: wait gave up = {gave_up}")
        L.lora_plan_status(plan, stream())          # cleared
        L.lora_plan_set_spin_limit(plan, 1 << 18)
        y = p.y.clone()
        L.lora_plan_apply(plan, None, x, x.shape[1], y, y.shape[1], stream())
        L.lora_plan_status(plan, stream())
        assert np.array_equal(D.from_device_bits(y), ref)
        with pytest.raises(L.LoraError) as e:
            L.lora_plan_set_spin_limit(plan, -1)
        assert e.value.code == L.LORA_E_ARG
    finally:
        L.lora_plan_destroy(plan)
    dw.release()


def test_plan_runs_on_other_compatible_tables():
    """A plan depends on the batch and ranks only: applied to another table
    with the same ranks (another layer's factors) it gives that table's
    result; a table with another rank is refused before anything runs."""
    c = RANDOM_CASES[1]
    w1 = random_workload(c)
    w2 = W.build_workload(name="other_layer", seed=77, dtype=w1.dtype, n_adapters=w1.n_adapters,
                          fixed_ranks=w1.ranks, seg_adapter=w1.seg_adapter,
                          seg_lens=np.diff(w1.seg_offset), projections=(("proj", c[2], c[3], "x"),))
    d1 = D.upload(w1, DEV)
    d2 = D.upload(w2, DEV)
    ref2 = run_fused(d2, "proj")
    p1, p2 = d1.projection("proj"), d2.projection("proj")
    plan = L.lora_plan_create(p1.table, d1.batch, stream())
    try:
        x2 = d2.xs["x"]
        y2 = p2.y.clone()
        L.lora_plan_apply(plan, p2.table, x2, x2.shape[1], y2, y2.shape[1], stream())
        torch.cuda.synchronize()
        assert np.array_equal(D.from_device_bits(y2), ref2)
        # shrink then expand as two launches: the same bits
        y3 = p2.y.clone()
        L.lora_plan_shrink(plan, p2.table, x2, x2.shape[1], stream())
        L.lora_plan_expand(plan, p2.table, y3, y3.shape[1], stream())
        torch.cuda.synchronize()
        assert np.array_equal(D.from_device_bits(y3), ref2)
        ranks3 = w1.ranks.copy()
        used = int(w1.seg_adapter[w1.seg_adapter >= 0][0])
        ranks3[used] = 8 if ranks3[used] != 8 else 16
        bad = L.lora_register_adapters(0, c[2], c[3], w1.dtype, p1.A_ptrs, p1.B_ptrs, ranks3,
                                       w1.scales, stream())
        try:
            with pytest.raises(L.LoraError) as e:
                L.lora_plan_apply(plan, bad, x2, x2.shape[1], y2, y2.shape[1], stream())
            assert e.value.code == L.LORA_E_RANK
        finally:
            L.lora_release_adapters(bad)
    finally:
        L.lora_plan_destroy(plan)
    d1.release()
    d2.release()


def test_permutation_invariance_bit_exact():
    w = random_workload(RANDOM_CASES[0])
    dw = D.upload(w, DEV)
    got = run_fused(dw, "proj")
    dw.release()
    perm = np.random.default_rng(3).permutation(w.n_rows)
    w2 = W.Workload(w.name, w.dtype, w.n_rows, w.seg_offset, w.seg_adapter[perm], w.ranks,
                    w.scales, {"x": w.xs["x"][perm]},
                    [W.Projection("proj", 4096, 4096, "x", w.projections[0].A,
                                  w.projections[0].B, w.projections[0].y[perm])])
    dw2 = D.upload(w2, DEV)
    got2 = run_fused(dw2, "proj")
    dw2.release()
    assert np.array_equal(got2, got[perm])


def test_edge_cases():
    w = random_workload(RANDOM_CASES[2])
    dw = D.upload(w, DEV)
    p = dw.projection("proj")
    x = dw.xs["x"]
    # empty batch and all-unadapted batch: nothing changes
    for so, sa in (([0], []), (w.seg_offset, np.full_like(w.seg_adapter, -1))):
        b = L.Batch(so, sa, n_rows=int(so[-1]))
        y = p.y.clone()
        ws = torch.empty(4096, dtype=torch.uint8, device=DEV)
        L.lora_apply_fused(p.table, b, x, x.shape[1], y, y.shape[1], ws, 4096, stream())
        torch.cuda.synchronize()
        assert torch.equal(y, p.y)
    # a single row
    b1 = L.Batch([0, 1], [2])
    y = p.y[:1].clone()
    ws, n = workspace(p.table, b1)
    L.lora_apply_fused(p.table, b1, x, x.shape[1], y, y.shape[1], ws, n, stream())
    torch.cuda.synchronize()
    ref = oracle.lora_apply([0, 1], [2], w.xs["x"][:1], w.projections[0].A, w.projections[0].B,
                            w.ranks, w.scales, w.projections[0].y[:1], w.dtype)
    compare(D.from_device_bits(y), ref, w.dtype, "single row")
    dw.release()
    # 8-wide projections with prompt-sized blocks: a single partial pass of
    # the LDS-staged shrink, a single partial column tile of the expand
    wt = W.small_random(77, dtype=W.BF16, h_in=8, h_out=8, n_adapters=3, rank_set=[8, 16, 256],
                        seg_lens=[70, 33, 5, 40], seg_adapter=np.array([0, 1, 2, 1], np.int32))
    dwt = D.upload(wt, DEV)
    got = run_fused(dwt, "proj")
    compare(got, oracle_full(wt, "proj"), wt.dtype, "h = 8")
    assert np.array_equal(run_plan(dwt, "proj"), got)
    dwt.release()


def test_errors_are_reported_not_enqueued():
    w = random_workload(RANDOM_CASES[0])
    dw = D.upload(w, DEV)
    p = dw.projection("proj")
    x = dw.xs["x"]
    y = p.y.clone()
    ws, n = workspace(p.table, dw.batch)
    with pytest.raises(L.LoraError) as e:
        L.lora_apply_fused(p.table, dw.batch, x, x.shape[1], y, y.shape[1], ws, n - 1, stream())
    assert e.value.code == L.LORA_E_WORKSPACE
    with pytest.raises(L.LoraError) as e:
        L.lora_apply_fused(p.table, dw.batch, x, x.shape[1], x, x.shape[1], ws, n, stream())
    assert e.value.code == L.LORA_E_OVERLAP
    with pytest.raises(L.LoraError) as e:
        L.lora_apply_fused(p.table, dw.batch, x.data_ptr() + 2, x.shape[1], y, y.shape[1], ws, n,
                           stream())
    assert e.value.code == L.LORA_E_ALIGN
    with pytest.raises(L.LoraError) as e:
        L.lora_apply_fused(p.table, L.Batch([0, 1], [99]), x, x.shape[1], y, y.shape[1], ws, n,
                           stream())
    assert e.value.code == L.LORA_E_INDEX
    # x spanning 2 GiB or more (buffer offsets are 32-bit): refused before any launch
    huge_ld = ((1 << 31) // (2 * max(1, w.n_rows - 1)) + 8) // 8 * 8
    with pytest.raises(L.LoraError) as e:
        L.lora_apply_fused(p.table, dw.batch, x, huge_ld, y, y.shape[1], ws, n, stream())
    assert e.value.code == L.LORA_E_SHAPE
    torch.cuda.synchronize()
    assert torch.equal(y, p.y)
    dw.release()


# ---------------------------------------------------------------------------
# the named workloads at full size
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", list(W.NAMED))
def test_named_workload_full_size(name):
    """Every row of every projection against the oracle, through the step
    launch the benchmark times, and that launch equal to the two-launch form
    bit for bit."""
    say(f"named workload {name}: generating")
    w = W.NAMED[name]()
    dw = D.upload(w, DEV)
    say(f"  uploaded, T={w.n_rows}")
    for p in w.projections:
        got = run_plan(dw, p.name)
        assert np.array_equal(got, run_fused(dw, p.name))   # one step launch == two launches
        ref = oracle_full(w, p.name)
        st = compare(got, ref, w.dtype, f"{name}/{p.name}", mag=magnitude(w, p.name))
        none = w.row_adapter() < 0
        assert np.array_equal(got[none], p.y[none])
        say(f"  {p.name}: all {w.n_rows} rows, {st}")
    dw.release()
