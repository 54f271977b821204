"""The fused base projection (Eq. 1 whole: y = round(x.W + s_g (x.A_g).B_g))
through the C ABI against the oracle, element by element.

Cases: ragged shapes (K and h_out not multiples of the tile), both tile
sizes (256 while whole tiles of 256 fill the compute units, 128 otherwise),
each with its last tiles split along K, six seeded random shapes, ranks that
need several 64-rank passes and ranks that are not multiples of 8, segments
without an adapter, several adapters in one row tile, binary16 intermediates
past 2^15, the single 1024-token prompt on every row, and the 16-segment
prompt batch (8437 rows) on sampled rows the oracle computes one by one
(every segment's first and last row, every row tile's first and last row).

Tolerance (tests/parity.py): rel-Frobenius <= 2e-3 and per element
max(3e-2, half an ulp + 1e-5|ref|), with the stricter rounding check allowed
the kernel's error bound, here the delta's (2^-14 s_g sum_j |v_j||B_jn|) plus
the base sum's float32 accumulation, K 2^-24 sum_k |x_k||W_kn|.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2401_11240_amd import workloads as W

from parity import compare

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


def run_base(dw, w, name="proj", batch=None, n_rows=None):
    p = dw.projection(name)
    pr = w.projection(name)
    b = batch or dw.batch
    x = dw.xs[p.x]
    wt = D.to_device_bits(np.ascontiguousarray(pr.W.T), DEV)
    y = torch.full((x.shape[0], p.h_out), 0x7FFF, dtype=torch.int16, device=DEV)   # a NaN in both formats: every row must be written
    n = L.lora_base_workspace_bytes(p.table, b)
    ws = torch.empty(max(n, 16), dtype=torch.uint8, device=DEV)
    L.lora_base_apply(p.table, b, x, x.shape[1], wt, wt.shape[1], y, y.shape[1], ws, n, stream())
    torch.cuda.synchronize()
    return D.from_device_bits(y)


def oracle_rows(w, rows, name="proj"):
    """The oracle on the given rows, each as its own one-row segment."""
    pr = w.projection(name)
    ra = w.row_adapter()
    rows = np.asarray(rows)
    so = np.arange(rows.size + 1, dtype=np.int32)
    return oracle.base_lora_apply(so, ra[rows], w.xs[pr.x][rows], pr.W, pr.A, pr.B, w.ranks, w.scales, w.dtype)


def allowance(w, rows, name="proj"):
    """The magnitude the stricter check scales by 2^-14: the delta's terms,
    plus K 2^-10 times the base sum's terms (K 2^-24 of them in all)."""
    pr = w.projection(name)
    ra = w.row_adapter()
    rows = np.asarray(rows)
    xf = np.abs(W.bits_to_f32(w.xs[pr.x][rows], w.dtype).astype(np.float64))
    Wf = np.abs(W.bits_to_f32(pr.W, w.dtype).astype(np.float64))
    mag = (pr.h_in * 2.0 ** -10) * (xf @ Wf)
    so = np.arange(rows.size + 1, dtype=np.int32)
    v = oracle.lora_shrink(so, ra[rows], w.xs[pr.x][rows], pr.A, w.ranks, w.dtype)
    for i, t in enumerate(rows):
        g = int(ra[t])
        if g >= 0:
            r = int(w.ranks[g])
            b = np.abs(W.bits_to_f32(pr.B[g], w.dtype).astype(np.float64)).reshape(r, pr.h_out)
            mag[i] += float(w.scales[g]) * (np.abs(v[i, :r]) @ b)
    return mag


def small_case(seed, dtype, h_in, h_out, ranks, seg_lens, seg_adapter):
    return W.build_workload(name=f"base_s{seed}", seed=seed, dtype=dtype, n_adapters=len(ranks),
                            fixed_ranks=ranks, seg_adapter=seg_adapter, seg_lens=seg_lens,
                            projections=(("proj", h_in, h_out, "x"),), base_weight=True)


SMALL = [
    # seed, dtype, h_in, h_out, ranks, seg_lens, seg_adapter
    (1, W.BF16, 520, 776, [8, 3, 128, 256], [1, 37, 300, 5, 1, 60], [0, 1, 2, -1, 3, 2]),
    (2, W.F16, 1032, 264, [16, 64, 40], [200, 56, 1, 1, 1, 3], [0, 1, 2, 0, -1, 1]),
    (3, W.BF16, 64, 8, [1, 2], [3, 250, 9], [1, 0, 1]),
    # split along K: 4200 x 4104 makes 289 tiles of 256 (more than the 256
    # compute units: the big tile, its last 33 tiles in two K ranges); 500 x
    # 3896 makes 8 of 256 (the small tile: 124 tiles in two K ranges); both
    # ragged in rows, columns and K, adapter runs crossing tile edges
    (5, W.BF16, 1032, 4104, [64, 8, 40], [1500, 700, 3, 1997], [0, 1, -1, 2]),
    (6, W.F16, 2056, 3896, [16, 128, 24], [130, 1, 250, 119], [1, 0, 2, 1]),
    # 289 whole tiles of 256 (K too short to split): a number of whole tiles
    # that the XCDs do not share evenly (so do cases 0 and 1, in tiles of 128)
    (7, W.F16, 520, 4104, [32, 8], [2100, 2100], [0, 1]),
]


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_cases_every_row(case):
    seed, dtype, h_in, h_out, ranks, lens, sa = SMALL[case]
    say(f"base case {case}: h_in={h_in} h_out={h_out} ranks={ranks} lens={lens}")
    w = small_case(*SMALL[case])
    dw = D.upload(w, DEV)
    got = run_base(dw, w)
    rows = np.arange(w.n_rows)
    ref = oracle_rows(w, rows)
    st = compare(got, ref, w.dtype, f"base case {case}", mag=allowance(w, rows))
    say("  ", st)
    dw.release()


def random_case(seed):
    """A seeded random shape: rows 1..3000 in 1..8 segments (some without an
    adapter), h_in and h_out multiples of 8 up to 2056 / 4104, ranks 1..128;
    every third case wide enough for tiles of 256 (at least 256 of them)."""
    rng = np.random.default_rng(1000 + seed)
    big = seed % 3 == 2
    n_seg = int(rng.integers(1, 9))
    total = int(rng.integers(4100, 4400)) if big else int(rng.integers(1, 3001))
    cuts = np.sort(rng.choice(np.arange(1, total), size=min(n_seg - 1, total - 1), replace=False)) if total > 1 else []
    lens = np.diff(np.concatenate([[0], cuts, [total]])).astype(int).tolist()
    n_ad = int(rng.integers(1, 5))
    ranks = [int(r) for r in rng.integers(1, 129, size=n_ad)]
    sa = [int(g) for g in rng.integers(-1, n_ad, size=len(lens))]
    h_in = 8 * int(rng.integers(1, 258))
    h_out = 8 * int(rng.integers(513, 514)) if big else 8 * int(rng.integers(1, 514))
    dtype = W.F16 if rng.integers(0, 2) else W.BF16
    return (2000 + seed, dtype, h_in, h_out, ranks, lens, sa)


@pytest.mark.parametrize("seed", range(6))
def test_random_shapes_every_row(seed):
    case = random_case(seed)
    _, dtype, h_in, h_out, ranks, lens, sa = case
    say(f"base random {seed}: dtype={dtype} h_in={h_in} h_out={h_out} ranks={ranks} lens={lens} adapters={sa}")
    w = small_case(*case)
    dw = D.upload(w, DEV)
    got = run_base(dw, w)
    rows = np.arange(w.n_rows)
    st = compare(got, oracle_rows(w, rows), w.dtype, f"base random {seed}", mag=allowance(w, rows))
    say("  ", st)
    dw.release()


def test_host_schedule_matches_the_device_plan():
    """lora_base_inspect, given this device's compute units, plans the same
    workspace as lora_base_workspace_bytes on a table of the device (the tile
    edge and the K split decide the partial-tile space)."""
    n_cu = torch.cuda.get_device_properties(DEV).multi_processor_count
    for case in [SMALL[0], SMALL[3], SMALL[4], random_case(2)]:
        w = small_case(*case)
        dw = D.upload(w, DEV)
        p = dw.projection("proj")
        pr = w.projection("proj")
        info = L.lora_base_inspect(L.Batch(w.seg_offset, w.seg_adapter), pr.h_in, pr.h_out, w.ranks, n_cu, 8)
        assert info["workspace_bytes"] == L.lora_base_workspace_bytes(p.table, dw.batch), (case[0], info)
        say(f"  case seed {case[0]}: tile {info['tile']}, split {info['split']}, grid {info['grid']}")
        dw.release()


def test_rows_without_adapter_are_the_plain_product_and_empty_batch():
    w = small_case(4, W.BF16, 256, 512, [8], [100, 30], [-1, -1])
    dw = D.upload(w, DEV)
    got = run_base(dw, w)
    pr = w.projection("proj")
    ref = W.bits_to_f32(w.xs["x"], w.dtype).astype(np.float64) @ W.bits_to_f32(pr.W, w.dtype).astype(np.float64)
    compare(got, ref, w.dtype, "no adapters", mag=allowance(w, np.arange(w.n_rows)))
    # an empty batch writes nothing
    p = dw.projection("proj")
    x = dw.xs["x"]
    wt = D.to_device_bits(np.ascontiguousarray(pr.W.T), DEV)
    y = torch.zeros((4, 512), dtype=torch.int16, device=DEV)
    ws = torch.empty(4096, dtype=torch.uint8, device=DEV)
    L.lora_base_apply(p.table, L.Batch([0], []), x, x.shape[1], wt, wt.shape[1], y, y.shape[1], ws, 4096, stream())
    torch.cuda.synchronize()
    assert int(y.abs().sum()) == 0
    # wt overlapping y, and ldw below h_in, are refused before anything runs
    n = L.lora_base_workspace_bytes(p.table, dw.batch)
    ws = torch.empty(n, dtype=torch.uint8, device=DEV)
    yy = torch.zeros((w.n_rows, 512), dtype=torch.int16, device=DEV)
    with pytest.raises(L.LoraError) as e:
        L.lora_base_apply(p.table, dw.batch, x, x.shape[1], yy, 256, yy, 512, ws, n, stream())
    assert e.value.code == L.LORA_E_OVERLAP
    with pytest.raises(L.LoraError) as e:
        L.lora_base_apply(p.table, dw.batch, x, x.shape[1], wt, 248, yy, 512, ws, n, stream())
    assert e.value.code == L.LORA_E_SHAPE
    dw.release()


def test_binary16_intermediate_past_2_15():
    """|s_g x.A_g| around 7e4: v is split after scaling by a power of two."""
    rng = np.random.default_rng(47)
    dt = W.F16
    h_in, h_out, T = 512, 512, 300
    x = rng.uniform(32.0, 64.0, (T, h_in)).astype(np.float32)
    x[7] = rng.standard_normal(h_in)
    A0 = rng.uniform(2.0, 4.0, (h_in, 16)).astype(np.float32)
    B0 = (rng.standard_normal((16, h_out)) * 1e-4).astype(np.float32)
    Wb = (rng.standard_normal((h_in, h_out)) * 1e-3).astype(np.float32)
    so = np.array([0, 260, 300], np.int32)
    w = W.Workload("base_big_v", dt, T, so, np.array([0, -1], np.int32), np.array([16], np.int32),
                   np.array([1.0], np.float32), {"x": W.to_bits(x, dt)},
                   [W.Projection("proj", h_in, h_out, "x", [W.to_bits(A0, dt)], [W.to_bits(B0, dt)],
                                 np.zeros((T, h_out), np.uint16), W.to_bits(Wb, dt))])
    v = oracle.lora_shrink(so, w.seg_adapter, w.xs["x"], w.projections[0].A, w.ranks, dt)
    say(f"  max |x.A| = {np.nanmax(np.abs(v)):.4g}")
    assert np.nanmax(np.abs(v)) > 32768
    dw = D.upload(w, DEV)
    got = run_base(dw, w)
    rows = np.arange(T)
    say("  ", compare(got, oracle_rows(w, rows), dt, "base big v", mag=allowance(w, rows)))
    dw.release()


def test_one_prompt_of_1024_tokens_every_row():
    w = W.BASE_NAMED["prefill_base_l1024"]()
    dw = D.upload(w, DEV)
    got = run_base(dw, w, "q_proj")
    rows = np.arange(w.n_rows)
    say("  ", compare(got, oracle_rows(w, rows, "q_proj"), w.dtype, "l1024", mag=allowance(w, rows, "q_proj")))
    dw.release()


def test_prompt_batch_8437_rows_sampled():
    w = W.BASE_NAMED["prefill_base"]()
    dw = D.upload(w, DEV)
    got = run_base(dw, w, "q_proj")
    assert np.all(np.isfinite(W.bits_to_f32(got, w.dtype)))       # every row written
    so = w.seg_offset
    pick = set()
    for s in range(len(so) - 1):
        pick.update([int(so[s]), int(so[s + 1]) - 1])
    for m0 in range(0, w.n_rows, 256):
        pick.update([m0, min(w.n_rows, m0 + 256) - 1])
    pick.update(int(t) for t in np.random.default_rng(9).choice(w.n_rows, 24, replace=False))
    rows = np.array(sorted(pick))
    say(f"  {rows.size} sampled rows of {w.n_rows}")
    st = compare(got[rows], oracle_rows(w, rows, "q_proj"), w.dtype, "prefill base",
                 mag=allowance(w, rows, "q_proj"))
    say("  ", st)
    dw.release()


def test_base_plan_equals_the_per_call_form_and_replays_in_a_graph():
    """lora_base_plan_apply runs the same kernels as lora_base_apply: equal bit
    for bit; on another table with the same ranks too; and recorded in a graph,
    every replay (eager work between them) equals the eager result."""
    for case in (0, 1):
        w = small_case(*SMALL[case])
        dw = D.upload(w, DEV)
        ref = run_base(dw, w)
        p = dw.projection("proj")
        pr = w.projection("proj")
        x = dw.xs[p.x]
        wt = D.to_device_bits(np.ascontiguousarray(pr.W.T), DEV)
        s = torch.cuda.Stream(DEV)
        plan = L.lora_base_plan_create(p.table, dw.batch, s)
        try:
            y = torch.zeros_like(p.y)
            L.lora_base_plan_apply(plan, None, x, x.shape[1], wt, wt.shape[1], y, y.shape[1], s)
            torch.cuda.synchronize()
            assert np.array_equal(D.from_device_bits(y), ref), f"case {case}"
            # another upload of the same workload: its own table, same ranks
            dw2 = D.upload(w, DEV)
            p2 = dw2.projection("proj")
            y2 = torch.zeros_like(p.y)
            L.lora_base_plan_apply(plan, p2.table, dw2.xs[p2.x], x.shape[1], wt, wt.shape[1], y2, y2.shape[1], s)
            torch.cuda.synchronize()
            assert np.array_equal(D.from_device_bits(y2), ref)
            dw2.release()
            g = torch.cuda.CUDAGraph()
            y3 = torch.zeros_like(p.y)
            with torch.cuda.graph(g, stream=s):
                L.lora_base_plan_apply(plan, None, x, x.shape[1], wt, wt.shape[1], y3, y3.shape[1], s)
            for rep in range(3):
                y3.fill_(0)
                torch.cuda.synchronize()
                g.replay()
                torch.cuda.synchronize()
                assert np.array_equal(D.from_device_bits(y3), ref), f"case {case} replay {rep}"
            del g
        finally:
            torch.cuda.synchronize()
            L.lora_base_plan_destroy(plan)
            dw.release()
