"""HIP path vs the oracle for the cases that reach the less common code paths:

* more than 128 distinct adapters in one step (the launch's argument table
  holds 128 groups; the step launch then reads every factor pointer from the
  device-resident registry, and the separate launches do so for the groups
  beyond 128) -- the large adapter pools of the paper's evaluation (Section
  7.1: 128 to 512 adapters);
* binary16 intermediates beyond the format's range (|x . A| > 65504), where
  the expand must scale v before splitting it into 16-bit parts;
* re-planning one plan for successive batches (continuous batching, Section
  2.2), eagerly and in recorded graphs, with no device memory taken;
* the calls that cannot be recorded refusing a capturing stream.

Every output is compared with the oracle element by element.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2401_11240_amd import workloads as W

from parity import compare, compare_v

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


def oracle_rows(w, batch_so, batch_sa, n, name="proj"):
    p = w.projection(name)
    return oracle.lora_apply(batch_so, batch_sa, w.xs[p.x][:n], p.A, p.B, w.ranks, w.scales, p.y[:n],
                             w.dtype)


# ---------------------------------------------------------------------------
# more than 128 distinct adapters
# ---------------------------------------------------------------------------

def test_more_than_128_distinct_adapters():
    w = W.build_workload(name="pool512", seed=31, dtype=W.BF16, n_adapters=512,
                         rank_set=[8, 16, 32, 64], adapter_law="uniform", n_segments=302,
                         seg_lens=[1] * 300 + [40, 40], projections=(("proj", 1024, 2048, "x"),))
    ra = w.row_adapter()
    n_groups = np.unique(ra[ra >= 0]).size
    say(f"  {w.n_rows} rows, {n_groups} distinct adapters")
    assert n_groups > 128
    dw = D.upload(w, DEV)
    p = dw.projection("proj")
    x = dw.xs["x"]
    ref = oracle_rows(w, w.seg_offset, w.seg_adapter, w.n_rows)

    # step launch: every factor pointer from the registry
    y1 = p.y.clone()
    plan = L.lora_plan_create(p.table, dw.batch, stream())
    try:
        L.lora_plan_apply(plan, None, x, x.shape[1], y1, y1.shape[1], stream())
        L.lora_plan_status(plan, stream())
        # the two launches of the plan: registry for groups beyond 128
        y2 = p.y.clone()
        L.lora_plan_shrink(plan, None, x, x.shape[1], stream())
        L.lora_plan_expand(plan, None, y2, y2.shape[1], stream())
        torch.cuda.synchronize()
    finally:
        L.lora_plan_destroy(plan)
    g1 = D.from_device_bits(y1)
    say("  step launch", compare(g1, ref, w.dtype, "pool512 step"))
    assert np.array_equal(D.from_device_bits(y2), g1)

    # lora_apply_fused, lora_shrink, lora_expand
    n = L.lora_workspace_bytes(p.table, dw.batch)
    ws = torch.empty(n, dtype=torch.uint8, device=DEV)
    y3 = p.y.clone()
    L.lora_apply_fused(p.table, dw.batch, x, x.shape[1], y3, y3.shape[1], ws, n, stream())
    torch.cuda.synchronize()
    assert np.array_equal(D.from_device_bits(y3), g1)
    ldv = 64
    v = torch.zeros((w.n_rows, ldv), dtype=torch.float32, device=DEV)
    L.lora_shrink(p.table, dw.batch, x, x.shape[1], v, ldv, ws, n, stream())
    torch.cuda.synchronize()
    vr = np.nan_to_num(oracle.lora_shrink(w.seg_offset, w.seg_adapter, w.xs["x"], w.projections[0].A,
                                          w.ranks, w.dtype, ldv=ldv))
    mask = np.zeros_like(vr, dtype=bool)
    for t in range(w.n_rows):
        if ra[t] >= 0:
            mask[t, :w.ranks[ra[t]]] = True
    compare_v(np.where(mask, v.cpu().numpy(), 0.0), np.where(mask, vr, 0.0), "pool512 shrink")
    y4 = p.y.clone()
    L.lora_expand(p.table, dw.batch, v, ldv, y4, y4.shape[1], ws, n, stream())
    torch.cuda.synchronize()
    assert np.array_equal(D.from_device_bits(y4), g1)
    dw.release()


# ---------------------------------------------------------------------------
# binary16 intermediates beyond 65504
# ---------------------------------------------------------------------------

def big_v_workload():
    """fp16, h_in 512: adapter 0 has |x . A| around 7e4 (past binary16's
    65504), adapter 1 ordinary values; rows of both in one batch, and one
    prompt segment of adapter 0 (a row block of several subtiles)."""
    rng = np.random.default_rng(44)
    h_in, h_out, T = 512, 1024, 1 + 1 + 1 + 37 + 1
    ranks = np.array([16, 32], np.int32)
    x = rng.uniform(32.0, 64.0, (T, h_in)).astype(np.float32)
    x[3] *= -1.0                                        # negative v too
    A0 = rng.uniform(2.0, 4.0, (h_in, 16)).astype(np.float32)
    B0 = (rng.standard_normal((16, h_out)) * 1e-4).astype(np.float32)
    A1 = (rng.standard_normal((h_in, 32)) / np.sqrt(h_in)).astype(np.float32)
    B1 = (rng.standard_normal((32, h_out)) / np.sqrt(32)).astype(np.float32)
    x[4] = rng.standard_normal(h_in)                    # a row of ordinary values among adapter 0's large ones
    y = rng.standard_normal((T, h_out)).astype(np.float32)
    dt = W.F16
    seg_lens = [1, 1, 1, 37, 1]
    seg_ad = [0, 1, 0, 0, 1]
    so = np.concatenate([[0], np.cumsum(seg_lens)]).astype(np.int32)
    return W.Workload("big_v_f16", dt, T, so, np.asarray(seg_ad, np.int32), ranks,
                      np.array([1.0, 0.5], np.float32), {"x": W.to_bits(x, dt)},
                      [W.Projection("proj", h_in, h_out, "x", [W.to_bits(A0, dt), W.to_bits(A1, dt)],
                                    [W.to_bits(B0, dt), W.to_bits(B1, dt)], W.to_bits(y, dt))])


def test_fp16_intermediate_beyond_binary16_range():
    w = big_v_workload()
    vr = oracle.lora_shrink(w.seg_offset, w.seg_adapter, w.xs["x"], w.projections[0].A, w.ranks, w.dtype,
                            ldv=32)
    vmax = float(np.nanmax(np.abs(vr)))
    say(f"  max |x.A| = {vmax:.4g}")
    assert vmax > 65504
    ref = oracle_rows(w, w.seg_offset, w.seg_adapter, w.n_rows)
    dw = D.upload(w, DEV)
    p = dw.projection("proj")
    x = dw.xs["x"]
    n = L.lora_workspace_bytes(p.table, dw.batch)
    ws = torch.empty(n, dtype=torch.uint8, device=DEV)
    y = p.y.clone()
    L.lora_apply_fused(p.table, dw.batch, x, x.shape[1], y, y.shape[1], ws, n, stream())
    torch.cuda.synchronize()
    got = D.from_device_bits(y)
    say("  fused", compare(got, ref, w.dtype, "big v fused"))
    y2 = p.y.clone()
    plan = L.lora_plan_create(p.table, dw.batch, stream())
    try:
        L.lora_plan_apply(plan, None, x, x.shape[1], y2, y2.shape[1], stream())
        L.lora_plan_status(plan, stream())
    finally:
        L.lora_plan_destroy(plan)
    assert np.array_equal(D.from_device_bits(y2), got)
    # expand from a caller v with values up to 1e6
    rng = np.random.default_rng(45)
    v_in = rng.standard_normal((w.n_rows, 32)).astype(np.float32)
    big = w.row_adapter() == 0
    big[5] = False                                           # a row of small values beside them
    v_in[big] *= np.float32(3e5)
    y3 = p.y.clone()
    L.lora_expand(p.table, dw.batch, torch.from_numpy(v_in).to(DEV), 32, y3, y3.shape[1], ws, n, stream())
    torch.cuda.synchronize()
    ref_e = oracle.lora_expand(w.seg_offset, w.seg_adapter, v_in, w.projections[0].B, w.ranks, w.scales,
                               w.projections[0].y, w.dtype)
    say("  expand", compare(D.from_device_bits(y3), ref_e, w.dtype, "big v expand"))
    dw.release()


# ---------------------------------------------------------------------------
# re-planning
# ---------------------------------------------------------------------------

def replan_setup():
    T = 200
    w = W.build_workload(name="replan", seed=61, dtype=W.BF16, n_adapters=10,
                         rank_set=[8, 16, 32, 64, 128], seg_adapter=[0], seg_lens=[T],
                         projections=(("proj", 2048, 3072, "x"),))
    rng = np.random.default_rng(62)
    batches = []
    # decode tokens; decode tokens and two prompts; a few tokens
    for lens in ([1] * 24, [1] * 30 + [70, 1, 1, 45], [1] * 5):
        sa = rng.integers(-1, 10, size=len(lens)).astype(np.int32)
        sa[0] = 3
        so = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        batches.append((so, sa))
    return w, batches


def test_replan_three_batches_eager_and_recorded():
    w, batches = replan_setup()
    dw = D.upload(w, DEV)
    p = dw.projection("proj")
    x = dw.xs["x"]
    Lb = [L.Batch(so, sa) for so, sa in batches]
    need = max(L.lora_plan_bytes(p.table, b) for b in Lb)
    plan = L.lora_plan_create_reserved(p.table, Lb[0], need, stream())
    ys = [p.y.clone() for _ in range(6)]
    side = torch.cuda.Stream(DEV)
    graphs = []
    try:
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info(DEV)[0]
        for i, (b, (so, sa)) in enumerate(zip(Lb, batches)):
            L.lora_plan_update(plan, None, b, stream())
            # eager
            y = ys[2 * i]
            L.lora_plan_apply(plan, None, x, x.shape[1], y, y.shape[1], stream())
            L.lora_plan_status(plan, stream())
            n = b.n_rows
            ref = oracle_rows(w, so, sa, n)
            got = D.from_device_bits(y)
            say(f"  batch {i}: {n} rows", compare(got[:n], ref, w.dtype, f"replan {i}"))
            assert np.array_equal(got[n:], w.projections[0].y[n:])
            graphs.append(None)
        torch.cuda.synchronize()
        assert torch.cuda.mem_get_info(DEV)[0] == free0      # re-planning took no device memory
        # recorded: one graph per batch, recorded after its update, replayed
        # with eager work between replays; the previous batch's graph then
        # replays stale and does nothing
        prev = None
        for i, (b, (so, sa)) in enumerate(zip(Lb, batches)):
            L.lora_plan_update(plan, None, b, stream())
            torch.cuda.synchronize()
            if prev is not None:
                g_old, y_old = prev
                before = y_old.clone()
                g_old.replay()
                torch.cuda.synchronize()
                assert torch.equal(y_old, before)
                with pytest.raises(L.LoraError) as e:
                    L.lora_plan_status(plan, stream())
                assert e.value.code == L.LORA_E_STALE
            y = ys[2 * i + 1]
            side.wait_stream(torch.cuda.current_stream(DEV))
            g = torch.cuda.CUDAGraph()
            with torch.cuda.stream(side):
                with torch.cuda.graph(g, stream=side):
                    L.lora_plan_apply(plan, None, x, x.shape[1], y, y.shape[1], side)
            torch.cuda.synchronize()
            n = b.n_rows
            ref = oracle_rows(w, so, sa, n)
            for rep in range(3):
                y.copy_(p.y)
                torch.cuda.synchronize()
                g.replay()
                torch.cuda.synchronize()
                got = D.from_device_bits(y)
                compare(got[:n], ref, w.dtype, f"replan graph {i} replay {rep}")
                assert np.array_equal(got, D.from_device_bits(ys[2 * i])), (i, rep)
                # eager work between replays
                y2 = p.y.clone()
                L.lora_plan_apply(plan, None, x, x.shape[1], y2, y2.shape[1], stream())
                torch.cuda.synchronize()
                assert np.array_equal(D.from_device_bits(y2), D.from_device_bits(ys[2 * i]))
            L.lora_plan_status(plan, stream())
            prev = (g, y)
        # a batch past the capacity is refused and the plan keeps working
        big = L.Batch([0, 200], [7])
        with pytest.raises(L.LoraError) as e:
            L.lora_plan_update(plan, None, big, stream())
        assert e.value.code == L.LORA_E_WORKSPACE
        y = p.y.clone()
        L.lora_plan_apply(plan, None, x, x.shape[1], y, y.shape[1], stream())
        L.lora_plan_status(plan, stream())
        assert np.array_equal(D.from_device_bits(y), D.from_device_bits(ys[4]))
        del prev, g
    finally:
        L.lora_plan_destroy(plan)
    dw.release()


def test_ring_calls_refuse_capture():
    w, batches = replan_setup()
    dw = D.upload(w, DEV)
    p = dw.projection("proj")
    x = dw.xs["x"]
    b = L.Batch(*batches[0])
    n = L.lora_workspace_bytes(p.table, b)
    ws = torch.empty(n, dtype=torch.uint8, device=DEV)
    y = p.y.clone()
    v = torch.zeros((b.n_rows, 128), dtype=torch.float32, device=DEV)
    plan = L.lora_plan_create(p.table, b, stream())
    side = torch.cuda.Stream(DEV)
    side.wait_stream(torch.cuda.current_stream(DEV))
    codes = []
    g = torch.cuda.CUDAGraph()
    try:
        with torch.cuda.stream(side):
            with torch.cuda.graph(g, stream=side):
                v.mul_(1.0)                 # the graph is not empty
                for call in (lambda: L.lora_apply_fused(p.table, b, x, x.shape[1], y, y.shape[1], ws, n, side),
                             lambda: L.lora_shrink(p.table, b, x, x.shape[1], v, 128, ws, n, side),
                             lambda: L.lora_expand(p.table, b, v, 128, y, y.shape[1], ws, n, side),
                             lambda: L.lora_plan_update(plan, None, b, side)):
                    try:
                        call()
                        codes.append(0)
                    except L.LoraError as e:
                        codes.append(e.code)
        torch.cuda.synchronize()
        g.replay()                      # an empty graph
        torch.cuda.synchronize()
        assert torch.equal(y, p.y)
    finally:
        L.lora_plan_destroy(plan)
    assert codes == [L.LORA_E_CAPTURE] * 4, codes
    dw.release()
