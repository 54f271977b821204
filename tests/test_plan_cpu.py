"""The planner's work list, checked on the host (no GPU): lora_plan_inspect
reports every work item a plan would launch and its grid position.

The single step launch relies on these properties: an item only ever waits
for items earlier in the grid (shrink, then reduce, then expand items of a
row block), so every wait ends; the items of a row block cover its K range,
its columns and its v exactly once; a grid laid out per XCD keeps each row
block on one XCD and the XCDs balanced.
"""
import numpy as np
import pytest

from paper_2401_11240_amd import lora as L

KIND_SHRINK, KIND_EXPAND, KIND_REDUCE = 1, 2, 3


def random_batch(rng, n_adapters):
    n_seg = int(rng.integers(1, 90))
    lens = []
    for _ in range(n_seg):
        lens.append(1 if rng.random() < 0.7 else int(rng.integers(2, 300)))
    adapters = [int(rng.integers(-1, n_adapters)) for _ in range(n_seg)]
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    return L.Batch(off, adapters), off, adapters


def partitions(ranges, total):
    """True when the [lo, lo + len) ranges tile [0, total) exactly."""
    ranges = sorted(ranges)
    at = 0
    for lo, n in ranges:
        if lo != at or n <= 0:
            return False
        at += n
    return at == total


STAGE_CHUNKS = 1024            # 16-byte chunks of one LDS buffer of the LDS-staged shrink
SHRINK_LDS = 4 * STAGE_CHUNKS * 16
EXPAND_YS_OFF = 32 * 1024       # expand: v fragments below, the staged y tile above
EXPAND_VMAX_OFF = EXPAND_YS_OFF + 33 * 1024 + 256 - 16


def ceil_to(v, m):
    return (v + m - 1) // m * m


def check_lds_fit(rank, nrows, sh, ex):
    """Every item's staging fits the LDS its kernel body lays out: a shrink
    pass of a block of more than 16 rows (rank a multiple of 8) in one
    16 KiB buffer of the LDS-staged body (A rows rounded to whole 1 KiB wave
    loads, then the x rows), other passes in the register-staged body's
    space; an expand item's v fragments below the y tile, its y tile (and
    the columns it walks) within the rest."""
    ms = 1 if nrows <= 16 else (2 if nrows <= 32 else 4)
    rp = ceil_to(rank, 16)
    for sub in set(sh["sub"].tolist()):
        stage = ceil_to(sub * (rank // 8), 64) + 2 * ms * sub
        if ms > 1 and rank % 8 == 0 and stage <= STAGE_CHUNKS:
            assert sub % 32 == 0 and (sub % 64 == 0 or sub == 32) and sub <= 512
        else:
            wn = 4 if ms == 1 else (4 if rp // 16 >= 4 else (2 if rp // 16 >= 2 else 1))
            staged = (rp + ms * 16) * (sub // 8 + 1) * 16
            red = (4 // wn) * ms * 16 * (rp + 4) * 4 if wn < 4 else 0
            assert max(staged, red) <= SHRINK_LDS, (rank, nrows, sub)
    q = 32768 // (rp * 512)
    q = 4 if q >= 4 else (2 if q >= 2 else 1)
    while q * ms > 4:
        q //= 2
    tiles = 2 if ms == 4 else 1
    assert np.all(ex["len"] <= 256 * q * tiles), (rank, nrows)
    assert ms * (rp // 16) * 64 * 16 <= EXPAND_YS_OFF
    if ms > 1:
        assert EXPAND_YS_OFF + ms * 16 * (32 * q + 1) * 16 <= EXPAND_VMAX_OFF


def check_plan(items, h_in, h_out, n_xcd):
    grid = items[items["grid_pos"] >= 0]
    extra = items[items["grid_pos"] < 0]
    assert np.array_equal(grid["grid_pos"], np.arange(len(grid)))
    assert np.all(extra["kind"] == KIND_REDUCE)
    real = grid[grid["kind"] > 0]
    if n_xcd == 1:
        assert len(real) == len(grid)       # no empty slots without a layout
    laid_out = len(real) != len(grid)
    for rb in np.unique(real["row_block"]):
        mine = real[real["row_block"] == rb]
        sh = mine[mine["kind"] == KIND_SHRINK]
        ex = mine[mine["kind"] == KIND_EXPAND]
        rd = mine[mine["kind"] == KIND_REDUCE]
        allrd = extra[extra["row_block"] == rb]
        nsplit, pstride, rank, nrows = (int(mine[0][f]) for f in ("nsplit", "pstride", "rank", "nrows"))
        assert 1 <= nrows <= 64 and (nrows <= 32 or (rank + 15) // 16 * 16 <= 128)
        assert pstride == nrows * ((rank + 7) // 8 * 8)
        # K ranges, column tiles and v slices each covered exactly once
        assert len(sh) == nsplit and partitions(zip(sh["lo"], sh["len"]), h_in)
        assert np.all(sh["sub"] % 32 == 0) and np.all(sh["len"] % 8 == 0)
        assert len(ex) >= 1 and partitions(zip(ex["lo"], ex["len"]), h_out)
        assert np.all(ex["len"] % 8 == 0)
        check_lds_fit(rank, nrows, sh, ex)
        assert partitions(zip(allrd["lo"], allrd["len"]), pstride)
        direct = set(ex["sub"].tolist())
        assert len(direct) == 1
        if direct == {1}:
            assert len(rd) == 0                # expand items add the partial blocks themselves
        else:
            assert partitions(zip(rd["lo"], rd["len"]), pstride)
        # forward progress: every item waits only on earlier grid positions
        last_shrink = sh["grid_pos"].max()
        if len(rd):
            assert rd["grid_pos"].min() > last_shrink
            assert ex["grid_pos"].min() > rd["grid_pos"].max()
        assert ex["grid_pos"].min() > last_shrink
        if laid_out:
            assert len(set((mine["grid_pos"] % n_xcd).tolist())) == 1
    if laid_out:
        # balance of the streamed bytes over the XCDs (the planner's criterion)
        load = np.zeros(n_xcd)
        for rb in np.unique(real["row_block"]):
            mine = real[real["row_block"] == rb]
            r, n = int(mine[0]["rank"]), int(mine[0]["nrows"])
            load[int(mine[0]["grid_pos"]) % n_xcd] += (r + n) * h_in * 2 + (r + 2 * n) * h_out * 2
        assert 4 * load.max() * n_xcd <= 5 * load.sum()
    else:
        kinds = real["kind"]
        order = {KIND_SHRINK: 0, KIND_REDUCE: 1, KIND_EXPAND: 2}
        ranks = [order[int(k)] for k in kinds]
        assert ranks == sorted(ranks)          # list order: all shrink, all reduce, all expand


@pytest.mark.parametrize("seed", range(40))
def test_random_plans(seed):
    rng = np.random.default_rng(1000 + seed)
    n_adapters = int(rng.integers(1, 40))
    ranks = [int(rng.choice([8, 16, 32, 64, 128, 256])) if rng.random() < 0.8 else int(rng.integers(1, 257))
             for _ in range(n_adapters)]
    h_in = int(rng.integers(1, 2049)) * 8
    h_out = int(rng.integers(1, 2049)) * 8
    b, off, adapters = random_batch(rng, n_adapters)
    adapted = sum(int(off[i + 1] - off[i]) for i, a in enumerate(adapters) if a >= 0)
    for n_xcd in (1, 8):
        items = L.lora_plan_inspect(b, h_in, h_out, ranks, n_xcd=n_xcd)
        check_plan(items, h_in, h_out, n_xcd)
        grid = items[(items["grid_pos"] >= 0) & (items["kind"] > 0)]
        # every adapted row lies in exactly one row block
        blocks = {}
        for it in grid:
            blocks[int(it["row_block"])] = int(it["nrows"])
        assert sum(blocks.values()) == adapted


def test_decode_headline_is_laid_out_and_few_adapters_are_not():
    from paper_2401_11240_amd import workloads as W
    w = W.NAMED["decode_mixed"]()
    p = w.projections[0]
    items = L.lora_plan_inspect(L.Batch(w.seg_offset, w.seg_adapter), p.h_in, p.h_out, w.ranks, n_xcd=8)
    grid = items[items["grid_pos"] >= 0]
    assert (grid["kind"] == 0).any()           # laid out per XCD (slots without work)
    check_plan(items, p.h_in, p.h_out, 8)
    # one adapter for every row: its row blocks cannot be spread, list order
    b = L.Batch([0, 64], [0])
    items = L.lora_plan_inspect(b, 4096, 4096, [64], n_xcd=8)
    assert not (items[items["grid_pos"] >= 0]["kind"] == 0).any()
    check_plan(items, 4096, 4096, 8)


@pytest.mark.parametrize("name", ["prefill", "llama13b_layer"])
def test_named_workload_plans(name):
    """The benchmark's prompt-sized and mixed batches: forward progress,
    exact coverage and LDS fit of every item, for every projection."""
    from paper_2401_11240_amd import workloads as W
    w = W.NAMED[name]()
    for p in w.projections:
        items = L.lora_plan_inspect(L.Batch(w.seg_offset, w.seg_adapter), p.h_in, p.h_out, w.ranks, n_xcd=8)
        check_plan(items, p.h_in, p.h_out, 8)


def test_inspect_errors():
    b = L.Batch([0, 1], [0])
    with pytest.raises(L.LoraError) as e:
        L.lora_plan_inspect(b, 4100, 4096, [8])
    assert e.value.code == L.LORA_E_SHAPE
    with pytest.raises(L.LoraError) as e:
        L.lora_plan_inspect(b, 4096, 4096, [300])
    assert e.value.code == L.LORA_E_RANK
    with pytest.raises(L.LoraError) as e:
        L.lora_plan_inspect(L.Batch([0, 1], [3]), 4096, 4096, [8])
    assert e.value.code == L.LORA_E_INDEX
    assert len(L.lora_plan_inspect(L.Batch([0, 5], [-1]), 4096, 4096, [8])) == 0
