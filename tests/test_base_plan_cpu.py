"""The fused base GEMM's schedule, checked on the host (no GPU):
lora_base_inspect reports the tile edge, the whole and K-split tiles and the
launch's grid that lora_base_apply would use.

Checked: the tile rule (tiles of 256 while they fill the compute units, else
128); a K split only of a last, partial round of tiles, in even ranges of at
least 8 stages that cover K; and, following the workgroup-to-tile mapping the
header states (XCD shares of the panel order, then the split tiles' ranges),
that the grid runs every tile's K exactly once and nothing else.  The two
named prompt workloads get the schedules their kernel traces record.
"""
import numpy as np
import pytest

from paper_2401_11240_amd import lora as L
from paper_2401_11240_amd import workloads as W

MIN_SPLIT_STAGES = 8


def ceil_div(a, b):
    return (a + b - 1) // b


def tile_coords(tile, n_mt, n_nt, panel):
    """Row and column tile of a tile index in the panel order (panels of
    `panel` row tiles, column by column inside a panel)."""
    per_panel = panel * n_nt
    pn = tile // per_panel
    h = min(panel, n_mt - pn * panel)
    u = tile - pn * per_panel
    nt = u // h
    return pn * panel + (u - nt * h), nt


def workgroup_work(info, n_xcd):
    """(tile, k0, k1) of every workgroup of the grid that runs work, by the
    mapping lora.h states."""
    slots = n_xcd * info["per_xcd"]
    n_tiles = info["n_mt"] * info["n_nt"]
    out = []
    for p in range(info["grid"]):
        if p < slots:
            q = p // n_xcd
            tile = (p - q * n_xcd) * info["per_xcd"] + q
            if tile < info["n_whole"]:
                out.append((tile, 0, info["n_stages"]))
        else:
            u = p - slots
            tile = info["n_whole"] + u // info["split"]
            r = u - (tile - info["n_whole"]) * info["split"]
            k0 = r * info["chunk"]
            k1 = min(info["n_stages"], k0 + info["chunk"])
            if tile < n_tiles and k0 < k1:
                out.append((tile, k0, k1))
    return out


def check_schedule(info, M, h_in, h_out, n_cu, n_xcd):
    big = ceil_div(M, 256) * ceil_div(h_out, 256)
    assert info["tile"] == (256 if big >= n_cu else 128)
    T = info["tile"]
    assert info["stage_k"] * T * 4 == 64 * 1024                     # 64 KiB stages
    assert info["n_mt"] == ceil_div(M, T) and info["n_nt"] == ceil_div(h_out, T)
    assert info["n_stages"] % 2 == 0 and (info["n_stages"] - 2) * info["stage_k"] < h_in <= info["n_stages"] * info["stage_k"]
    n_tiles = info["n_mt"] * info["n_nt"]
    if info["split"] > 1:
        assert info["n_whole"] % n_cu == 0 and info["n_whole"] < n_tiles
        assert info["chunk"] % 2 == 0 and info["chunk"] >= MIN_SPLIT_STAGES
        assert (info["split"] - 1) * info["chunk"] < info["n_stages"] <= info["split"] * info["chunk"]
        # the split round does not ask for more workgroups than compute units
        assert (n_tiles - info["n_whole"]) * info["split"] <= n_cu
        part = (n_tiles - info["n_whole"]) * info["split"] * T * T * 4
        assert info["workspace_bytes"] >= part
    else:
        assert info["n_whole"] == n_tiles
    # the panel order is a bijection of the tiles
    seen = {tile_coords(t, info["n_mt"], info["n_nt"], info["panel"]) for t in range(n_tiles)}
    assert len(seen) == n_tiles and all(0 <= m < info["n_mt"] and 0 <= n < info["n_nt"] for m, n in seen)
    # every tile's K exactly once
    cover = {}
    for tile, k0, k1 in workgroup_work(info, n_xcd):
        cover.setdefault(tile, []).append((k0, k1))
    assert sorted(cover) == list(range(n_tiles))
    for tile, ranges in cover.items():
        ranges.sort()
        at = 0
        for k0, k1 in ranges:
            assert k0 == at, (tile, ranges)
            at = k1
        assert at == info["n_stages"], (tile, ranges)


def batch_of(lens, adapters):
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    return L.Batch(off, adapters), int(off[-1])


def test_named_prompt_schedules():
    # the grids the kernel traces record: 640 workgroups (512 whole tiles of
    # 256, then 16 tiles x 8 K ranges) and 256 (whole tiles of 128)
    w = W.BASE_NAMED["prefill_base"]()
    p = w.projections[0]
    info = L.lora_base_inspect(L.Batch(w.seg_offset, w.seg_adapter), p.h_in, p.h_out, w.ranks, 256, 8)
    assert (info["tile"], info["n_whole"], info["split"], info["chunk"], info["grid"]) == (256, 512, 8, 8, 640)
    check_schedule(info, w.n_rows, p.h_in, p.h_out, 256, 8)
    w = W.BASE_NAMED["prefill_base_l1024"]()
    p = w.projections[0]
    info = L.lora_base_inspect(L.Batch(w.seg_offset, w.seg_adapter), p.h_in, p.h_out, w.ranks, 256, 8)
    assert (info["tile"], info["n_whole"], info["split"], info["grid"]) == (128, 256, 1, 256)
    check_schedule(info, w.n_rows, p.h_in, p.h_out, 256, 8)


@pytest.mark.parametrize("seed", range(40))
def test_random_schedules(seed):
    rng = np.random.default_rng(500 + seed)
    n_cu = int(rng.choice([64, 80, 256, 304]))
    n_xcd = int(rng.choice([1, 4, 8]))
    M_target = int(rng.choice([1, 7, 300, 1024, 2500, 4200, 9000]))
    n_seg = int(rng.integers(1, 6))
    cuts = np.sort(rng.choice(np.arange(1, M_target), size=min(n_seg - 1, max(M_target - 1, 0)), replace=False)) \
        if M_target > 1 else np.array([], dtype=int)
    lens = np.diff(np.concatenate([[0], cuts, [M_target]])).astype(int).tolist()
    ranks = [int(r) for r in rng.integers(1, 129, size=3)]
    adapters = [int(a) for a in rng.integers(-1, 3, size=len(lens))]
    h_in = 8 * int(rng.integers(1, 1100))
    h_out = 8 * int(rng.integers(1, 1100))
    b, M = batch_of(lens, adapters)
    info = L.lora_base_inspect(b, h_in, h_out, ranks, n_cu, n_xcd)
    check_schedule(info, M, h_in, h_out, n_cu, n_xcd)


def test_inspect_refuses_bad_shapes():
    b, _ = batch_of([5], [0])
    with pytest.raises(L.LoraError) as e:
        L.lora_base_inspect(b, 100, 64, [8], 256, 8)
    assert e.value.code == L.LORA_E_SHAPE
    with pytest.raises(L.LoraError) as e:
        L.lora_base_inspect(b, 64, 64, [300], 256, 8)
    assert e.value.code == L.LORA_E_RANK
