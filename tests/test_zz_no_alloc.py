"""lora_apply_fused_static (the entry point that allocates nothing: its
workspace is the library's static device array) against lora_apply_fused
with a caller workspace and against the oracle, element by element, on two
calls in a row, the second with a smaller batch; device memory unchanged by
the calls; a batch too large for the array refused before anything runs."""
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


def test_static_scratch_entry_point_matches_workspace_entry_point():
    # one set of adapters; the first batch 64 decode tokens and a 90-row
    # prompt, the second 9 decode tokens over the same rows of x and y
    w = W.build_workload(name="static", seed=71, dtype=W.F16, n_adapters=24,
                         rank_set=[8, 16, 32, 64], adapter_law="zipf", n_segments=65,
                         seg_lens=[1] * 64 + [90], projections=(("proj", 4096, 4096, "x"),))
    dw = D.upload(w, DEV)
    p = dw.projection("proj")
    x = dw.xs["x"]
    so2 = np.arange(10, dtype=np.int32)
    sa2 = np.array([5, 0, -1, 3, 3, 17, 0, 1, 23], np.int32)
    batches = [(w.seg_offset, w.seg_adapter), (so2, sa2)]
    Lb = [L.Batch(so, sa) for so, sa in batches]
    refs = []
    for (so, sa), b in zip(batches, Lb):
        n = b.n_rows
        refs.append(oracle.lora_apply(so, sa, w.xs["x"][:n], p_A(w), p_B(w), w.ranks, w.scales,
                                      w.projections[0].y[:n], w.dtype))
    # the workspace entry point
    want = []
    for b in Lb:
        n = L.lora_workspace_bytes(p.table, b)
        ws = torch.empty(n, dtype=torch.uint8, device=DEV)
        y = p.y.clone()
        L.lora_apply_fused(p.table, b, x, x.shape[1], y, y.shape[1], ws, n, stream())
        torch.cuda.synchronize()
        want.append(D.from_device_bits(y))
        del ws
    ys = [p.y.clone(), p.y.clone()]
    # the first call on a device sets up (looks up the static array, which
    # the runtime maps with the library's code object); memory is measured
    # from there on
    L.lora_apply_fused_static(p.table, Lb[1], x, x.shape[1], ys[1], ys[1].shape[1], stream())
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info(DEV)[0]
    for rep in range(2):
        for y in ys:
            y.copy_(p.y)
        # two calls in a row, no synchronisation between them
        L.lora_apply_fused_static(p.table, Lb[0], x, x.shape[1], ys[0], ys[0].shape[1], stream())
        L.lora_apply_fused_static(p.table, Lb[1], x, x.shape[1], ys[1], ys[1].shape[1], stream())
        torch.cuda.synchronize()
        for i, b in enumerate(Lb):
            got = D.from_device_bits(ys[i])
            assert np.array_equal(got, want[i]), (rep, i)
            n = b.n_rows
            st = compare(got[:n], refs[i], w.dtype, f"static call {i}")
            assert np.array_equal(got[n:], w.projections[0].y[n:])
            say(f"  rep {rep} call {i}: {n} rows, {st}")
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info(DEV)[0] == free0
    # a batch whose workspace exceeds the static array (16384 prompt rows of a
    # rank-256 adapter): refused before anything runs, y untouched
    A = torch.zeros((4096, 256), dtype=torch.int16, device=DEV)
    B = torch.zeros((256, 4096), dtype=torch.int16, device=DEV)
    t2 = L.lora_register_adapters(0, 4096, 4096, W.F16, [A], [B], [256], [1.0], stream())
    try:
        big = L.Batch([0, 16384], [0])
        need = L.lora_workspace_bytes(t2, big)
        say(f"  large batch needs {need} bytes")
        assert need > 16 << 20
        xb = torch.zeros((16384, 4096), dtype=torch.int16, device=DEV)
        yb = torch.zeros((16384, 4096), dtype=torch.int16, device=DEV)
        with pytest.raises(L.LoraError) as e:
            L.lora_apply_fused_static(t2, big, xb, 4096, yb, 4096, stream())
        assert e.value.code == L.LORA_E_WORKSPACE
        torch.cuda.synchronize()
        assert int(yb.abs().sum()) == 0
    finally:
        L.lora_release_adapters(t2)
    dw.release()


def p_A(w):
    return w.projections[0].A


def p_B(w):
    return w.projections[0].B
