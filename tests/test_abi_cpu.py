"""The C-ABI library on the host: it loads, exports every symbol the header
declares, plans like the oracle groups, and rejects bad arguments before any
GPU work.  No GPU is needed (no compute call is made)."""
import os
import re

import numpy as np
import pytest

import oracle
from paper_2401_11240_amd import build as B
from paper_2401_11240_amd import lora as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def built():
    if not os.path.exists(B.lib_path()):
        B.build()
    L.load()


def header_functions():
    with open(os.path.join(ROOT, "include", "lora.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(lora_\w+)\s*\(", text, flags=re.M)))


def sched_header_functions():
    with open(os.path.join(ROOT, "include", "lora_sched.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|double)\s+(lora_\w+)\s*\(", text, flags=re.M)))


def cold_header_functions():
    with open(os.path.join(ROOT, "include", "lora_coldstart.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|double)\s+(lora_\w+)\s*\(", text, flags=re.M)))


def test_header_and_binding_agree():
    assert header_functions() == sorted(L.EXPORTS)
    from paper_2401_11240_amd import sched as SC
    assert sched_header_functions() == sorted(SC.EXPORTS)
    from paper_2401_11240_amd import coldstart as CS
    assert cold_header_functions() == sorted(CS.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = L.load()
    for name in header_functions():
        assert hasattr(lib, name), name
    # and from the dynamic symbol table itself
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", B.lib_path()], capture_output=True,
                         text=True, check=True).stdout
    syms = {ln.split()[-1] for ln in out.splitlines() if ln.strip()}
    for name in header_functions() + sched_header_functions() + cold_header_functions():
        assert name in syms, name


def test_abi_version():
    assert L.lora_abi_version() == 4


def test_group_rows_hand_example_matches_golden():
    import json
    with open(os.path.join(ROOT, "tests", "golden", "group_rows.json")) as f:
        g = json.load(f)
    perm, goff, gad = L.lora_group_rows(L.Batch(g["seg_offset"], g["seg_adapter"], g["n_rows"]), 3)
    assert perm.tolist() == g["perm"]
    assert goff.tolist() == g["group_off"]
    assert gad.tolist() == g["group_adapter"]


@pytest.mark.parametrize("seed", range(30))
def test_group_rows_bit_exact_vs_oracle(seed):
    rng = np.random.default_rng(1000 + seed)
    S = int(rng.integers(0, 80))
    lens = rng.integers(0, 6, S) if seed % 3 else np.ones(S, np.int64)
    n_ad = int(rng.integers(1, 12))
    sa = rng.integers(-1, n_ad, S).astype(np.int32)
    so = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    lib = L.lora_group_rows(L.Batch(so, sa), n_ad)
    ref = oracle.group_rows(int(so[-1]), so, sa)
    for a, b in zip(lib, ref):
        assert np.array_equal(a, b)


def test_group_rows_named_workloads_vs_oracle():
    from paper_2401_11240_amd import workloads as W
    for mk in (W.decode_q_proj_rank8, W.decode_mixed_rank):
        w = mk()
        lib = L.lora_group_rows(L.Batch(w.seg_offset, w.seg_adapter), w.n_adapters)
        ref = oracle.group_rows(w.n_rows, w.seg_offset, w.seg_adapter)
        for a, b in zip(lib, ref):
            assert np.array_equal(a, b)


@pytest.mark.parametrize("so,sa,code", [
    ([0, 2, 3], [0, 5], L.LORA_E_INDEX),       # adapter index too large
    ([0, 2, 3], [0, -2], L.LORA_E_INDEX),      # below -1
    ([1, 2, 3], [0, 1], L.LORA_E_SHAPE),       # first offset not zero
    ([0, 3, 2], [0, 1], L.LORA_E_SHAPE),       # decreasing offsets
])
def test_batch_validation_codes(so, sa, code):
    with pytest.raises(L.LoraError) as e:
        L.lora_group_rows(L.Batch(so, sa), 3)
    assert e.value.code == code
    assert L.lora_last_error()


def test_batch_n_rows_mismatch():
    with pytest.raises(L.LoraError) as e:
        L.lora_group_rows(L.Batch([0, 2, 3], [0, 1], n_rows=4), 3)
    assert e.value.code == L.LORA_E_SHAPE


def test_empty_batch_is_valid():
    perm, goff, gad = L.lora_group_rows(L.Batch([0], []), 3)
    assert perm.size == 0 and gad.size == 0 and goff.tolist() == [0]


# Registration arguments are checked before any device call, so these run on
# a machine without a GPU.
FAKE = 0x10000  # 16-byte aligned fake device address, never dereferenced


@pytest.mark.parametrize("kw,code", [
    (dict(h_in=4100), L.LORA_E_SHAPE),
    (dict(h_out=0), L.LORA_E_SHAPE),
    (dict(dtype=7), L.LORA_E_ARG),
    (dict(ranks=[0, 8]), L.LORA_E_RANK),
    (dict(ranks=[8, 257]), L.LORA_E_RANK),
    (dict(A_ptrs=[FAKE + 8, FAKE]), L.LORA_E_ALIGN),
    (dict(B_ptrs=[FAKE, 0]), L.LORA_E_ARG),
    (dict(device=-1), L.LORA_E_ARG),
])
def test_register_validation_codes(kw, code):
    args = dict(device=0, h_in=4096, h_out=4096, dtype=L.LORA_F16, A_ptrs=[FAKE, FAKE],
                B_ptrs=[FAKE, FAKE], ranks=[8, 16], scales=[1.0, 1.0])
    args.update(kw)
    with pytest.raises(L.LoraError) as e:
        L.lora_register_adapters(**args)
    assert e.value.code == code


def test_null_table_rejected():
    with pytest.raises(L.LoraError) as e:
        L.lora_workspace_bytes(None, L.Batch([0, 1], [0]))
    assert e.value.code == L.LORA_E_ARG
