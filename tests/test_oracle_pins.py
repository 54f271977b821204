"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each pin is chosen so that a plausible slip in the oracle (a dropped term, a
swapped index, a transposed factor, a wrong adapter, a double rounding) makes
at least one of them fail.  No test here needs a GPU.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from paper_2401_11240_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _bits(vals, dtype):
    a = np.asarray(vals, dtype=np.float32)
    return W.to_bits(a, dtype)


# ---------------------------------------------------------------------------
# 16-bit formats
# ---------------------------------------------------------------------------

def test_widen_f16_all_patterns_match_numpy():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.widen(bits, oracle.F16)
    ref = bits.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


def test_widen_bf16_all_patterns_match_torch():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.widen(bits, oracle.BF16)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


def test_round_f16_matches_numpy_direct_from_double():
    rng = np.random.default_rng(7)
    vals = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.integers(-9, 6, 20000),
        np.array([0.0, -0.0, 65504.0, 65519.99, 65520.0, 1e6, -1e6, 2.0 ** -24, 2.0 ** -25,
                  2.0 ** -25 * 1.0000001, 3 * 2.0 ** -26, 6.1e-5, 1.0 + 2.0 ** -11,
                  1.0 + 3 * 2.0 ** -11, 1.0 + 2.0 ** -11 + 2.0 ** -40]),
    ])
    # halfway points between neighbouring halves: ties go to the even neighbour
    h = np.arange(0x0001, 0x7BFF, 97, dtype=np.uint16)
    lo = h.view(np.float16).astype(np.float64)
    hi = (h + 1).view(np.float16).astype(np.float64)
    vals = np.concatenate([vals, (lo + hi) / 2, -(lo + hi) / 2])
    got = oracle.round_bits(vals, oracle.F16)
    with np.errstate(over="ignore"):
        ref = vals.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, ref)


def test_round_bf16_brute_force_midpoints():
    """Every positive finite bfloat16 b: b itself is fixed; the midpoint to the
    next value goes to the even one; a hair off the midpoint goes to the
    nearer one."""
    b = np.arange(0x0001, 0x7F7F, dtype=np.uint16)
    lo = (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    hi = ((b.astype(np.uint32) + 1) << 16).view(np.float32).astype(np.float64)
    mid = (lo + hi) / 2
    eps = (hi - lo) * 2.0 ** -20
    assert np.array_equal(oracle.round_bits(lo, oracle.BF16), b)
    even = np.where(b % 2 == 0, b, b + 1).astype(np.uint16)
    assert np.array_equal(oracle.round_bits(mid, oracle.BF16), even)
    assert np.array_equal(oracle.round_bits(mid - eps, oracle.BF16), b)
    assert np.array_equal(oracle.round_bits(mid + eps, oracle.BF16), (b + 1).astype(np.uint16))
    assert np.array_equal(oracle.round_bits(-mid, oracle.BF16), (even | 0x8000).astype(np.uint16))
    # overflow: beyond max finite + half a unit (2^119) goes to infinity,
    # just below it stays at max finite
    mx = float((np.uint32(0x7F7F) << 16).view(np.float32))
    assert oracle.round_bits(np.array([mx + 2.0 ** 119 * 1.01]), oracle.BF16)[0] == 0x7F80
    assert oracle.round_bits(np.array([mx + 2.0 ** 119 * 0.99]), oracle.BF16)[0] == 0x7F7F


def test_round_bf16_matches_torch_on_float32_inputs():
    # From float32 inputs a single rounding is what torch does too.
    rng = np.random.default_rng(3)
    f = (rng.standard_normal(50000) * 10.0 ** rng.integers(-30, 30, 50000)).astype(np.float32)
    got = oracle.round_bits(f.astype(np.float64), oracle.BF16)
    ref = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, ref)


# ---------------------------------------------------------------------------
# grouping of rows by adapter
# ---------------------------------------------------------------------------

def test_group_rows_hand_worked_example():
    g = _golden("group_rows.json")
    perm, goff, gad = oracle.group_rows(g["n_rows"], g["seg_offset"], g["seg_adapter"])
    assert perm.tolist() == g["perm"]
    assert goff.tolist() == g["group_off"]
    assert gad.tolist() == g["group_adapter"]


@pytest.mark.parametrize("seed", range(20))
def test_group_rows_properties_random(seed):
    rng = np.random.default_rng(seed)
    S = int(rng.integers(0, 40))
    lens = rng.integers(0, 5, S)
    sa = rng.integers(-1, 6, S).astype(np.int32)
    so = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(so[-1])
    row_ad = np.repeat(sa, lens)
    perm, goff, gad = oracle.group_rows(T, so, sa)
    active = np.nonzero(row_ad >= 0)[0]
    assert sorted(perm.tolist()) == active.tolist()
    assert len(set(gad.tolist())) == len(gad)
    firsts = []
    for g in range(len(gad)):
        rows = perm[goff[g]:goff[g + 1]]
        assert len(rows) > 0
        assert np.all(np.diff(rows) > 0)
        assert np.all(row_ad[rows] == gad[g])
        firsts.append(rows[0])
        # first use of this adapter is this group's first row
        assert rows[0] == np.nonzero(row_ad == gad[g])[0][0]
    assert firsts == sorted(firsts)


# ---------------------------------------------------------------------------
# the delta
# ---------------------------------------------------------------------------

def _tiny_from_golden():
    g = _golden("tiny_delta.json")
    dt = W.F16
    x = _bits(g["x"], dt)
    y = _bits(g["y"], dt)
    A = [_bits(a, dt) for a in g["A"]]
    B = [_bits(b, dt) for b in g["B"]]
    return g, dt, x, y, A, B


def test_apply_hand_worked_example():
    g, dt, x, y, A, B = _tiny_from_golden()
    out = oracle.lora_apply(g["seg_offset"], g["seg_adapter"], x, A, B, g["ranks"], g["scales"], y, dt)
    assert out.tolist() == g["out_expected"]


def test_shrink_hand_worked_example():
    g, dt, x, y, A, B = _tiny_from_golden()
    v = oracle.lora_shrink(g["seg_offset"], g["seg_adapter"], x, A, g["ranks"], dt, ldv=2)
    for t, row in enumerate(g["v_expected"]):
        for j, val in enumerate(row):
            if val is None:
                continue
            assert v[t, j] == val


def _rand_small(rng, dtype, h_in, h_out, n_ad, ranks, T, with_none=True):
    lo = -1 if with_none else 0
    sa = rng.integers(lo, n_ad, T).astype(np.int32)
    so = np.arange(T + 1, dtype=np.int32)
    x = W.normal_bits(rng, (T, h_in), 1.0, dtype)
    y = W.normal_bits(rng, (T, h_out), 1.0, dtype)
    A = [W.normal_bits(rng, (h_in, r), 1 / np.sqrt(h_in), dtype) for r in ranks]
    B = [W.normal_bits(rng, (r, h_out), 1 / np.sqrt(r), dtype) for r in ranks]
    scales = (rng.random(n_ad) * 3 + 0.5).astype(np.float32)
    return so, sa, x, y, A, B, np.asarray(ranks, np.int32), scales


def _small_ints(rng, shape, lo=-4, hi=5):
    return rng.integers(lo, hi, shape).astype(np.int64)


@pytest.mark.parametrize("dtype", [W.F16, W.BF16])
@pytest.mark.parametrize("seed", range(4))
def test_apply_exact_integers_vs_merged_weight(dtype, seed):
    """Small-integer inputs make every product and sum exact in double; the
    exact result through the merged weight W' = A.B (Eq. 1's right-hand side,
    other association) in Python integers must equal the oracle exactly."""
    rng = np.random.default_rng(100 + seed)
    h_in, h_out, n_ad = 6, 5, 3
    ranks = [1, 3, 8]
    T = 7
    sa = rng.integers(-1, n_ad, T).astype(np.int32)
    so = np.arange(T + 1, dtype=np.int32)
    xi = _small_ints(rng, (T, h_in))
    yi = _small_ints(rng, (T, h_out), -16, 17)
    Ai = [_small_ints(rng, (h_in, r)) for r in ranks]
    Bi = [_small_ints(rng, (r, h_out)) for r in ranks]
    scales = np.array([0.5, 2.0, 0.25], dtype=np.float32)
    to = lambda a: _bits(a, dtype)
    out = oracle.lora_apply(so, sa, to(xi), [to(a) for a in Ai], [to(b) for b in Bi], ranks,
                            scales, to(yi), dtype)
    for t in range(T):
        g = int(sa[t])
        for n in range(h_out):
            exact = Fraction(int(yi[t, n]))
            if g >= 0:
                merged = [sum(int(Ai[g][k, j]) * int(Bi[g][j, n]) for j in range(ranks[g]))
                          for k in range(h_in)]
                exact += Fraction(float(scales[g])) * sum(int(xi[t, k]) * merged[k] for k in range(h_in))
            assert Fraction(out[t, n]) == exact, (t, n)


@pytest.mark.parametrize("dtype", [W.F16, W.BF16])
def test_merge_identity_fp64(dtype):
    """x.(W + s.A.B) == x.W + s.(x.A).B (Eq. 1) with W dense and random."""
    rng = np.random.default_rng(11)
    h, r, T = 256, 8, 5
    x = W.normal_bits(rng, (T, h), 1.0, dtype)
    A = W.normal_bits(rng, (h, r), 1 / np.sqrt(h), dtype)
    B = W.normal_bits(rng, (r, h), 1 / np.sqrt(r), dtype)
    Wd = rng.standard_normal((h, h)) / np.sqrt(h)
    s = 1.75
    xd, Ad, Bd = (oracle.widen(a, dtype) for a in (x, A, B))
    lhs = xd @ (Wd + s * (Ad @ Bd))
    zero_y = np.zeros((T, h), dtype=np.uint16)
    delta = oracle.lora_apply([0, T], [0], x, [A], [B], [r], [s], zero_y, dtype)
    rhs = xd @ Wd + delta
    assert np.max(np.abs(lhs - rhs)) <= 1e-12 * np.max(np.abs(lhs))


def test_single_adapter_equals_dense_blas():
    rng = np.random.default_rng(5)
    dtype = W.BF16
    h_in, h_out, r, T = 40, 24, 7, 9
    x = W.normal_bits(rng, (T, h_in), 1.0, dtype)
    y = W.normal_bits(rng, (T, h_out), 1.0, dtype)
    A = W.normal_bits(rng, (h_in, r), 0.3, dtype)
    B = W.normal_bits(rng, (r, h_out), 0.3, dtype)
    s = 0.625
    out = oracle.lora_apply([0, 4, T], [0, 0], x, [A], [B], [r], [s], y, dtype)
    ref = oracle.widen(y, dtype) + s * ((oracle.widen(x, dtype) @ oracle.widen(A, dtype)) @ oracle.widen(B, dtype))
    np.testing.assert_allclose(out, ref, rtol=1e-13, atol=1e-13)


def test_zero_B_and_zero_A_leave_y_bit_identical():
    rng = np.random.default_rng(8)
    for dtype in (W.F16, W.BF16):
        so, sa, x, y, A, B, ranks, scales = _rand_small(rng, dtype, 32, 16, 3, [2, 5, 8], 10)
        zB = [np.zeros_like(b) for b in B]
        zA = [np.zeros_like(a) for a in A]
        for AA, BB in ((A, zB), (zA, B)):
            out = oracle.lora_apply(so, sa, x, AA, BB, ranks, scales, y, dtype)
            assert np.array_equal(oracle.round_bits(out, dtype), y)
            assert np.array_equal(out, oracle.widen(y, dtype))


def test_rows_without_adapter_are_untouched():
    rng = np.random.default_rng(9)
    so, sa, x, y, A, B, ranks, scales = _rand_small(rng, W.F16, 16, 16, 2, [4, 8], 12)
    sa[::2] = -1
    out = oracle.lora_apply(so, sa, x, A, B, ranks, scales, y, W.F16)
    none = np.nonzero(sa < 0)[0]
    assert np.array_equal(out[none], oracle.widen(y, W.F16)[none])
    some = np.nonzero(sa >= 0)[0]
    assert np.all(np.any(out[some] != oracle.widen(y, W.F16)[some], axis=1))


@pytest.mark.parametrize("seed", range(3))
def test_permutation_invariance_bit_exact(seed):
    rng = np.random.default_rng(200 + seed)
    so, sa, x, y, A, B, ranks, scales = _rand_small(rng, W.BF16, 48, 40, 4, [1, 3, 8, 16], 15)
    out = oracle.lora_apply(so, sa, x, A, B, ranks, scales, y, W.BF16)
    p = rng.permutation(15)
    out_p = oracle.lora_apply(so, sa[p], x[p], A, B, ranks, scales, y[p], W.BF16)
    assert np.array_equal(out_p, out[p])


def test_segments_equal_per_row_segments():
    """A long segment is the same as its rows each with the segment's adapter."""
    rng = np.random.default_rng(12)
    so_rows, sa_rows, x, y, A, B, ranks, scales = _rand_small(rng, W.F16, 24, 16, 3, [2, 4, 8], 9, False)
    so = np.array([0, 4, 5, 9], np.int32)
    sa = np.array([2, -1, 0], np.int32)
    rows_ad = np.repeat(sa, np.diff(so))
    a = oracle.lora_apply(so, sa, x, A, B, ranks, scales, y, W.F16)
    b = oracle.lora_apply(np.arange(10, dtype=np.int32), rows_ad, x, A, B, ranks, scales, y, W.F16)
    assert np.array_equal(a, b)


def test_power_of_two_scale_is_exact_and_linear():
    rng = np.random.default_rng(13)
    so, sa, x, y, A, B, ranks, scales = _rand_small(rng, W.F16, 32, 24, 3, [3, 8, 16], 8, False)
    zero_y = np.zeros_like(y)
    d1 = oracle.lora_apply(so, sa, x, A, B, ranks, np.ones(3, np.float32), zero_y, W.F16)
    d4 = oracle.lora_apply(so, sa, x, A, B, ranks, np.full(3, 4.0, np.float32), zero_y, W.F16)
    d_quarter = oracle.lora_apply(so, sa, x, A, B, ranks, np.full(3, 0.25, np.float32), zero_y, W.F16)
    assert np.array_equal(d4, 4.0 * d1)
    assert np.array_equal(d_quarter, 0.25 * d1)
    d3 = oracle.lora_apply(so, sa, x, A, B, ranks, np.full(3, 3.0, np.float32), zero_y, W.F16)
    np.testing.assert_allclose(d3, 3.0 * d1, rtol=1e-15, atol=1e-15)


def test_rank_concatenation_adds_deltas():
    rng = np.random.default_rng(14)
    dt = W.BF16
    h_in, h_out, T = 64, 32, 6
    x = W.normal_bits(rng, (T, h_in), 1.0, dt)
    A1 = W.normal_bits(rng, (h_in, 3), 0.2, dt)
    A2 = W.normal_bits(rng, (h_in, 5), 0.2, dt)
    B1 = W.normal_bits(rng, (3, h_out), 0.5, dt)
    B2 = W.normal_bits(rng, (5, h_out), 0.5, dt)
    zero_y = np.zeros((T, h_out), np.uint16)
    seg = ([0, T], [0])
    d1 = oracle.lora_apply(*seg, x, [A1], [B1], [3], [1.0], zero_y, dt)
    d2 = oracle.lora_apply(*seg, x, [A2], [B2], [5], [1.0], zero_y, dt)
    d12 = oracle.lora_apply(*seg, x, [np.concatenate([A1, A2], 1)], [np.concatenate([B1, B2], 0)],
                            [8], [1.0], zero_y, dt)
    np.testing.assert_allclose(d12, d1 + d2, rtol=1e-13, atol=1e-13)


def selector_adapters(h_in, h_out, ranks, dtype, rng):
    """A_g[k,j] = 1 iff k = c_g + j; B_g[j,n] = 1 iff n = e_g + j."""
    A, B, c, e = [], [], [], []
    for r in ranks:
        cg = int(rng.integers(0, h_in - r + 1))
        eg = int(rng.integers(0, h_out - r + 1))
        a = np.zeros((h_in, r), np.float32)
        b = np.zeros((r, h_out), np.float32)
        for j in range(r):
            a[cg + j, j] = 1.0
            b[j, eg + j] = 1.0
        A.append(W.to_bits(a, dtype))
        B.append(W.to_bits(b, dtype))
        c.append(cg)
        e.append(eg)
    return A, B, c, e


@pytest.mark.parametrize("dtype", [W.F16, W.BF16])
def test_selector_adapters_closed_form(dtype):
    """d[t,n] = s_g * x[t, c_g + n - e_g] for n in [e_g, e_g + r_g), else 0:
    pins which adapter each row uses and the [k,j] / [j,n] layouts."""
    rng = np.random.default_rng(15)
    h_in, h_out = 40, 48
    ranks = [1, 4, 8, 3]
    A, B, c, e = selector_adapters(h_in, h_out, ranks, dtype, rng)
    T = 11
    sa = rng.integers(-1, 4, T).astype(np.int32)
    so = np.arange(T + 1, dtype=np.int32)
    x = W.normal_bits(rng, (T, h_in), 1.0, dtype)
    scales = np.array([2.0, 0.5, 4.0, 1.0], np.float32)
    zero_y = np.zeros((T, h_out), np.uint16)
    out = oracle.lora_apply(so, sa, x, A, B, ranks, scales, zero_y, dtype)
    xd = oracle.widen(x, dtype)
    for t in range(T):
        g = int(sa[t])
        exp = np.zeros(h_out)
        if g >= 0:
            for n in range(e[g], e[g] + ranks[g]):
                exp[n] = scales[g] * xd[t, c[g] + n - e[g]]
        assert np.array_equal(out[t], exp), t


def test_apply_row_matches_full_apply():
    rng = np.random.default_rng(16)
    so, sa, x, y, A, B, ranks, scales = _rand_small(rng, W.BF16, 64, 48, 3, [8, 16, 5], 10)
    full = oracle.lora_apply(so, sa, x, A, B, ranks, scales, y, W.BF16)
    rows = [0, 3, 7, 9]
    part = oracle.lora_apply_rows(rows, so, sa, x, A, B, ranks, scales, y, W.BF16)
    assert np.array_equal(part, full[rows])


def test_shrink_then_expand_matches_apply():
    rng = np.random.default_rng(17)
    so, sa, x, y, A, B, ranks, scales = _rand_small(rng, W.F16, 64, 32, 3, [8, 16, 2], 10)
    v = oracle.lora_shrink(so, sa, x, A, ranks, W.F16)
    v32 = np.nan_to_num(v).astype(np.float32)
    out = oracle.lora_expand(so, sa, v32, B, ranks, scales, y, W.F16)
    full = oracle.lora_apply(so, sa, x, A, B, ranks, scales, y, W.F16)
    np.testing.assert_allclose(out, full, rtol=1e-6, atol=1e-6)
    # brute force of the shrink itself on one row: plain Python sums
    xd = oracle.widen(x, W.F16)
    t = int(np.nonzero(sa >= 0)[0][0])
    g = int(sa[t])
    Ad = oracle.widen(A[g], W.F16)
    for j in range(ranks[g]):
        assert abs(v[t, j] - sum(xd[t, k] * Ad[k, j] for k in range(64))) <= 1e-12


# ---------------------------------------------------------------------------
# traffic accounting
# ---------------------------------------------------------------------------

def test_adapter_bytes_match_paper_worked_numbers():
    """Section 2.3 C1: a rank-64 Q/K/V adapter of Llama2-7B is about 100 MiB,
    about the KV cache of 200 tokens."""
    g = _golden("adapter_bytes.json")
    h, L, r = g["hidden"], g["layers"], g["rank"]
    per_rank = W.adapter_bytes_per_rank([(h, h)] * len(g["projections"]), L)
    total = per_rank * r
    mib = total / 2 ** 20
    assert abs(mib - g["approx_adapter_MiB"]) / g["approx_adapter_MiB"] < 0.05
    kv = 2 * L * h * 2 * g["kv_tokens"]
    assert abs(total - kv) / kv < 0.05


def test_algorithmic_bytes_counts_distinct_adapters_once():
    w = W.build_workload(name="t", seed=0, dtype=W.F16, n_adapters=3, fixed_ranks=[8, 16, 4],
                         seg_adapter=[0, 0, 1, -1, 0], projections=(("p", 32, 64, "x"),))
    # adapters 0 and 1 used; 4 adapted rows
    exp = 2 * ((8 + 16) * (32 + 64) + 4 * 32 + 4 * 2 * 64)
    assert W.algorithmic_bytes(w) == exp
    assert W.algorithmic_flops(w) == 2 * (8 * 3 + 16) * (32 + 64)


# ---------------------------------------------------------------------------
# Eq. 1 whole: the base projection with the delta (oracle.base_lora_apply)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", [W.F16, W.BF16])
@pytest.mark.parametrize("seed", range(4))
def test_base_lora_exact_integers_vs_merged_weight(dtype, seed):
    """x.W + s.(x.A).B equals x.(W + s.A.B) (Eq. 1, the merged weight W') in
    exact integer arithmetic; W is not square, so a transposed W fails."""
    rng = np.random.default_rng(300 + seed)
    h_in, h_out, n_ad = 6, 5, 3
    ranks = [2, 1, 4]
    T = 8
    sa = rng.integers(-1, n_ad, T).astype(np.int32)
    so = np.arange(T + 1, dtype=np.int32)
    xi = _small_ints(rng, (T, h_in))
    Wi = _small_ints(rng, (h_in, h_out), -6, 7)
    Ai = [_small_ints(rng, (h_in, r)) for r in ranks]
    Bi = [_small_ints(rng, (r, h_out)) for r in ranks]
    scales = np.array([0.5, 4.0, 0.125], dtype=np.float32)
    to = lambda a: _bits(a, dtype)
    out = oracle.base_lora_apply(so, sa, to(xi), to(Wi), [to(a) for a in Ai], [to(b) for b in Bi], ranks,
                                 scales, dtype)
    assert out.shape == (T, h_out)
    for t in range(T):
        g = int(sa[t])
        for n in range(h_out):
            merged = [Fraction(int(Wi[k, n])) for k in range(h_in)]
            if g >= 0:
                for k in range(h_in):
                    merged[k] += Fraction(float(scales[g])) * sum(int(Ai[g][k, j]) * int(Bi[g][j, n])
                                                                  for j in range(ranks[g]))
            exact = sum(int(xi[t, k]) * merged[k] for k in range(h_in))
            assert Fraction(out[t, n]) == exact, (t, n)


def test_base_lora_without_adapters_is_blas_matmul():
    """Rows with adapter -1 get x.W alone: numpy's BLAS product of the widened
    inputs (another implementation) agrees to double rounding."""
    rng = np.random.default_rng(21)
    dtype = W.BF16
    h_in, h_out, T = 96, 40, 11
    x = W.normal_bits(rng, (T, h_in), 1.0, dtype)
    Wb = W.normal_bits(rng, (h_in, h_out), 1 / np.sqrt(h_in), dtype)
    A = W.normal_bits(rng, (h_in, 8), 0.1, dtype)
    B = W.normal_bits(rng, (8, h_out), 0.1, dtype)
    out = oracle.base_lora_apply([0, T], [-1], x, Wb, [A], [B], [8], [1.0], dtype)
    ref = oracle.widen(x, dtype) @ oracle.widen(Wb, dtype)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_base_lora_with_zero_weight_is_the_delta():
    """W = 0 leaves s.(x.A).B: the delta oracle on a zero base output."""
    rng = np.random.default_rng(22)
    dtype = W.F16
    h_in, h_out, T = 48, 24, 6
    x = W.normal_bits(rng, (T, h_in), 1.0, dtype)
    ranks = [3, 8]
    A = [W.normal_bits(rng, (h_in, r), 0.2, dtype) for r in ranks]
    B = [W.normal_bits(rng, (r, h_out), 0.2, dtype) for r in ranks]
    so, sa = [0, 2, 3, 6], [1, -1, 0]
    out = oracle.base_lora_apply(so, sa, x, np.zeros((h_in, h_out), np.uint16), A, B, ranks, [2.0, 0.5], dtype)
    ref = oracle.lora_apply(so, sa, x, A, B, ranks, [2.0, 0.5], np.zeros((T, h_out), np.uint16), dtype)
    assert np.array_equal(out, ref)


def test_base_lora_brute_force_tiny():
    """Pure-Python loops of Eq. 1 on tiny shapes, in the order y' = xW + s(xA)B."""
    rng = np.random.default_rng(23)
    dtype = W.BF16
    h_in, h_out, T = 5, 7, 4
    ranks = [2, 3]
    x = W.normal_bits(rng, (T, h_in), 1.0, dtype)
    Wb = W.normal_bits(rng, (h_in, h_out), 0.5, dtype)
    A = [W.normal_bits(rng, (h_in, r), 0.5, dtype) for r in ranks]
    B = [W.normal_bits(rng, (r, h_out), 0.5, dtype) for r in ranks]
    so, sa, scales = [0, 1, 3, 4], [1, 0, -1], [0.75, 1.5]
    out = oracle.base_lora_apply(so, sa, x, Wb, A, B, ranks, scales, dtype)
    xf, Wf = oracle.widen(x, dtype), oracle.widen(Wb, dtype)
    row_ad = [1, 0, 0, -1]
    for t in range(T):
        g = row_ad[t]
        for n in range(h_out):
            base = sum(float(xf[t, k]) * float(Wf[k, n]) for k in range(h_in))
            d = 0.0
            if g >= 0:
                Af, Bf = oracle.widen(A[g], dtype), oracle.widen(B[g], dtype)
                v = [sum(float(xf[t, k]) * float(Af[k, j]) for k in range(h_in)) for j in range(ranks[g])]
                d = scales[g] * sum(v[j] * float(Bf[j, n]) for j in range(ranks[g]))
            assert abs(out[t, n] - (base + d)) <= 1e-12 * (1 + abs(base + d)), (t, n)
