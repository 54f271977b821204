"""Comparison of HIP outputs with the oracle (test helper).

Tolerance (16-bit outputs, against the oracle's unrounded double result):
  * relative Frobenius error  ||gpu - ref|| / ||ref||  <= 2e-3;
  * per element |gpu - ref| <= max(3e-2, ulp(ref)/2 + 1e-5 |ref|), where ulp
    is the storage format's unit in the last place at |ref|.  The second term
    is the rounding every correct 16-bit result may carry: for bfloat16 with
    |ref| >= 8 half an ulp is 2^-5 > 3e-2, so a literal 3e-2 would fail
    correctly rounded results.
A stricter check rides along: against the oracle rounded once to the storage
format, at most 1% of the elements differ at all (they may only where the
exact value sits next to a rounding boundary and the kernel's arithmetic lands
on the other side), and each that differs is the neighbouring 16-bit value or
within one ulp plus the kernel's own error bound.  That bound follows from
its arithmetic: the expand feeds v to the MFMA as a high and a low 16-bit part
whose sum is v to a relative 2^-16 (bfloat16: 8 + 8 significant bits; 2^-22
for binary16), and the float32 sums over the rank and over h_in add about
r 2^-24 and h_in 2^-24 of their terms' magnitudes.  So the delta's error is at
most about 2^-15 times M = s_g sum_j |v_j| |B_jn| (plus the shrink's share).
The check allows ulp(ref) + 2^-14 M (``mag``, from the oracle's v); where y and
the delta nearly cancel that is several ulps of the small result.  Without
``mag`` the allowance is one ulp plus 1e-5 times the output's RMS.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2401_11240_amd import workloads as W

REL_FROB = 2e-3
MAX_ABS = 3e-2


def ulp(ref: np.ndarray, dtype: int) -> np.ndarray:
    a = np.abs(ref)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    if dtype == W.F16:
        return 2.0 ** (np.maximum(e, -14) - 10)
    return 2.0 ** (np.maximum(e, -126) - 7)


def bits_to_f64(bits: np.ndarray, dtype: int) -> np.ndarray:
    return W.bits_to_f32(bits, dtype).astype(np.float64)


def magnitude(w, name: str) -> np.ndarray:
    """M[t, n] = s_g sum_j |v_tj| |B_g[j, n]| for rows with adapter g (0
    elsewhere), v from the oracle's shrink: the scale of the terms the
    delta's float32 sums add up."""
    p = w.projection(name)
    v = oracle.lora_shrink(w.seg_offset, w.seg_adapter, w.xs[p.x], p.A, w.ranks, w.dtype)
    ra = w.row_adapter()
    out = np.zeros((w.n_rows, p.h_out), dtype=np.float64)
    for g in np.unique(ra[ra >= 0]):
        rows = np.nonzero(ra == g)[0]
        r = int(w.ranks[g])
        b = np.abs(W.bits_to_f32(p.B[g], w.dtype).astype(np.float64)).reshape(r, p.h_out)
        out[rows] = float(w.scales[g]) * (np.abs(v[rows, :r]) @ b)
    return out


def compare(gpu_bits: np.ndarray, ref: np.ndarray, dtype: int, what: str = "", mag=None) -> dict:
    gpu = bits_to_f64(gpu_bits, dtype)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite output"
    err = gpu - ref
    nref = np.linalg.norm(ref)
    rel = float(np.linalg.norm(err) / nref) if nref > 0 else float(np.linalg.norm(err))
    bound = np.maximum(MAX_ABS, 0.5 * ulp(ref, dtype) + 1e-5 * np.abs(ref))
    worst = float(np.max(np.abs(err) / bound)) if err.size else 0.0
    rounded = oracle.round_bits(ref, dtype)
    diff = gpu_bits != rounded
    frac = float(diff.mean()) if diff.size else 0.0
    one_ulp = True
    bad = ""
    if diff.any():
        gi = gpu_bits[diff].astype(np.int32)
        ri = rounded[diff].astype(np.int32)
        # same sign: neighbouring patterns differ by one in the integer
        # encoding; across zero, the error itself is below one ulp
        same_sign = (gi & 0x8000) == (ri & 0x8000)
        if mag is None:
            rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
            extra = 1e-5 * rms
        else:
            extra = 2.0 ** -14 * np.asarray(mag, dtype=np.float64)[diff]
        ok = (same_sign & (np.abs(gi - ri) <= 1)) | (
            np.abs(err[diff]) <= ulp(ref[diff], dtype) * 1.0001 + extra)
        one_ulp = bool(np.all(ok))
        if not one_ulp:
            idx = np.argwhere(diff)[~ok][:5]
            bad = "; ".join(f"{tuple(int(v) for v in i)}: gpu={gpu[tuple(i)]!r} ref={ref[tuple(i)]!r}"
                            for i in idx)
    stats = dict(rel_frob=rel, max_abs=float(np.max(np.abs(err))) if err.size else 0.0,
                 worst_over_bound=worst, frac_not_rne=frac)
    assert rel <= REL_FROB, f"{what}: rel Frobenius {rel:.3e} > {REL_FROB} ({stats})"
    assert worst <= 1.0, f"{what}: element error beyond bound ({stats})"
    assert one_ulp, f"{what}: a result is more than one ulp from the rounded oracle ({stats}) {bad}"
    assert frac <= 0.01, f"{what}: {frac:.4f} of results differ from the rounded oracle ({stats})"
    return stats


def compare_v(gpu_v: np.ndarray, ref_v: np.ndarray, what: str = "") -> dict:
    """float32 shrink result against the double oracle."""
    err = gpu_v.astype(np.float64) - ref_v
    n = np.linalg.norm(ref_v)
    rel = float(np.linalg.norm(err) / n) if n > 0 else float(np.linalg.norm(err))
    mx = float(np.max(np.abs(err))) if err.size else 0.0
    scale = float(np.max(np.abs(ref_v))) if ref_v.size else 1.0
    assert rel <= 1e-5, f"{what}: v rel Frobenius {rel:.3e}"
    assert mx <= 1e-4 * max(scale, 1e-30) + 1e-30, f"{what}: v max abs {mx:.3e}"
    return dict(rel_frob=rel, max_abs=mx)
