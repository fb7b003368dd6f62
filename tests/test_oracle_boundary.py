"""Pins for the oracle's BOUNDARY distribution (paper section 3.4, Tier 1:
generated inputs cover boundary values).

The sixteen patterns per element type are this library's definition; what
pins them here is numpy / torch: each pattern is checked by the value class it
decodes to (signed zeros, smallest and largest subnormals, smallest normal,
+-1 and its neighbours, +-largest finite, infinities, quiet and signalling
NaN) using finfo / iinfo and nextafter, not by retyping the bit table.  The
selection rate and the distribution of the other elements are pinned by
binomial bands, a chi-square test over the sixteen patterns and a
Kolmogorov-Smirnov test against N(0, sigma^2)."""
import math

import numpy as np
import pytest
import torch
from scipy import stats

import oracle
from workloads import Alloc, Compare, Injection, Workload

FLOATS = ("f32", "bf16", "f16", "fp8e4m3")
TORCH_T = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16,
           "fp8e4m3": torch.float8_e4m3fn}
NP_UINT = {1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}


def _fill(dtype, n, rate, sigma=1.0, seed=0xB0B, alloc_id=5, injections=(), variant=0):
    w = Workload("t", "", seed, [Alloc(alloc_id, dtype, 1, n, n, 0, 0, "boundary", rate, sigma)],
                 list(injections), [])
    P = oracle.Prepared(w)
    return w, P.fill_arena(variant)[:w.allocs[0].data_bytes]


def _float_values(dtype, raw):
    t = torch.from_numpy(raw.copy())
    return t.view(TORCH_T[dtype]).double().numpy()


def _expected_float_classes(dtype):
    """The sixteen patterns by position, as (value, sign bit); a NaN pattern
    has "nan", "qnan" or "snan" in place of the value."""
    if dtype == "f32":
        fi = np.finfo(np.float32)
        sub_min, tiny, fmax = float(fi.smallest_subnormal), float(fi.tiny), float(fi.max)
        below1 = float(np.nextafter(np.float32(1), np.float32(0)))
        above1 = float(np.nextafter(np.float32(1), np.float32(2)))
    elif dtype == "f16":
        fi = np.finfo(np.float16)
        sub_min, tiny, fmax = float(fi.smallest_subnormal), float(fi.tiny), float(fi.max)
        below1 = float(np.nextafter(np.float16(1), np.float16(0)))
        above1 = float(np.nextafter(np.float16(1), np.float16(2)))
    else:
        fi = torch.finfo(TORCH_T[dtype])
        sub_min, tiny, fmax = float(fi.smallest_normal) * fi.eps, float(fi.smallest_normal), float(fi.max)
        below1, above1 = 1.0 - fi.eps / 2, 1.0 + fi.eps
    sub_max = tiny - sub_min
    inf = math.inf
    rows = [(0.0, 0), (0.0, 1), (sub_min, 0), (-sub_min, 1), (sub_max, 0), (tiny, 0), (1.0, 0), (-1.0, 1),
            (below1, 0), (above1, 0), (fmax, 0), (-fmax, 1)]
    if dtype == "fp8e4m3":
        second = float(torch.tensor(fmax).to(TORCH_T[dtype]).view(torch.uint8).sub(1)
                        .view(TORCH_T[dtype]).double())
        rows += [("nan", 0), ("nan", 1), ("nan", 0), (second, 0)]
    else:
        rows += [(inf, 0), (-inf, 1), ("qnan", 0), ("snan", 0)]
    return rows


@pytest.mark.parametrize("dtype", FLOATS)
def test_float_patterns_are_the_stated_value_classes(dtype):
    n = 1 << 14
    w, raw = _fill(dtype, n, 1.0)
    es = w.allocs[0].esize
    bits = raw.view(NP_UINT[es]).astype(np.uint64)
    vals = _float_values(dtype, raw)
    exp = _expected_float_classes(dtype)
    # each expected class occurs, and nothing else does
    sign = ((bits >> np.uint64(8 * es - 1)) & np.uint64(1)).astype(np.int64)
    isnan = np.isnan(vals)
    for v, s in exp:
        if isinstance(v, str):
            hit = isnan & (sign == s)
            if v in ("qnan", "snan"):
                quiet = np.uint64(1 << ({"f32": 23, "bf16": 7, "f16": 10}[dtype] - 1))
                hit &= ((bits & quiet) != 0) == (v == "qnan")
        else:
            hit = ~isnan & (vals == v) & (sign == s)
        assert hit.any(), (dtype, v, s)
    allowed = np.zeros(n, dtype=bool)
    for v, s in exp:
        if not isinstance(v, str):
            allowed |= ~isnan & (vals == v) & (sign == s)
    assert np.all(allowed | isnan)
    # the sixteen positions are drawn uniformly: chi-square over bit patterns
    # (fp8 repeats 0x7F at two positions: its expected count is doubled)
    uniq, cnt = np.unique(bits, return_counts=True)
    expect = np.array([(2 if (dtype == "fp8e4m3" and u == 0x7F) else 1) * n / 16 for u in uniq.tolist()])
    assert len(uniq) == (15 if dtype == "fp8e4m3" else 16)
    assert stats.chisquare(cnt, expect).pvalue > 1e-4


@pytest.mark.parametrize("dtype,np_t", [("i32", np.int32), ("i64", np.int64), ("u8", np.uint8)])
def test_integer_patterns_include_the_extremes(dtype, np_t):
    n = 1 << 13
    _, raw = _fill(dtype, n, 1.0)
    got = set(raw.view(np_t).tolist())
    ii = np.iinfo(np_t)
    if dtype == "u8":
        expect = {0, 1, 255, 128, 127, 129, 126}
    else:
        expect = {0, 1, -1, int(ii.min), int(ii.max), int(ii.min) + 1, int(ii.max) - 1}
    assert expect <= got
    assert len(got) == 16
    # half of the remaining patterns are the alternating bit patterns
    width = 8 * np.dtype(np_t).itemsize
    alt = int("01" * (width // 2), 2)
    alt_vals = {alt, (~alt) & ((1 << width) - 1)}
    got_u = {v & ((1 << width) - 1) for v in got}
    assert alt_vals <= got_u


@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32"])
@pytest.mark.parametrize("rate", [0.0, 0.01, 0.25])
def test_rate_and_other_elements(dtype, rate):
    n = 200_000
    sigma = 3.0
    w, raw = _fill(dtype, n, rate, sigma)
    es = w.allocs[0].esize
    if dtype == "i32":
        _, raw1 = _fill(dtype, n, 1.0, sigma)
        patterns = set(raw1.view(np.uint32).tolist())
        v = raw.view(np.uint32)
        hits = np.isin(v, np.array(sorted(patterns), dtype=np.uint32))
        # a raw 32-bit draw equals one of 16 patterns with probability 16 / 2^32
        k = int(hits.sum())
        assert abs(k - rate * n) <= 5 * math.sqrt(n * rate * (1 - rate)) + 2
        # other elements: uniform bits
        other = v[~hits]
        assert stats.chisquare(np.bincount((other & 0xFF).astype(np.int64), minlength=256)).pvalue > 1e-4
        return
    # bit patterns of the sixteen (pinned by value class above), minus the
    # +-1 family that N(0, sigma^2) values can also round to
    _, raw1 = _fill(dtype, 4096, 1.0, sigma)
    uint = NP_UINT[es]
    pats = np.unique(raw1.view(uint))
    v1 = _float_values(dtype, raw1)
    ones = np.unique(raw1.view(uint)[np.isfinite(v1) & (np.abs(v1) >= 0.5) & (np.abs(v1) <= 2.0)])
    assert ones.size == 4
    strict_pats = np.setdiff1d(pats, ones)
    assert strict_pats.size == 12
    v = raw.view(uint)
    hits = np.isin(v, strict_pats)
    k = int(hits.sum())
    p = rate * 12 / 16
    assert abs(k - p * n) <= 5 * math.sqrt(n * p * (1 - p)) + 2, (k, p * n)
    # the others: N(0, sigma^2) rounded to the type
    vals = _float_values(dtype, raw)[~hits & ~np.isin(v, ones)]
    assert stats.kstest(vals / sigma, "norm").pvalue > 1e-4


def test_boundary_values_through_the_compare():
    """A boundary-filled reference against candidates with bit flips and NaN /
    Inf injections: the oracle's counts equal a numpy rendering of the
    tolerance rule on the decoded values."""
    n = 50_000
    atol, rtol = 1e-3, 1e-3
    for dtype in ("f32", "bf16", "f16", "fp8e4m3"):
        inj = [Injection(0, "flip_bit", arg=-1, rate=0.02),
               Injection(0, "step_within", rate=0.01, atol=atol, rtol=rtol),
               Injection(0, "set_nan", rate=0.001)]
        if dtype != "fp8e4m3":
            inj.append(Injection(0, "set_inf", arg=1, rate=0.001))
        w = Workload("t", "", 77, [Alloc(1, dtype, 1, n, n, 0, 0, "boundary", 0.2, 2.0)], inj,
                     [Compare(0, "tolerance", "equal", atol, rtol)])
        P = oracle.Prepared(w)
        ref = P.fill_arena(0)
        cand = P.fill_arena(1)
        r = oracle.diff_workload(w, cand, ref)[0]
        es = w.allocs[0].esize
        ra = ref[:n * es]
        ca = cand[:n * es]
        A = _float_values(dtype, ca)
        B = _float_values(dtype, ra)
        same_bits = ra.view(NP_UINT[es]) == ca.view(NP_UINT[es])
        nan_a, nan_b = np.isnan(A), np.isnan(B)
        with np.errstate(invalid="ignore", over="ignore"):
            close = np.abs(A - B) <= atol + rtol * np.abs(B)
        finite = np.isfinite(A) & np.isfinite(B)
        match = np.where(same_bits, True,
                         np.where(nan_a | nan_b, nan_a & nan_b,
                                  np.where(finite, close, False)))
        mism = np.flatnonzero(~match)
        assert r["mismatches"] == mism.size, dtype
        assert r["first_mismatch"] == (int(mism[0]) if mism.size else -1)
        assert r["bitwise_mismatches"] == int((~same_bits).sum())
        assert r["nonfinite_mismatches"] == int((~match & ~finite).sum())
        with np.errstate(invalid="ignore"):
            d = np.abs(A - B)[finite]
        assert r["max_abs"] == (float(d.max()) if d.size else 0.0)


def test_step_within_leaves_nonfinite_boundary_values_alone():
    n = 4096
    inj = [Injection(0, "step_within", rate=1.0, atol=0.0, rtol=0.0)]
    w, ref = _fill("f16", n, 1.0, injections=inj)
    _, cand = _fill("f16", n, 1.0, injections=inj, variant=1)
    A = _float_values("f16", cand)
    B = _float_values("f16", ref)
    keep = ~np.isfinite(B)
    assert keep.any()
    assert np.array_equal(cand.view(np.uint16)[keep], ref.view(np.uint16)[keep])
    # finite ones moved by one unit in the last place, away from or toward zero
    fin = np.isfinite(B)
    step = np.abs(cand.view(np.uint16)[fin].astype(np.int64) - ref.view(np.uint16)[fin].astype(np.int64))
    # +-0 steps to the smallest subnormal of its sign: one unit as well
    assert set(step.tolist()) == {1}
    assert np.all(np.isfinite(A[fin]) | (np.abs(B[fin]) == float(np.finfo(np.float16).max)))
