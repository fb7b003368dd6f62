"""Pins for the CPU oracle's comparison (paper section 3.2, Eq. 1 and iota) and
guard check (section 3.4): numpy.isclose (the same definition, evaluated by a
library), exhaustive small-dtype pair tables, the NaN/Inf truth table,
constructed exact tolerance boundaries, brute force over every (index, bit) of
tiny buffers and every byte of tiny guards, and invariants."""
import itertools

import numpy as np
import pytest
import torch

import oracle
from workloads import ESIZE


def _np_view(dtype, raw):
    """fp64 values of raw patterns via numpy / torch casts (not the oracle)."""
    raw = np.asarray(raw)
    if dtype == "f32":
        return raw.astype(np.uint32).view(np.float32).astype(np.float64)
    if dtype == "f16":
        return raw.astype(np.uint16).view(np.float16).astype(np.float64)
    if dtype == "bf16":
        return torch.from_numpy(raw.astype(np.uint16).view(np.int16)).view(torch.bfloat16).to(
            torch.float64).numpy()
    if dtype == "fp8e4m3":
        return torch.from_numpy(raw.astype(np.uint8)).view(torch.float8_e4m3fn).to(
            torch.float64).numpy()
    raise ValueError(dtype)


_NP_INT = {1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}


def _as_bytes(dtype, raw):
    return np.ascontiguousarray(np.asarray(raw).astype(_NP_INT[ESIZE[dtype]])).view(np.uint8)


def _diff(dtype, a_raw, b_raw, mode="tolerance", policy="equal", atol=0.0, rtol=0.0,
          rows=None, cols=None, sa=None, sb=None):
    a = _as_bytes(dtype, a_raw)
    b = _as_bytes(dtype, b_raw)
    n = len(a_raw)
    if rows is None:
        rows, cols, sa, sb = 1, n, n, n
    return oracle.diff_segment(dtype, mode, policy, rows, cols, sa, sb, atol, rtol, a, b)


def _expected_from_isclose(dtype, a_raw, b_raw, atol, rtol, equal_nan):
    A = _np_view(dtype, a_raw)
    B = _np_view(dtype, b_raw)
    with np.errstate(invalid="ignore", over="ignore"):
        close = np.isclose(A, B, rtol=rtol, atol=atol, equal_nan=equal_nan)
    mism = ~close
    return mism, A, B


def _check_against_isclose(dtype, a_raw, b_raw, atol, rtol, policy):
    res = _diff(dtype, a_raw, b_raw, policy=policy, atol=atol, rtol=rtol)
    mism, A, B = _expected_from_isclose(dtype, a_raw, b_raw, atol, rtol, policy == "equal")
    assert res["mismatches"] == int(mism.sum())
    idx = np.flatnonzero(mism)
    assert res["first_mismatch"] == (int(idx[0]) if idx.size else -1)
    bw = np.asarray(a_raw) != np.asarray(b_raw)
    assert res["bitwise_mismatches"] == int(bw.sum())
    bidx = np.flatnonzero(bw)
    assert res["first_bitwise"] == (int(bidx[0]) if bidx.size else -1)
    nonfin = ~(np.isfinite(A) & np.isfinite(B))
    assert res["nonfinite_mismatches"] == int((mism & nonfin).sum())
    return res


@pytest.mark.parametrize("atol,rtol", [(0.125, 0.125), (0.0, 0.0), (1e-3, 0.0), (0.0, 0.5)])
@pytest.mark.parametrize("policy", ["equal", "strict"])
def test_fp8_all_pairs_vs_isclose(atol, rtol, policy):
    a, b = np.meshgrid(np.arange(256, dtype=np.uint64), np.arange(256, dtype=np.uint64))
    _check_against_isclose("fp8e4m3", a.ravel(), b.ravel(), atol, rtol, policy)


@pytest.mark.parametrize("dtype,atol,rtol", [("bf16", 1e-2, 1.6e-2), ("f16", 1e-3, 1e-3)])
def test_16bit_pairs_strided_vs_isclose(dtype, atol, rtol):
    # every a against a strided sample of b (2^16 x 2^9 pairs)
    a = np.arange(1 << 16, dtype=np.uint64)
    for off in range(0, 1 << 16, 127):
        b = (a * 40503 + off) & 0xFFFF      # a permutation of the 16-bit patterns
        _check_against_isclose(dtype, a, b, atol, rtol, "equal")
        if off > 2000:
            break
    # neighbours: every pattern against the next one (1-ulp and sign-crossing pairs)
    _check_against_isclose(dtype, a, (a + 1) & 0xFFFF, atol, rtol, "equal")
    _check_against_isclose(dtype, a, a ^ 0x8000, atol, rtol, "strict")


def test_f32_random_vs_isclose():
    rng = np.random.default_rng(7)
    n = 1 << 18
    b = rng.standard_normal(n).astype(np.float32)
    a = b.copy()
    pert = rng.integers(0, n, size=n // 8)
    a[pert] += (rng.standard_normal(pert.size) * 1e-5).astype(np.float32)
    a_raw = a.view(np.uint32).astype(np.uint64)
    b_raw = b.view(np.uint32).astype(np.uint64)
    specials = np.array([0x7FC00000, 0x7F800000, 0xFF800000, 0x80000000, 0, 1, 0x7F7FFFFF],
                        dtype=np.uint64)
    a_raw[:49] = np.repeat(specials, 7)
    b_raw[:49] = np.tile(specials, 7)
    for policy in ("equal", "strict"):
        _check_against_isclose("f32", a_raw, b_raw, 1e-5, 1e-5, policy)


def test_nan_inf_truth_table():
    """Every ordered pair of {finite, +0, -0, +Inf, -Inf, qNaN, other NaN}."""
    vals = {"one": 0x3F800000, "pz": 0, "nz": 0x80000000, "pinf": 0x7F800000,
            "ninf": 0xFF800000, "qnan": 0x7FC00000, "nan2": 0xFFC00001}
    names = list(vals)
    for pa, pb in itertools.product(names, names):
        for policy in ("equal", "strict"):
            r = _diff("f32", [vals[pa]], [vals[pb]], policy=policy, atol=1e-5, rtol=1e-5)
            a_nan, b_nan = pa.endswith("nan") or pa == "nan2", pb.endswith("nan") or pb == "nan2"
            if a_nan or b_nan:
                expect = not (a_nan and b_nan and policy == "equal")
            elif pa in ("pinf", "ninf") or pb in ("pinf", "ninf"):
                expect = pa != pb
            else:
                # finite: 1 vs 1 and +0 vs -0 are within tolerance, 1 vs 0 is not
                expect = (pa == "one") != (pb == "one")
            assert r["mismatches"] == int(expect), (pa, pb, policy)
            assert r["bitwise_mismatches"] == int(vals[pa] != vals[pb])
            nonfin = pa not in ("one", "pz", "nz") or pb not in ("one", "pz", "nz")
            assert r["nonfinite_mismatches"] == int(expect and nonfin)


def test_signed_zero():
    r = _diff("f32", [0x80000000], [0], atol=0.0, rtol=0.0)
    assert r["mismatches"] == 0 and r["bitwise_mismatches"] == 1 and r["first_bitwise"] == 0
    assert r["max_abs"] == 0.0 and r["max_rel"] == 0.0


def test_tolerance_boundary_is_inclusive_and_exact():
    """b = 1, t = atol + rtol*1 with atol=2^-10, rtol=2^-12 (exact in fp64):
    a = b + t lies exactly on the boundary (match); the next fp32 above
    (mismatch)."""
    atol, rtol = 2.0 ** -10, 2.0 ** -12
    b = np.float32(1.0)
    a_on = np.float32(1.0 + atol + rtol)             # exactly representable
    a_over = np.nextafter(a_on, np.float32(2))
    a_under = np.nextafter(a_on, np.float32(0))
    raw = lambda v: int(np.float32(v).view(np.uint32))
    for a, expect in ((a_on, 0), (a_over, 1), (a_under, 0)):
        r = _diff("f32", [raw(a)], [raw(b)], atol=atol, rtol=rtol)
        assert r["mismatches"] == expect
    # boundary symmetry below b
    r = _diff("f32", [raw(1.0 - atol - rtol)], [raw(b)], atol=atol, rtol=rtol)
    assert r["mismatches"] == 0
    # rtol scales |b|, not |a|: b = 0, a = tiny -> only atol counts
    r = _diff("f32", [raw(2.0 ** -20)], [raw(0.0)], atol=0.0, rtol=1.0)
    assert r["mismatches"] == 1
    r = _diff("f32", [raw(0.0)], [raw(2.0 ** -20)], atol=0.0, rtol=1.0)
    assert r["mismatches"] == 0


def test_maxima_closed_forms():
    b = np.array([1.0, 2.0, -4.0, 0.0, 8.0, 3.0], dtype=np.float32)
    a = np.array([1.0, 2.5, -4.0, 0.25, 6.0, np.nan], dtype=np.float32)
    r = _diff("f32", a.view(np.uint32), b.view(np.uint32), atol=0.0, rtol=0.0)
    # finite pairs: |d| = 0, .5, 0, .25, 2 ; rel = 0, .25, 0, inf (b=0, d>0), .25
    assert r["max_abs"] == 2.0
    assert r["max_rel"] == float("inf")
    assert r["mismatches"] == 4 and r["first_mismatch"] == 1 and r["nonfinite_mismatches"] == 1
    b2 = np.array([4.0, 0.0, 1.0], dtype=np.float32)
    a2 = np.array([5.0, 0.0, 1.125], dtype=np.float32)
    r = _diff("f32", a2.view(np.uint32), b2.view(np.uint32), atol=1.0, rtol=0.0)
    assert r["max_abs"] == 1.0 and r["max_rel"] == 0.25 and r["mismatches"] == 0
    # relative error is d / |b| correctly rounded: 1/3
    r = _diff("f32", np.array([4.0], np.float32).view(np.uint32), np.array([3.0], np.float32).view(np.uint32))
    assert r["max_rel"] == 1.0 / 3.0


def test_bitwise_mode_fields():
    b = np.arange(10, dtype=np.uint32)
    a = b.copy()
    a[[3, 7]] ^= 1 << 31
    r = _diff("i32", a, b, mode="bitwise")
    assert r == {"mismatches": 2, "first_mismatch": 3, "bitwise_mismatches": 2, "first_bitwise": 3,
                 "nonfinite_mismatches": 0, "max_abs": 0.0, "max_rel": 0.0}
    with pytest.raises(ValueError):
        _diff("i32", a, b, mode="tolerance")


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16", "fp8e4m3", "i32", "i64", "u8"])
def test_single_bit_flip_every_index_and_bit(dtype):
    es = ESIZE[dtype]
    n = 5
    rng = np.random.default_rng(8)
    b = rng.integers(0, 1 << (8 * es) if es < 8 else 1 << 62, size=n, dtype=np.uint64)
    if dtype in ("f32", "bf16", "f16", "fp8e4m3"):
        # finite values only in the base
        _, vals = oracle.decode_n(dtype, b)
        cls, _ = oracle.decode_n(dtype, b)
        b[cls != 0] = 0
    for i in range(n):
        for bit in range(8 * es):
            a = b.copy()
            a[i] ^= np.uint64(1) << np.uint64(bit)
            r = _diff(dtype, a, b, mode="bitwise")
            assert r["bitwise_mismatches"] == 1 and r["first_bitwise"] == i
            assert r["mismatches"] == 1 and r["first_mismatch"] == i


def test_identical_buffers_give_zero_results():
    rng = np.random.default_rng(9)
    for dtype in ("f32", "bf16", "f16", "fp8e4m3"):
        raw = rng.integers(0, 1 << (8 * ESIZE[dtype]), size=4096, dtype=np.uint64)
        r = _diff(dtype, raw, raw, policy="equal", atol=0.0, rtol=0.0)
        assert r == {"mismatches": 0, "first_mismatch": -1, "bitwise_mismatches": 0,
                     "first_bitwise": -1, "nonfinite_mismatches": 0, "max_abs": 0.0, "max_rel": 0.0}


def test_strided_rows_skip_padding_and_use_logical_index():
    rows, cols, sa, sb = 3, 4, 6, 5
    b = np.zeros(rows * sb, dtype=np.uint32)
    a = np.zeros(rows * sa, dtype=np.uint32)
    a[1 * sa + 4] = 7          # padding of row 1: never read
    a[2 * sa + 1] = 5          # logical index 2*4+1 = 9
    r = _diff("i32", a, b, mode="bitwise", rows=rows, cols=cols, sa=sa, sb=sb)
    assert r["bitwise_mismatches"] == 1 and r["first_bitwise"] == 9


def test_invariants_monotone_split_and_policy():
    rng = np.random.default_rng(10)
    n = 50000
    b = (rng.standard_normal(n) * 3).astype(np.float16)
    a = b.copy()
    k = rng.integers(0, n, size=4000)
    a[k] = (a[k].astype(np.float32) * (1 + rng.standard_normal(k.size).astype(np.float32) * 1e-2)).astype(np.float16)
    a[k[:10]] = np.nan
    b[k[10:15]] = np.inf
    ar, br = a.view(np.uint16).astype(np.uint64), b.view(np.uint16).astype(np.uint64)
    prev = None
    for atol in (0.0, 1e-4, 1e-3, 1e-2, 1e-1):
        r = _diff("f16", ar, br, atol=atol, rtol=1e-3)
        if prev is not None:
            assert r["mismatches"] <= prev
        prev = r["mismatches"]
        assert r["mismatches"] <= r["bitwise_mismatches"]          # EQUAL policy
        if r["mismatches"]:
            assert r["first_mismatch"] >= r["first_bitwise"]
    # split additivity: counts add, first = min, maxima = max
    whole = _diff("f16", ar, br, atol=1e-3, rtol=1e-3)
    cut = 31337
    p1 = _diff("f16", ar[:cut], br[:cut], atol=1e-3, rtol=1e-3)
    p2 = _diff("f16", ar[cut:], br[cut:], atol=1e-3, rtol=1e-3)
    for f in ("mismatches", "bitwise_mismatches", "nonfinite_mismatches"):
        assert whole[f] == p1[f] + p2[f]
    for f in ("first_mismatch", "first_bitwise"):
        cands = [v for v in (p1[f], p2[f] + cut if p2[f] >= 0 else -1) if v >= 0]
        assert whole[f] == (min(cands) if cands else -1)
    assert whole["max_abs"] == max(p1["max_abs"], p2["max_abs"])
    assert whole["max_rel"] == max(p1["max_rel"], p2["max_rel"])
    # rtol = 0 and no non-finite: no mismatch <=> max_abs <= atol
    fin = np.isfinite(a) & np.isfinite(b)
    r = _diff("f16", ar[fin], br[fin], atol=0.01, rtol=0.0)
    assert (r["mismatches"] == 0) == (r["max_abs"] <= 0.01)
    # swapping a and b with rtol = 0 gives the same verdicts
    r2 = _diff("f16", br[fin], ar[fin], atol=0.01, rtol=0.0)
    assert r2["mismatches"] == r["mismatches"] and r2["max_abs"] == r["max_abs"]


def test_guard_check_every_byte_of_tiny_guards():
    seed, aid = 0x1234, 7
    n = 48
    lo = np.array([oracle.canary_byte(seed, aid, 0, p) for p in range(n)], dtype=np.uint8)
    hi = np.array([oracle.canary_byte(seed, aid, 1, p) for p in range(n)], dtype=np.uint8)
    assert oracle.guard_check(seed, aid, lo, hi) == {"bad_lo": 0, "bad_hi": 0,
                                                     "first_bad_lo": -1, "first_bad_hi": -1, "bad_pad": 0, "first_bad_pad": -1}
    assert not np.array_equal(lo, hi)          # the two sides carry different canaries
    for p in range(n):
        for side in (0, 1):
            l2, h2 = lo.copy(), hi.copy()
            (l2 if side == 0 else h2)[p] ^= 0x40
            r = oracle.guard_check(seed, aid, l2, h2)
            if side == 0:
                assert r == {"bad_lo": 1, "bad_hi": 0, "first_bad_lo": p, "first_bad_hi": -1, "bad_pad": 0, "first_bad_pad": -1}
            else:
                assert r == {"bad_lo": 0, "bad_hi": 1, "first_bad_lo": -1, "first_bad_hi": p, "bad_pad": 0, "first_bad_pad": -1}
    # another seed or buffer id gives other canaries
    assert oracle.guard_check(seed + 1, aid, lo, hi)["bad_lo"] > n // 2
    assert oracle.guard_check(seed, aid + 1, lo, hi)["bad_lo"] > n // 2


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16", "fp8e4m3"])
@pytest.mark.parametrize("policy", ["equal", "strict"])
def test_pairwise_bulk_equals_one_element_segments_and_numpy(dtype, policy):
    """The bulk per-pair loop (what the GPU's per-pair rule is compared with,
    pair by pair) against one-element segments of the oracle's own diff, and
    against numpy: isclose for the outcome, fp64 |A - B| and |A - B| / |B| for
    the maxima of finite pairs whose bits differ."""
    rng = np.random.default_rng(31)
    bits = 8 * ESIZE[dtype]
    a = rng.integers(0, 1 << bits, size=3000, dtype=np.uint64)
    b = a.copy()
    b[0::3] ^= np.uint64(1) << rng.integers(0, bits, size=b[0::3].size).astype(np.uint64)
    b[1::3] = rng.integers(0, 1 << bits, size=b[1::3].size, dtype=np.uint64)
    atol, rtol = 1e-3, 2.0 ** -7
    flags, mabs, mrel = oracle.compare_pair_n(dtype, "tolerance", policy, atol, rtol, a, b)
    for k in range(0, a.size, 7):
        r = _diff(dtype, a[k:k + 1], b[k:k + 1], policy=policy, atol=atol, rtol=rtol)
        assert flags[k] == (r["bitwise_mismatches"] | r["mismatches"] << 1 | r["nonfinite_mismatches"] << 2)
        assert (mabs[k], mrel[k]) == (r["max_abs"], r["max_rel"])
    mism, A, B = _expected_from_isclose(dtype, a, b, atol, rtol, policy == "equal")
    if policy == "strict":
        mism = mism | np.isnan(B)
    assert np.array_equal((flags >> 1) & 1, mism.astype(np.uint8))
    assert np.array_equal(flags & 1, (a != b).astype(np.uint8))
    fin = np.isfinite(A) & np.isfinite(B) & (a != b)
    with np.errstate(divide="ignore", invalid="ignore"):
        d = np.abs(A - B)
        rel = np.where(B != 0, d / np.abs(B), np.where(d == 0, 0.0, np.inf))
    assert np.array_equal(mabs, np.where(fin, d, 0.0))
    assert np.array_equal(mrel, np.where(fin, rel, 0.0))
