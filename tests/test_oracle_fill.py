"""Pins for the CPU oracle's guarded fill (paper section 3.4, Tier 1: seeded
deterministic inputs, allocations with canary-initialised guards) and for the
closed-form results of the five workloads at oracle-friendly sizes.

The fill is this library's own definition; what pins it here is statistics
(the normal transform is pinned to extended-precision libm in
test_oracle_primitives), numpy's nextafter / isclose for the perturbations,
and closed forms: counts that follow from how each workload is constructed."""
import math

import numpy as np
import pytest
import torch
from scipy import stats

import oracle
import workloads
from workloads import Alloc, Compare, Injection, Workload

FLOAT = ("f32", "bf16", "f16", "fp8e4m3")
INTACT = {"bad_lo": 0, "bad_hi": 0, "first_bad_lo": -1, "first_bad_hi": -1, "bad_pad": 0,
          "first_bad_pad": -1}


def _values(dtype, raw_bytes):
    """fp64 values of a little-endian byte array via numpy / torch casts."""
    if dtype == "f32":
        return raw_bytes.view(np.float32).astype(np.float64)
    if dtype == "f16":
        return raw_bytes.view(np.float16).astype(np.float64)
    if dtype == "bf16":
        return torch.from_numpy(raw_bytes.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
    if dtype == "fp8e4m3":
        return torch.from_numpy(raw_bytes.copy()).view(torch.float8_e4m3fn).double().numpy()
    if dtype == "i32":
        return raw_bytes.view(np.int32).astype(np.float64)
    if dtype == "i64":
        return raw_bytes.view(np.int64).astype(np.float64)
    raise ValueError(dtype)


def _data(w, arena, k):
    a = w.allocs[k]
    o = w.data_offset(k)
    return arena[o:o + a.data_bytes]


def _logical(w, arena, k):
    """Logical elements (row padding removed) as a byte array."""
    a = w.allocs[k]
    d = _data(w, arena, k)
    es = a.esize
    if a.rows <= 1 or a.stride == a.cols:
        return d[:a.n_elements * es]
    full = np.zeros(a.rows * a.stride * es, dtype=np.uint8)
    full[:d.size] = d
    return full.reshape(a.rows, a.stride * es)[:, :a.cols * es].reshape(-1)


@pytest.mark.parametrize("dtype,sigma", [("f32", 1.0), ("bf16", 8.0), ("f16", 1.0), ("fp8e4m3", 1.0)])
def test_normal_fill_statistics(dtype, sigma):
    n = 200_003
    w = Workload("t", "", 0xBEEF, [Alloc(3, dtype, 1, n, n, 0, 0, "normal", 0.5, sigma,
                                         saturate=dtype == "fp8e4m3")], [], [])
    arena = oracle.Prepared(w).fill_arena(0, threads=8)
    v = _values(dtype, _logical(w, arena, 0))
    z = (v - 0.5) / sigma
    assert np.all(np.isfinite(v))
    tol = 5 / math.sqrt(n)
    assert abs(z.mean()) < tol * (3 if dtype == "fp8e4m3" else 1)
    assert abs(z.var() - 1) < 10 * tol * (3 if dtype == "fp8e4m3" else 1)
    if dtype in ("f32", "f16", "bf16"):
        # quantisation of bf16 (8 bits) is visible to KS at this n; check f32/f16 tightly
        if dtype != "bf16":
            assert stats.kstest(z, "norm").pvalue > 1e-4
        # tails: fraction beyond 3 sigma within 5 sd of its binomial expectation
        p3 = 2 * stats.norm.sf(3)
        cnt = np.sum(np.abs(z) > 3)
        assert abs(cnt - n * p3) < 5 * math.sqrt(n * p3)


def test_uniform_int_fill_range_and_uniformity():
    n = 100_000
    w = Workload("t", "", 77, [Alloc(0, "i32", 1, n, n, 0, 0, "uniform_int", i0=-5, i1=1019),
                               Alloc(1, "i64", 1, n, n, 0, 0, "uniform_int", i0=0, i1=1 << 24)], [], [])
    arena = oracle.Prepared(w).fill_arena(0)
    v = _logical(w, arena, 0).view(np.int32)
    assert v.min() >= -5 and v.max() < 1019
    counts = np.bincount(v + 5, minlength=1024)
    assert stats.chisquare(counts).pvalue > 1e-4
    v64 = _logical(w, arena, 1).view(np.int64)
    assert v64.min() >= 0 and v64.max() < (1 << 24)
    assert stats.chisquare(np.bincount(v64 >> 14, minlength=1024)).pvalue > 1e-4


def test_bits_fill_bytes_uniform():
    n = 1 << 16
    w = Workload("t", "", 5, [Alloc(0, "u8", 1, n, n, 0, 0, "bits")], [], [])
    b = _logical(w, oracle.Prepared(w).fill_arena(0), 0)
    assert stats.chisquare(np.bincount(b, minlength=256)).pvalue > 1e-4


def test_fill_is_deterministic_and_range_consistent():
    a = Alloc(9, "bf16", 7, 33, 40, 24, 40, "normal", 0.0, 2.0)
    w = Workload("t", "", 1234, [a], [Injection(0, "flip_bit", arg=-1, rate=0.1)], [])
    P = oracle.Prepared(w)
    whole = P.fill_range(0, 1, 0, a.total_bytes)
    assert np.array_equal(whole, P.fill_range(0, 1, 0, a.total_bytes))
    for off in (0, 1, 15, 16, 23, 24, 25, 100, a.total_bytes - 17):
        for ln in (1, 7, 16, 33):
            ln = min(ln, a.total_bytes - off)
            assert np.array_equal(P.fill_range(0, 1, off, ln), whole[off:off + ln])
    # another seed changes the data and the guards
    w2 = Workload("t", "", 1235, [a], w.injections, [])
    other = oracle.Prepared(w2).fill_range(0, 1, 0, a.total_bytes)
    assert np.mean(other != whole) > 0.5


def test_values_do_not_depend_on_row_stride():
    base = dict(alloc_id=4, dtype="f16", rows=9, cols=21, guard_lo=16, guard_hi=8, dist="normal")
    w1 = Workload("t", "", 99, [Alloc(stride=21, **base)], [], [])
    w2 = Workload("t", "", 99, [Alloc(stride=29, **base)], [], [])
    l1 = _logical(w1, oracle.Prepared(w1).fill_arena(0), 0)
    l2 = _logical(w2, oracle.Prepared(w2).fill_arena(0), 0)
    assert np.array_equal(l1, l2)


def test_guards_intact_after_fill_and_guard_writes_detected():
    a = Alloc(2, "f32", 1, 100, 100, 64, 72, "normal")
    inj = [Injection(0, "guard_write_lo", arg=3, index=5),
           Injection(0, "guard_write_hi", arg=1, index=71),
           Injection(0, "guard_write_hi", sides="both", arg=2, index=10)]
    w = Workload("t", "", 42, [a], inj, [])
    P = oracle.Prepared(w)
    ref = P.fill_arena(0)
    cand = P.fill_arena(1)
    g_ref = oracle.guard_workload(w, ref)[0]
    g_cand = oracle.guard_workload(w, cand)[0]
    assert g_ref == {"bad_lo": 0, "bad_hi": 2, "first_bad_lo": -1, "first_bad_hi": 10, "bad_pad": 0, "first_bad_pad": -1}
    assert g_cand == {"bad_lo": 3, "bad_hi": 3, "first_bad_lo": 5, "first_bad_hi": 10, "bad_pad": 0, "first_bad_pad": -1}
    # data untouched by guard writes
    assert np.array_equal(_data(w, ref, 0), _data(w, cand, 0))


def test_point_injections_touch_only_their_elements():
    n = 4000
    a = Alloc(0, "f32", 1, n, n, 0, 0, "normal")
    idx = [3, 17, 999, 2500, 3999]
    inj = [Injection(0, "step_within", index=idx[0], atol=1e-5, rtol=1e-5),
           Injection(0, "set_beyond", index=idx[1], atol=1e-5, rtol=1e-5),
           Injection(0, "flip_bit", arg=-1, index=idx[2]),
           Injection(0, "set_nan", index=idx[3]),
           Injection(0, "set_inf", arg=1, index=idx[4])]
    w = Workload("t", "", 11, [a], inj, [])
    P = oracle.Prepared(w)
    r = _logical(w, P.fill_arena(0), 0).view(np.uint32)
    c = _logical(w, P.fill_arena(1), 0).view(np.uint32)
    diff = np.flatnonzero(r != c)
    assert diff.tolist() == idx
    rv, cv = r.view(np.float32), c.view(np.float32)
    # step: the fp32 neighbour of b
    assert cv[idx[0]] in (np.nextafter(rv[idx[0]], np.float32(np.inf)),
                          np.nextafter(rv[idx[0]], np.float32(-np.inf)))
    assert not np.isclose(float(cv[idx[1]]), float(rv[idx[1]]), atol=1e-5, rtol=1e-5)
    assert bin(int(r[idx[2]] ^ c[idx[2]])).count("1") == 1
    assert np.isnan(cv[idx[3]])
    assert cv[idx[4]] == -np.inf


@pytest.mark.parametrize("dtype,atol,rtol", [("f16", 1e-3, 1e-3), ("fp8e4m3", 0.125, 0.125),
                                             ("f32", 1e-5, 1e-5), ("bf16", 1e-2, 1.6e-2)])
def test_step_within_and_set_beyond_classify_as_built(dtype, atol, rtol):
    n = 3000
    a = Alloc(0, dtype, 1, n, n, 0, 0, "normal", saturate=dtype == "fp8e4m3")
    rng = np.random.default_rng(3)
    idx = rng.permutation(n)[:400]
    inj = [Injection(0, "step_within", index=int(i), atol=atol, rtol=rtol) for i in idx[:200]]
    inj += [Injection(0, "set_beyond", index=int(i), atol=atol, rtol=rtol) for i in idx[200:]]
    w = Workload("t", "", 21, [a], inj, [])
    P = oracle.Prepared(w)
    rv = _values(dtype, _logical(w, P.fill_arena(0), 0))
    cv = _values(dtype, _logical(w, P.fill_arena(1), 0))
    close = np.isclose(cv, rv, atol=atol, rtol=rtol)
    assert close[idx[:200]].all()
    assert not close[idx[200:]].any()
    assert np.all(cv[idx[:200]] != rv[idx[:200]]) or dtype == "fp8e4m3"


def test_rate_rule_counts_and_both_sides():
    n = 400_000
    a = Alloc(0, "bf16", 1, n, n, 0, 0, "normal", 0.0, 8.0)
    w = Workload("t", "", 8, [a], [Injection(0, "flip_bit", arg=0, rate=0.01),
                                  Injection(0, "flip_bit", sides="both", arg=5, rate=0.001)], [])
    P = oracle.Prepared(w)
    r = _logical(w, P.fill_arena(0), 0).view(np.uint16)
    c = _logical(w, P.fill_arena(1), 0).view(np.uint16)
    c2 = _logical(w, P.fill_arena(2), 0).view(np.uint16)
    x = r ^ c
    flips = np.flatnonzero(x)
    assert set(np.unique(x[flips]).tolist()) <= {1, 1 | 32, 32}
    # candidate-only rule: ~1% of elements; binomial 5-sigma band
    k = np.count_nonzero(x & 1)
    assert abs(k - 0.01 * n) < 5 * math.sqrt(n * 0.01 * 0.99)
    # the 'both' rule is identical on every side, so it never shows in a diff
    # except where the candidate rule also selects the element (last rule wins)
    assert np.count_nonzero(x == 32) == 0
    # different candidates draw different positions
    assert np.count_nonzero((r ^ c2) & 1) > 0 and not np.array_equal(c, c2)


# ------------------------------------------------------------ closed forms
def _run(w, threads=8):
    P = oracle.Prepared(w)
    ref = P.fill_arena(0, threads)
    cand = P.fill_arena(1, threads)
    return P, ref, cand, oracle.diff_workload(w, cand, ref), oracle.guard_workload(w, cand)


def test_closed_form_single_fp32():
    w = workloads.single_fp32(small=True)
    P, ref, cand, res, guards = _run(w)
    r = res[0]
    within = [j.index for j in w.injections if j.kind == "step_within"]
    beyond = [j.index for j in w.injections if j.kind == "set_beyond"]
    assert r["mismatches"] == 32 and r["first_mismatch"] == min(beyond)
    assert r["bitwise_mismatches"] == 64 and r["first_bitwise"] == min(within + beyond)
    assert r["nonfinite_mismatches"] == 0
    gw = [j for j in w.injections if j.kind.startswith("guard")][0]
    g = guards[0]
    side = "lo" if gw.kind.endswith("lo") else "hi"
    other = "hi" if side == "lo" else "lo"
    assert g[f"bad_{side}"] == 4 and g[f"first_bad_{side}"] == gw.index
    assert g[f"bad_{other}"] == 0 and g[f"first_bad_{other}"] == -1
    # the reference state's guards are intact
    assert oracle.guard_workload(w, ref)[0]["bad_lo"] == 0
    # max_abs dominated by the beyond perturbations: at least 4t - ulp of them
    assert r["max_abs"] > 4 * 1e-5 * 0.9


def test_closed_form_padded_bf16():
    w = workloads.padded_bf16(small=True)
    P, ref, cand, res, _ = _run(w)
    eq, strict = res
    n = w.allocs[0].n_elements
    assert eq["mismatches"] == 55                 # 50 unmatched NaN + 5 unmatched Inf
    assert strict["mismatches"] == 105            # + the 50 matched NaN under the strict policy
    assert eq["nonfinite_mismatches"] == 55 and strict["nonfinite_mismatches"] == 105
    specials = {j.index for j in w.injections if j.rate is None}
    lc = _logical(w, cand, 0).view(np.uint16)
    lr = _logical(w, ref, 0).view(np.uint16)
    x = lc ^ lr
    nonspecial = np.ones(n, bool)
    nonspecial[list(specials)] = False
    F = int(np.count_nonzero(x[nonspecial]))
    assert np.all(x[nonspecial][x[nonspecial] != 0] == 1)      # last-bit flips only
    assert abs(F - 0.01 * (n - 110)) < 5 * math.sqrt(n * 0.01)
    assert eq["bitwise_mismatches"] == F + 55
    # row padding is not part of the data compared, and matched specials agree
    matched = [j.index for j in w.injections if j.sides == "both"]
    assert np.all(lc[matched] == lr[matched])


def test_closed_form_decode_state():
    w = workloads.decode_state(small=True)
    P, ref, cand, res, _ = _run(w)
    for k, r in enumerate(res):
        c = w.compares[k]
        if c.mode == "bitwise":
            assert r["bitwise_mismatches"] == 64 and r["mismatches"] == 64
        else:
            assert r["mismatches"] == 32 and r["bitwise_mismatches"] == 64
            beyond = [j.index for j in w.injections if j.alloc == c.alloc and j.kind == "set_beyond"]
            assert r["first_mismatch"] == min(beyond)
        assert r["nonfinite_mismatches"] == 0


def test_closed_form_int_lowp():
    w = workloads.int_lowp(small=True)
    P, ref, cand, res, _ = _run(w)
    for k, r in enumerate(res):
        assert r["bitwise_mismatches"] == 16
        idx = sorted(j.index for j in w.injections if j.alloc == k)
        assert r["first_bitwise"] == idx[0]
    # fp8: the tolerance verdict of each flipped element, classified by isclose
    a = w.allocs[2]
    lc = _values("fp8e4m3", _logical(w, cand, 2))
    lr = _values("fp8e4m3", _logical(w, ref, 2))
    idx = np.array(sorted(j.index for j in w.injections if j.alloc == 2))
    close = np.isclose(lc[idx], lr[idx], atol=0.125, rtol=0.125, equal_nan=True)
    assert res[2]["mismatches"] == int((~close).sum())


def test_closed_form_sweep_small():
    w = workloads.sweep(small=True)
    P, ref, cand, res, guards = _run(w)
    assert all(g == INTACT for g in guards)
    total_bw = 0
    for k, r in enumerate(res):
        lc = _logical(w, cand, k)
        lr = _logical(w, ref, k)
        es = w.allocs[k].esize
        x = (lc ^ lr).reshape(-1, es)
        diff_el = np.flatnonzero(x.any(axis=1))
        assert r["bitwise_mismatches"] == diff_el.size
        assert r["first_bitwise"] == (int(diff_el[0]) if diff_el.size else -1)
        # single random-bit flips only
        for e in diff_el:
            assert sum(bin(int(v)).count("1") for v in x[e]) == 1
        total_bw += diff_el.size
    n_el = sum(a.n_elements for a in w.allocs)
    assert abs(total_bw - 1e-6 * n_el) < 5 * math.sqrt(n_el * 1e-6) + 3


# ------------------------------------------------------------ row-pad canaries
def _pad_mask(a):
    """Data-region bytes that are row padding: element (q // es) has column >= cols."""
    q = np.arange(a.data_bytes)
    return (q // a.esize) % a.stride >= a.cols


@pytest.mark.parametrize("dtype,rows,cols,stride", [("f32", 5, 7, 10), ("bf16", 4, 13, 16), ("u8", 6, 5, 9),
                                                    ("i64", 3, 2, 5), ("f16", 1, 9, 12), ("fp8e4m3", 4, 8, 8)])
def test_pad_check_flags_exactly_the_pad_bytes(dtype, rows, cols, stride):
    """Brute force: invert each data-region byte in turn; the pad check counts it
    iff numpy's pad mask says it is padding."""
    a = Alloc(6, dtype, rows, cols, stride, 16, 16, "normal" if dtype in FLOAT else "bits")
    w = Workload("t", "", 0x9AD, [a], [], [])
    arena = oracle.Prepared(w).fill_arena(0)
    o = w.data_offset(0)
    data = arena[o:o + a.data_bytes].copy()
    assert oracle.pad_check(w, 0, data) == {"bad_pad": 0, "first_bad_pad": -1}
    mask = _pad_mask(a)
    for q in range(a.data_bytes):
        d2 = data.copy()
        d2[q] ^= 0xFF
        r = oracle.pad_check(w, 0, d2)
        assert r == ({"bad_pad": 1, "first_bad_pad": q} if mask[q] else {"bad_pad": 0, "first_bad_pad": -1})
    # a different seed's pads do not pass
    w2 = Workload("t", "", 0x9AE, [a], [], [])
    if mask.sum() >= 8:
        assert oracle.pad_check(w2, 0, data)["bad_pad"] >= mask.sum() // 2


def test_pad_write_injection():
    a = Alloc(8, "bf16", 9, 30, 37, 32, 32, "normal", 0.0, 4.0)
    es = a.esize
    pitch = a.stride * es
    # row 2: bytes 3..8 of its padding; row 7: the last pad byte of the row
    inj = [Injection(0, "pad_write", arg=6, index=2 * pitch + a.cols * es + 3),
           Injection(0, "pad_write", sides="both", arg=1, index=7 * pitch + pitch - 1)]
    w = Workload("t", "", 0x51, [a], inj, [])
    P = oracle.Prepared(w)
    ref, cand = P.fill_arena(0), P.fill_arena(1)
    g_ref = oracle.guard_workload(w, ref)[0]
    g_cand = oracle.guard_workload(w, cand)[0]
    assert g_ref["bad_pad"] == 1 and g_ref["first_bad_pad"] == 7 * pitch + pitch - 1
    assert g_cand["bad_pad"] == 7 and g_cand["first_bad_pad"] == 2 * pitch + a.cols * es + 3
    assert g_cand["bad_lo"] == 0 and g_cand["bad_hi"] == 0
    # the written bytes are the complement of the reference's pad bytes; elements untouched
    o = w.data_offset(0)
    x = ref[o:o + a.data_bytes] ^ cand[o:o + a.data_bytes]
    assert np.flatnonzero(x).tolist() == list(range(2 * pitch + a.cols * es + 3, 2 * pitch + a.cols * es + 9))
    assert set(x[x != 0].tolist()) == {0xFF}
    assert np.array_equal(_logical(w, ref, 0), _logical(w, cand, 0))
