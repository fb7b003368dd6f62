"""Pins for the oracle's cosine term c = cos(K'(x), O(x)) of Eq. 1, and for
the test-side model of the library's documented summation order.

The oracle computes each of the sums a*b, a*a, b*b exactly (a fixed-point
accumulator) and rounds it once.  What pins it: exact rational arithmetic
(Python's Fraction, whose conversion to float rounds correctly) on values of
extreme range, with cancellation, subnormals and ties; math.fsum, which also
returns the correctly rounded sum, on large inputs; exact integer sums; the
independence of the result from the order in which elements are visited
(strided, transposed, broadcast and shared-result views against gathered
copies); closed-form special cases.

The order model (tests/cosine_order.py) is pinned by hand-computed cases in
which its association differs from a sequential sum, by numpy level-by-level
pairing for its tree, and by the error bound of its order against the exact
oracle."""
import math
import struct
from fractions import Fraction

import numpy as np
import pytest

import cosine_order
import oracle

U = 2.0 ** -53


def gamma(k: int) -> float:
    """gamma_k = k u / (1 - k u): the bound on the relative error of k roundings."""
    return k * U / (1.0 - k * U)


def _cos(dtype, a, b, rows=None, cols=None, sa=None, sb=None):
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    n = a.size
    if rows is None:
        rows, cols, sa, sb = 1, n, n, n
    return oracle.cosine_segment(dtype, rows, cols, sa, sb, a.view(np.uint8), b.view(np.uint8))


def _bits(v: float) -> int:
    return struct.unpack("<Q", struct.pack("<d", v))[0]


def _exact(values) -> float:
    return float(sum((Fraction(v) for v in values), Fraction(0)))


# ---------------------------------------------------------------- exact sums
def test_exact_sum_against_fractions():
    rng = np.random.default_rng(11)
    for trial in range(300):
        n = int(rng.integers(1, 60))
        mant = rng.standard_normal(n)
        exps = rng.integers(-1100, 1000, size=n) if trial % 3 == 0 else rng.integers(-60, 60, size=n)
        x = np.ldexp(mant, exps)
        if trial % 4 == 1:                       # cancellation: add the negatives of some terms
            k = rng.integers(0, n, size=n // 2 + 1)
            x = np.concatenate([x, -x[k], rng.standard_normal(3) * 2.0 ** -1070])
        x = x[np.isfinite(x)]
        rng.shuffle(x)
        assert _bits(oracle.exact_sum(x)) == _bits(_exact(x.tolist())), x


def test_exact_sum_ties_and_edges():
    p53 = 2.0 ** 53
    cases = [
        ([p53, 1.0], p53),                       # halfway: to the even neighbour below
        ([p53, 3.0], p53 + 4),                   # halfway: to the even neighbour above
        ([p53, 1.0, 2.0 ** -1000], p53 + 2),     # just above halfway
        ([-p53, -1.0], -p53),
        ([-p53, -1.0, -(2.0 ** -1074)], -p53 - 2),
        ([2.0 ** -1074, 2.0 ** -1074], 2.0 ** -1073),
        ([2.0 ** -1022, -(2.0 ** -1074)], 2.0 ** -1022 - 2.0 ** -1074),   # a subnormal result
        ([1e300, 1.0, -1e300], 1.0),
        ([1.0, 1e-300, -1.0], 1e-300),
        ([], 0.0),
        ([0.0, -0.0], 0.0),
    ]
    for x, want in cases:
        got = oracle.exact_sum(np.array(x, dtype=np.float64))
        assert _bits(got) == _bits(want), (x, got, want)
    assert _bits(oracle.exact_sum(np.array([2.0 ** -1074, -(2.0 ** -1074)]))) == _bits(0.0)   # +0, not -0
    big = np.finfo(np.float64).max
    assert oracle.exact_sum(np.array([big, big])) == math.inf
    assert oracle.exact_sum(np.array([big, -big, big])) == big


def test_exact_sum_against_fsum_large():
    rng = np.random.default_rng(12)
    for scale in (1.0, 1e-200, 1e200):
        x = rng.standard_normal(400_000) * scale * 10.0 ** rng.integers(-12, 12, size=400_000)
        assert _bits(oracle.exact_sum(x)) == _bits(math.fsum(x.tolist()))


# ---------------------------------------------------------------- cosine sums
def _decoded(dtype, n, rng, scale=1.0, noise=0.05):
    """Raw element arrays of one dtype and their exact float64 values (torch / numpy casts)."""
    import torch
    x = rng.standard_normal(n) * scale
    y = x + rng.standard_normal(n) * noise * scale
    if dtype == "f32":
        a, b = x.astype(np.float32), y.astype(np.float32)
        return a, b, a.astype(np.float64), b.astype(np.float64)
    if dtype == "f16":
        a, b = x.astype(np.float16), y.astype(np.float16)
        return a, b, a.astype(np.float64), b.astype(np.float64)
    if dtype == "bf16":
        a = torch.from_numpy(x).to(torch.bfloat16)
        b = torch.from_numpy(y).to(torch.bfloat16)
        return (a.view(torch.int16).numpy().copy(), b.view(torch.int16).numpy().copy(),
                a.double().numpy(), b.double().numpy())
    a = torch.from_numpy(np.clip(x, -448, 448)).to(torch.float8_e4m3fn)
    b = torch.from_numpy(np.clip(y, -448, 448)).to(torch.float8_e4m3fn)
    return (a.view(torch.uint8).numpy().copy(), b.view(torch.uint8).numpy().copy(),
            a.double().numpy(), b.double().numpy())


@pytest.mark.parametrize("dtype,scale", [("f32", 1.0), ("f32", 1e30), ("f16", 100.0), ("bf16", 8.0),
                                         ("fp8e4m3", 1.0), ("fp8e4m3", 200.0)])
def test_sums_are_the_correctly_rounded_exact_sums(dtype, scale):
    """Every product of two values of these types is exact in float64, so the
    exact sums are math.fsum of the float64 products, rounded once."""
    rng = np.random.default_rng(4)
    a, b, A, B = _decoded(dtype, 200_003, rng, scale)
    ok = np.isfinite(A) & np.isfinite(B)
    A, B = A[ok], B[ok]
    r = _cos(dtype, a, b)
    assert r["pairs"] == int(ok.sum())
    for key, terms in (("sum_ab", A * B), ("sum_aa", A * A), ("sum_bb", B * B), ("sum_abs_ab", np.abs(A * B))):
        assert _bits(r[key]) == _bits(math.fsum(terms.tolist())), key
    want = r["sum_ab"] / (math.sqrt(r["sum_aa"]) * math.sqrt(r["sum_bb"]))
    assert _bits(r["cosine"]) == _bits(want)


def test_sums_of_extreme_products_against_fractions():
    """fp32 values from the smallest subnormal to the largest finite: products
    from 2^-298 to 2^256, summed exactly."""
    rng = np.random.default_rng(13)
    bits = rng.integers(0, 1 << 32, size=4000, dtype=np.uint64).astype(np.uint32)
    bits[::7] &= 0x807FFFFF                      # many subnormals
    a = bits[:2000].view(np.float32).copy()
    b = bits[2000:].view(np.float32).copy()
    ok = np.isfinite(a) & np.isfinite(b)
    r = _cos("f32", a, b)
    A = [Fraction(float(v)) for v in a[ok]]
    B = [Fraction(float(v)) for v in b[ok]]
    assert r["pairs"] == int(ok.sum())
    assert _bits(r["sum_ab"]) == _bits(float(sum((x * y for x, y in zip(A, B)), Fraction(0))))
    assert _bits(r["sum_aa"]) == _bits(float(sum((x * x for x in A), Fraction(0))))
    assert _bits(r["sum_bb"]) == _bits(float(sum((y * y for y in B), Fraction(0))))


def test_exactly_representable_sums():
    rng = np.random.default_rng(3)
    for dtype, np_t in (("f32", np.float32), ("f16", np.float16)):
        n = 30_011
        a = rng.integers(-8, 9, size=n).astype(np_t)
        b = rng.integers(-8, 9, size=n).astype(np_t)
        r = _cos(dtype, a, b)
        ai, bi = a.astype(np.int64), b.astype(np.int64)
        assert r["sum_ab"] == float((ai * bi).sum())
        assert r["sum_aa"] == float((ai * ai).sum())
        assert r["sum_bb"] == float((bi * bi).sum())
        assert r["pairs"] == n
        assert r["cosine"] == r["sum_ab"] / (math.sqrt(r["sum_aa"]) * math.sqrt(r["sum_bb"]))


def test_order_does_not_matter():
    """The same elements visited in another order (a shuffled copy, row by row
    through a padded 2-D segment) give bit-identical results."""
    rng = np.random.default_rng(5)
    rows, cols, stride = 37, 3000, 3100
    full = (rng.standard_normal(rows * stride) * 10.0 ** rng.integers(-5, 5, rows * stride)).astype(np.float32)
    other = (full + rng.standard_normal(rows * stride).astype(np.float32) * 1e-3).astype(np.float32)
    r2d = _cos("f32", full, other, rows, cols, stride, stride)
    la = full.reshape(rows, stride)[:, :cols].ravel().copy()
    lb = other.reshape(rows, stride)[:, :cols].ravel().copy()
    perm = rng.permutation(la.size)
    for x, y in ((la, lb), (la[perm].copy(), lb[perm].copy()), (la[::-1].copy(), lb[::-1].copy())):
        assert _cos("f32", x, y) == r2d


def test_special_cases():
    rng = np.random.default_rng(6)
    a = rng.standard_normal(50_000).astype(np.float32)
    r = _cos("f32", a, a)
    assert r["sum_ab"] == r["sum_aa"] == r["sum_bb"] and abs(r["cosine"] - 1.0) <= 2 * U
    r = _cos("f32", a, -a)
    assert abs(r["cosine"] + 1.0) <= 2 * U
    z = np.zeros(1000, np.float32)
    assert _cos("f32", z, z)["cosine"] == 1.0
    assert _cos("f32", a[:1000], z)["cosine"] == 0.0
    assert _cos("f32", z, a[:1000])["cosine"] == 0.0
    o1 = np.array([1, 0, 2, 0] * 256, np.float32)     # orthogonal by construction
    o2 = np.array([0, 3, 0, -1] * 256, np.float32)
    assert _cos("f32", o1, o2)["cosine"] == 0.0
    ri = _cos("i32", np.arange(10, dtype=np.int32), np.arange(10, dtype=np.int32))
    assert math.isnan(ri["cosine"]) and ri["pairs"] == 0 and ri["sum_ab"] == 0.0
    re = oracle.cosine_segment("f32", 0, 5, 5, 5, z.view(np.uint8), z.view(np.uint8))
    assert re["pairs"] == 0 and re["cosine"] == 1.0


def test_nonfinite_pairs_are_excluded():
    rng = np.random.default_rng(7)
    a = rng.standard_normal(9000).astype(np.float32)
    b = (a + rng.standard_normal(9000).astype(np.float32) * 0.1).astype(np.float32)
    a2, b2 = a.copy(), b.copy()
    idx = [3, 100, 4095, 8999]
    a2[idx[0]] = np.nan
    b2[idx[1]] = np.inf
    a2[idx[2]] = -np.inf
    b2[idx[3]] = np.nan
    r = _cos("f32", a2, b2)
    keep = np.setdiff1d(np.arange(9000), idx)
    r0 = _cos("f32", a[keep].copy(), b[keep].copy())
    assert r["pairs"] == 9000 - 4
    assert r == r0


@pytest.mark.parametrize("dtype,np_t", [("f32", np.float32), ("f16", np.float16)])
def test_nd_views_equal_their_gathered_copies(dtype, np_t):
    """Transposed, stepped, broadcast and unit-dimension views: the N-D cosine
    equals the cosine of numpy's gathered copy of the same view."""
    rng = np.random.default_rng(8)
    base_a = rng.standard_normal((6, 10, 34, 50)).astype(np_t)
    base_b = (base_a + rng.standard_normal(base_a.shape).astype(np_t) * np_t(0.01)).astype(np_t)
    es = base_a.itemsize
    views = [lambda t: t, lambda t: t.transpose(2, 0, 3, 1), lambda t: t[:, ::3, 5:30:2, ::-1][..., ::-1],
             lambda t: t[1:4, None, :, 7], lambda t: np.broadcast_to(t[0, 0, 0], (9, 50))]
    for f in views:
        va, vb = f(base_a), f(base_b)
        off_a = (va.__array_interface__["data"][0] - base_a.ctypes.data) if va.size else 0
        off_b = (vb.__array_interface__["data"][0] - base_b.ctypes.data) if vb.size else 0
        if any(s < 0 for s in va.strides):
            continue
        part = (list(va.shape), [s // es for s in va.strides], [s // es for s in vb.strides], off_a, off_b)
        got = oracle.cosine_nd(dtype, [part], base_a.view(np.uint8).ravel(), base_b.view(np.uint8).ravel())
        want = _cos(dtype, np.ascontiguousarray(va).ravel(), np.ascontiguousarray(vb).ravel())
        assert got == want, f


def test_nd_segments_sharing_a_result_are_one_vector():
    rng = np.random.default_rng(9)
    n_seg, blk = 5, 300
    a = rng.standard_normal(n_seg * blk).astype(np.float32)
    b = rng.standard_normal(n_seg * blk).astype(np.float32)
    parts = [([blk], [1], [1], 4 * blk * k, 4 * blk * k) for k in range(n_seg)]
    whole = oracle.cosine_nd("f32", parts[::-1], a.view(np.uint8), b.view(np.uint8))
    assert whole == _cos("f32", a, b)
    e = oracle.cosine_nd("f32", [], a.view(np.uint8), a.view(np.uint8))
    assert e["cosine"] == 1.0 and e["pairs"] == 0


# ---------------------------------------------------------------- the order model
def test_model_tree_power_of_two_equals_level_pairing():
    rng = np.random.default_rng(1)
    for k in range(0, 13):
        x = rng.standard_normal(1 << k) * 10.0 ** rng.integers(-8, 8, size=1 << k)
        y = x.copy()
        while y.size > 1:
            y = y[0::2] + y[1::2]
        assert cosine_order.pairwise_tree(x) == y[0]


def test_model_tree_general_n_recursion():
    rng = np.random.default_rng(2)

    def rec(x):                                   # the definition, written recursively
        if len(x) == 1:
            return x[0]
        h = 1
        while 2 * h < len(x):
            h *= 2
        return rec(x[:h]) + rec(x[h:])

    for n in list(range(1, 70)) + [255, 256, 257, 1000, 4097]:
        x = (rng.standard_normal(n) * 10.0 ** rng.integers(-6, 6, size=n)).tolist()
        assert cosine_order.pairwise_tree(x) == rec(x), n


def _model(dtype, a, b):
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    return cosine_order.cosine_2d(dtype, 1, a.size, a.size, b.size, a.view(np.uint8), b.view(np.uint8))


def test_model_butterfly_order_hand_computed():
    """In one block, a*b = 2^54 on lane 0 and 2 on lanes 1 and 3: the butterfly
    adds lanes 1 and 3 first (4), and 2^54 + 4 is exact, where a sequential
    sum rounds 2^54 + 2 back to 2^54 twice."""
    a = np.zeros(1024, np.float32)
    b = np.zeros(1024, np.float32)
    a[0], b[0] = 2.0 ** 27, 2.0 ** 27          # chunk 0 -> lane 0
    a[4], b[4] = 1.0, 2.0                      # chunk 1 -> lane 1
    a[12], b[12] = 1.0, 2.0                    # chunk 3 -> lane 3
    assert _model("f32", a, b)["sum_ab"] == 2.0 ** 54 + 4
    assert _cos("f32", a, b)["sum_ab"] == 2.0 ** 54 + 4      # exact, and exactly representable


def test_model_block_tree_order_hand_computed():
    """Three 4096-byte blocks whose sums are 2^54, 2, 2: the left-complete
    tree adds (2^54 + 2) + 2 = 2^54 (each step a tie to even); the exact sum
    2^54 + 4 is representable."""
    a = np.zeros(3 * 1024, np.float32)
    b = np.zeros(3 * 1024, np.float32)
    a[0], b[0] = 2.0 ** 27, 2.0 ** 27
    a[1024], b[1024] = 1.0, 2.0
    a[2048], b[2048] = 1.0, 2.0
    m = _model("f32", a, b)
    assert m["blocks"] == 3 and m["sum_ab"] == 2.0 ** 54
    assert _cos("f32", a, b)["sum_ab"] == 2.0 ** 54 + 4


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16", "fp8e4m3"])
def test_model_within_its_error_bound_of_the_exact_sums(dtype):
    """Each term passes through at most D = lane terms + 6 butterfly steps +
    the tree's depth roundings, so |model - exact| <= gamma_D * sum |t|."""
    rng = np.random.default_rng(14)
    a, b, _, _ = _decoded(dtype, 300_001, rng, 4.0, 0.5)
    m = _model(dtype, a, b)
    r = _cos(dtype, a, b)
    depth = cosine_order.lane_terms(dtype) + 6 + max(1, m["blocks"] - 1).bit_length()
    g = gamma(depth + 1)
    assert m["pairs"] == r["pairs"]
    assert abs(m["sum_ab"] - r["sum_ab"]) <= g * r["sum_abs_ab"]
    assert abs(m["sum_aa"] - r["sum_aa"]) <= g * r["sum_aa"]
    assert abs(m["sum_bb"] - r["sum_bb"]) <= g * r["sum_bb"]
    assert abs(m["cosine"] - r["cosine"]) <= 2.5 * g + 16 * U


def test_model_contiguous_rule_and_walk():
    """A padded 2-D segment is one row per row (blocks per row); a contiguous
    one is a single row; a transposed view walks memory order and merges
    into one row; a broadcast operand keeps its rows apart."""
    rng = np.random.default_rng(15)
    rows, cols, pitch = 30, 600, 700
    a = rng.standard_normal(rows * pitch).astype(np.float32)
    b = rng.standard_normal(rows * pitch).astype(np.float32)
    m = cosine_order.cosine_2d("f32", rows, cols, pitch, pitch, a.view(np.uint8), b.view(np.uint8))
    assert m["blocks"] == rows
    m1 = cosine_order.cosine_2d("f32", rows, pitch, pitch, pitch, a.view(np.uint8), b.view(np.uint8))
    assert m1["blocks"] == -(-rows * pitch * 4 // 4096)
    nd = cosine_order.cosine_nd("f32", [([rows, cols], [pitch, 1], [pitch, 1], 0, 0)], a.view(np.uint8),
                                b.view(np.uint8))
    assert nd == m
    R, C = 96, 80
    t = cosine_order.cosine_nd("f32", [([R, C], [1, R], [1, R], 0, 0)], a.view(np.uint8), b.view(np.uint8))
    assert t["blocks"] == -(-(R * C) // 1024)
    assert cosine_order.walk([R, C], [1, R], [1, R]) == [(R * C, 1, 1)]
    assert cosine_order.walk([64, 128], [128, 1], [0, 1]) == [(64, 128, 0), (128, 1, 1)]
    bc = cosine_order.cosine_nd("f32", [([64, 128], [128, 1], [0, 1], 0, 0)], a.view(np.uint8), b.view(np.uint8))
    assert bc["blocks"] == 64
