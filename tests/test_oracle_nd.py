"""Pins for the oracle's N-dimensional segments (paper section 3.4: Tier-1
inputs span shapes and strides; Tier-2 captures hold non-contiguous tensors
and block-table layouts).

numpy fixes what an N-D strided view means: each test builds a view with
numpy (transpose, slicing, broadcasting, as_strided), lets numpy gather it
into a contiguous copy, and checks the oracle's N-D compare over the raw
buffers against the plain 1-D compare of the gathered copies and against a
numpy rendering of the tolerance rule.  Brute force over every element of a
small 4-D view pins the logical (row-major) indexing."""
import numpy as np
import pytest

import oracle

INTACT = {"mismatches": 0, "first_mismatch": -1, "bitwise_mismatches": 0, "first_bitwise": -1,
          "nonfinite_mismatches": 0, "max_abs": 0.0, "max_rel": 0.0}


def _nd_of_view(v: np.ndarray, base: np.ndarray):
    """(byte offset of element 0 in base, strides in elements) of a numpy view."""
    es = v.itemsize
    off = v.__array_interface__["data"][0] - base.__array_interface__["data"][0]
    assert off % es == 0 and all(s % es == 0 for s in v.strides)
    return off, [s // es for s in v.strides]


def _check_view(va, vb, base_a, base_b, dtype="f32", mode="tolerance", policy="equal", atol=1e-3, rtol=1e-3):
    oa, sa = _nd_of_view(va, base_a)
    ob, sb = _nd_of_view(vb, base_b)
    got = oracle.diff_segment_nd(dtype, mode, policy, list(va.shape), sa, sb, atol, rtol,
                                 base_a.view(np.uint8), base_b.view(np.uint8), oa, ob)
    ca = np.ascontiguousarray(va).reshape(-1)
    cb = np.ascontiguousarray(vb).reshape(-1)
    flat = oracle.diff_segment(dtype, mode, policy, 1, ca.size, ca.size, ca.size, atol, rtol,
                               ca.view(np.uint8), cb.view(np.uint8))
    assert got == flat
    return got


def _pair(shape, seed, frac=0.01, dtype=np.float32):
    rng = np.random.default_rng(seed)
    b = rng.standard_normal(shape).astype(dtype)
    a = b.copy()
    flat = a.reshape(-1)
    k = max(1, int(frac * flat.size))
    idx = rng.choice(flat.size, size=k, replace=False)
    flat[idx] += rng.choice([-1.0, 1.0], size=k).astype(dtype) * rng.uniform(1e-5, 1e-1, size=k).astype(dtype)
    return a, b


def test_contiguous_nd_equals_flat():
    a, b = _pair((6, 7, 8, 9), 1)
    r = _check_view(a, b, a, b)
    assert r["mismatches"] > 0


@pytest.mark.parametrize("perm", [(1, 0, 2), (2, 1, 0), (0, 2, 1), (2, 0, 1)])
def test_transposed_views(perm):
    a, b = _pair((5, 11, 13), 2)
    _check_view(a.transpose(perm), b.transpose(perm), a, b)


def test_sliced_and_stepped_views():
    a, b = _pair((20, 30, 40), 3)
    r = _check_view(a[2:17:3, ::2, 5:33], b[2:17:3, ::2, 5:33], a, b)
    assert r["bitwise_mismatches"] > 0
    # different views of the two operands (same logical shape, other strides)
    b2 = np.ascontiguousarray(b[2:17:3, ::2, 5:33])
    _check_view(a[2:17:3, ::2, 5:33], b2, a, b2)


def test_broadcast_dimension():
    a, b = _pair((1, 50), 4)
    va = np.broadcast_to(a, (7, 50))
    vb = np.broadcast_to(b, (7, 50))
    r = _check_view(va, vb, a, b)
    single = _check_view(a[0], b[0], a, b)
    assert r["mismatches"] == 7 * single["mismatches"]
    assert r["first_mismatch"] == single["first_mismatch"]


def test_numpy_rule_on_a_permuted_bf16_like_layout():
    """Counts and first index against numpy's isclose on the gathered view."""
    a, b = _pair((8, 16, 12, 6), 5, frac=0.05)
    va, vb = a.transpose(2, 0, 3, 1), b.transpose(2, 0, 3, 1)
    r = _check_view(va, vb, a, b, atol=1e-3, rtol=1e-2)
    ca = np.ascontiguousarray(va).reshape(-1).astype(np.float64)
    cb = np.ascontiguousarray(vb).reshape(-1).astype(np.float64)
    bad = np.flatnonzero(~(np.abs(ca - cb) <= 1e-3 + 1e-2 * np.abs(cb)))
    assert r["mismatches"] == bad.size and r["first_mismatch"] == int(bad[0])
    assert r["max_abs"] == float(np.abs(ca - cb).max())


def test_brute_force_logical_index_of_every_element():
    base = np.arange(3 * 4 * 5 * 6, dtype=np.int32).reshape(3, 4, 5, 6)
    v = base.transpose(3, 1, 0, 2)[::2, 1:, :, ::2]            # shape (3, 3, 3, 3)
    off, st = _nd_of_view(v, base)
    logical = np.ascontiguousarray(v).reshape(-1)
    for i, val in enumerate(logical.tolist()):
        other = base.copy()
        other.reshape(-1)[val] ^= 1                            # the element at view index i
        r = oracle.diff_segment_nd("i32", "bitwise", "equal", list(v.shape), st, st, 0.0, 0.0,
                                   base.view(np.uint8), other.view(np.uint8), off, off, index_base=1000)
        assert r["mismatches"] == 1 and r["first_mismatch"] == 1000 + i


def test_empty_and_scalar_shapes():
    a = np.zeros(16, np.float32)
    b = np.ones(16, np.float32)
    for shape in ([0], [3, 0, 2], [0, 5]):
        r = oracle.diff_segment_nd("f32", "tolerance", "equal", shape, [1] * len(shape), [1] * len(shape),
                                   0.0, 0.0, a.view(np.uint8), b.view(np.uint8))
        assert r == INTACT
    r = oracle.diff_segment_nd("f32", "tolerance", "equal", [], [], [], 0.0, 0.0,
                               a.view(np.uint8), b.view(np.uint8), 8, 8, index_base=42)
    assert r["mismatches"] == 1 and r["first_mismatch"] == 42 and r["max_abs"] == 1.0


def test_block_table_layout_as_segments_sharing_a_result():
    """A paged cache: logical blocks of 16 rows x 64 values live in physical
    blocks picked by a block table.  One segment per logical block, each with
    index_base = its logical start, merged into one result, equals the
    compare of the gathered logical tensors."""
    rng = np.random.default_rng(6)
    n_phys, blk, width = 40, 16, 64
    pool_b = rng.standard_normal((n_phys, blk, width)).astype(np.float32)
    pool_a = pool_b.copy()
    table = rng.permutation(n_phys)[:23]
    for p in table[::3]:
        pool_a[p, rng.integers(0, blk), rng.integers(0, width)] += 1.0
    parts = []
    for j, p in enumerate(table.tolist()):
        off = p * blk * width * 4
        parts.append(oracle.diff_segment_nd("f32", "tolerance", "equal", [blk, width], [width, 1], [width, 1],
                                            1e-4, 1e-4, pool_a.view(np.uint8), pool_b.view(np.uint8),
                                            off, off, index_base=j * blk * width))
    merged = oracle.merge_results(parts)
    la = pool_a[table].reshape(-1)
    lb = pool_b[table].reshape(-1)
    flat = oracle.diff_segment("f32", "tolerance", "equal", 1, la.size, la.size, la.size, 1e-4, 1e-4,
                               la.view(np.uint8), lb.view(np.uint8))
    assert merged == flat
    assert merged["mismatches"] == len(table[::3])
