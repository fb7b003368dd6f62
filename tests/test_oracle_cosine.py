"""Pins for the oracle's cosine term c = cos(K'(x), O(x)) of Eq. 1.

The fp64 sums follow a defined order (4096-byte blocks, 64 lanes by chunk,
xor butterfly, left-complete pairwise tree over blocks).  What pins it:
exactly representable cases (small integers) against exact integer sums;
hand-computed cases where this association gives a different result than a
sequential sum; the perfect pairwise tree against numpy's level-by-level
pairing; and the error bound of the result against math.fsum.  The N-D
form (segments walked in memory order, several sharing a result) is pinned by
its reduction to the pinned 1-row and 2-D forms on contiguous and padded
views, by exact integer sums and block counts that follow from the walk on
transposed and broadcast views, and by the pinned tree over segments."""
import math

import numpy as np
import pytest

import oracle

LANE_BOUND = 64 + 6 + 40    # additions on one element's path: lane run, butterfly, tree depth


def _cos(dtype, a, b, rows=None, cols=None, sa=None, sb=None):
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    n = a.size
    if rows is None:
        rows, cols, sa, sb = 1, n, n, n
    return oracle.cosine_segment(dtype, rows, cols, sa, sb, a.view(np.uint8), b.view(np.uint8))


def test_pairwise_tree_power_of_two_equals_level_pairing():
    rng = np.random.default_rng(1)
    for k in range(0, 13):
        x = rng.standard_normal(1 << k) * 10.0 ** rng.integers(-8, 8, size=1 << k)
        y = x.copy()
        while y.size > 1:
            y = y[0::2] + y[1::2]               # numpy: elementwise, one rounding each
        assert oracle.pairwise_tree(x) == y[0]


def test_pairwise_tree_general_n_is_fold_of_binary_digits():
    rng = np.random.default_rng(2)
    for n in list(range(1, 70)) + [255, 256, 257, 1000, 4097]:
        x = rng.standard_normal(n) * 10.0 ** rng.integers(-6, 6, size=n)
        # perfect trees over the binary digits of n, left to right, folded from the right
        parts, start = [], 0
        for bit in reversed(range(n.bit_length())):
            if n >> bit & 1:
                y = x[start:start + (1 << bit)].copy()
                while y.size > 1:
                    y = y[0::2] + y[1::2]
                parts.append(y[0])
                start += 1 << bit
        acc = parts[-1]
        for p in reversed(parts[:-1]):
            acc = p + acc
        assert oracle.pairwise_tree(x) == acc, n


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
        assert r["pairs"] == n and r["blocks"] == -(-n * a.itemsize // 4096)
        assert r["cosine"] == r["sum_ab"] / (math.sqrt(r["sum_aa"]) * math.sqrt(r["sum_bb"]))


def test_butterfly_order_hand_computed():
    """Within one block: a*b = 2^54 on lane 0 and 2 on lanes 1 and 3.  The
    butterfly adds lanes 1 and 3 first (4) and then 2^54 + 4 is exact; a
    sequential sum would round 2^54 + 2 back to 2^54 twice."""
    a = np.zeros(1024, np.float32)
    b = np.zeros(1024, np.float32)
    a[0], b[0] = 2.0 ** 27, 2.0 ** 27          # chunk 0 -> lane 0
    a[4], b[4] = 1.0, 2.0                      # chunk 1 -> lane 1
    a[12], b[12] = 1.0, 2.0                    # chunk 3 -> lane 3
    r = _cos("f32", a, b)
    assert r["sum_ab"] == 2.0 ** 54 + 4
    seq = 0.0
    for x, y in zip(a.astype(np.float64), b.astype(np.float64)):
        seq = seq + x * y
    assert seq == 2.0 ** 54                     # the order matters here


def test_block_tree_order_hand_computed():
    """Three 4096-byte blocks whose sums are 2^54, 2, 2: the left-complete
    tree adds (2^54 + 2) + 2 = 2^54; the other association would give 2^54 + 4."""
    a = np.zeros(3 * 1024, np.float32)
    b = np.zeros(3 * 1024, np.float32)
    a[0], b[0] = 2.0 ** 27, 2.0 ** 27
    a[1024], b[1024] = 1.0, 2.0
    a[2048], b[2048] = 1.0, 2.0
    r = _cos("f32", a, b)
    assert r["blocks"] == 3
    assert r["sum_ab"] == 2.0 ** 54


@pytest.mark.parametrize("dtype,np_t,scale", [("f32", np.float32, 1.0), ("f16", np.float16, 1.0),
                                              ("bf16", None, 8.0), ("fp8e4m3", None, 1.0)])
def test_sums_within_error_bound_of_exact(dtype, np_t, scale):
    import torch
    rng = np.random.default_rng(4)
    n = 200_003
    x = rng.standard_normal(n) * scale
    y = x + rng.standard_normal(n) * 0.05 * scale
    if dtype == "bf16":
        a = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy()
        b = torch.from_numpy(y).to(torch.bfloat16).view(torch.int16).numpy()
        A = torch.from_numpy(a.copy()).view(torch.bfloat16).double().numpy()
        B = torch.from_numpy(b.copy()).view(torch.bfloat16).double().numpy()
    elif dtype == "fp8e4m3":
        a = torch.from_numpy(np.clip(x, -448, 448)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        b = torch.from_numpy(np.clip(y, -448, 448)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        A = torch.from_numpy(a.copy()).view(torch.float8_e4m3fn).double().numpy()
        B = torch.from_numpy(b.copy()).view(torch.float8_e4m3fn).double().numpy()
    else:
        a, b = x.astype(np_t), y.astype(np_t)
        A, B = a.astype(np.float64), b.astype(np.float64)
    r = _cos(dtype, a, b)
    u = 2.0 ** -53
    for key, terms in (("sum_ab", A * B), ("sum_aa", A * A), ("sum_bb", B * B)):
        exact = math.fsum(terms.tolist())
        assert abs(r[key] - exact) <= LANE_BOUND * u * float(np.abs(terms).sum()), key
    c_exact = math.fsum((A * B).tolist()) / math.sqrt(math.fsum((A * A).tolist()) * math.fsum((B * B).tolist()))
    assert abs(r["cosine"] - c_exact) <= 1e-12


def test_strided_rows_and_contiguous_rule():
    rng = np.random.default_rng(5)
    rows, cols, stride = 37, 3000, 3100
    full = rng.standard_normal(rows * stride).astype(np.float32)
    other = full + rng.standard_normal(rows * stride).astype(np.float32) * 1e-3
    r2d = _cos("f32", full, other, rows, cols, stride, stride)
    # the logical elements only (pads never read): compare with a gathered contiguous copy
    la = full.reshape(rows, stride)[:, :cols]
    lb = other.reshape(rows, stride)[:, :cols]
    exact = math.fsum((la.astype(np.float64) * lb.astype(np.float64)).ravel().tolist())
    assert abs(r2d["sum_ab"] - exact) <= 1e-10 * abs(exact)
    assert r2d["blocks"] == rows * -(-cols * 4 // 4096)
    # a segment whose rows are contiguous is one row: same sums as the 1-D view
    r_c = _cos("f32", la.copy(), lb.copy(), rows, cols, cols, cols)
    r_1 = _cos("f32", la.ravel().copy(), lb.ravel().copy())
    assert r_c == r_1


def test_special_cases():
    rng = np.random.default_rng(6)
    a = rng.standard_normal(50_000).astype(np.float32)
    r = _cos("f32", a, a)
    assert abs(r["cosine"] - 1.0) <= 4e-16
    r = _cos("f32", a, -a)
    assert abs(r["cosine"] + 1.0) <= 4e-16
    z = np.zeros(1000, np.float32)
    assert _cos("f32", z, z)["cosine"] == 1.0
    assert _cos("f32", a[:1000], z)["cosine"] == 0.0
    assert _cos("f32", z, a[:1000])["cosine"] == 0.0
    # orthogonal by construction
    o1 = np.array([1, 0, 2, 0] * 256, np.float32)
    o2 = np.array([0, 3, 0, -1] * 256, np.float32)
    assert _cos("f32", o1, o2)["cosine"] == 0.0
    # integer buffers: not defined
    ri = _cos("i32", np.arange(10, dtype=np.int32), np.arange(10, dtype=np.int32))
    assert math.isnan(ri["cosine"]) and ri["pairs"] == 0 and ri["sum_ab"] == 0.0
    # empty segment
    re = oracle.cosine_segment("f32", 0, 5, 5, 5, z.view(np.uint8), z.view(np.uint8))
    assert re["blocks"] == 0 and re["cosine"] == 1.0


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
    a3, b3 = a.copy(), b.copy()
    a3[idx] = 0.0
    b3[idx] = 0.0
    r0 = _cos("f32", a3, b3)
    assert r["pairs"] == 9000 - 4
    for k in ("sum_ab", "sum_aa", "sum_bb", "cosine"):
        assert r[k] == r0[k]


# ---------------------------------------------------------------- N-D segments
def _bits(x):
    import struct
    return {k: (struct.unpack("<Q", struct.pack("<d", v))[0] if isinstance(v, float) else v) for k, v in x.items()}


@pytest.mark.parametrize("dtype,np_t", [("f32", np.float32), ("f16", np.float16)])
def test_nd_contiguous_views_reduce_to_one_row(dtype, np_t):
    """A contiguous tensor of any shape (unit dimensions included) walks as one
    row: the N-D cosine equals the 1-row cosine of the flat buffer, bit for
    bit; a padded 2-D view equals the 2-D cosine with the same pitch."""
    rng = np.random.default_rng(7)
    a = rng.standard_normal(6 * 1 * 5 * 700).astype(np_t)
    b = (a + rng.standard_normal(a.size).astype(np_t) * np_t(0.01)).astype(np_t)
    flat = _cos(dtype, a, b)
    nd = oracle.cosine_nd(dtype, [([6, 1, 5, 700], [3500, 3500, 700, 1], [3500, 3500, 700, 1], 0, 0)],
                          a.view(np.uint8), b.view(np.uint8))
    assert _bits(nd) == _bits(flat)
    rows, cols, pitch = 30, 600, 700
    two_d = _cos(dtype, a, b, rows, cols, pitch, pitch)
    nd2 = oracle.cosine_nd(dtype, [([rows, cols], [pitch, 1], [pitch, 1], 0, 0)], a.view(np.uint8),
                           b.view(np.uint8))
    assert _bits(nd2) == _bits(two_d)
    assert nd2["blocks"] == rows                      # 600 elements per row: one block each


def test_nd_walk_order_blocks_and_exact_sums():
    """Views whose walk differs from the logical order: a transposed matrix
    walks memory order and merges into one row; a broadcast operand keeps
    rows apart.  With small integers every sum is exact, so the sums equal the
    integer dot products, and the block counts follow from the walk."""
    rng = np.random.default_rng(8)
    R, C = 96, 80                                     # a is stored [C, R]; the view is [R, C] (transposed)
    ai = rng.integers(-8, 9, size=(C, R))
    bi = rng.integers(-8, 9, size=(C, R))
    a = ai.astype(np.float32)
    b = bi.astype(np.float32)
    t = oracle.cosine_nd("f32", [([R, C], [1, R], [1, R], 0, 0)], a.view(np.uint8), b.view(np.uint8))
    assert t["sum_ab"] == float((ai * bi).sum()) and t["sum_aa"] == float((ai * ai).sum())
    assert t["sum_bb"] == float((bi * bi).sum())
    assert t["blocks"] == -(-(R * C) // 1024) and t["pairs"] == R * C
    # b broadcast along rows: 64 rows of 128 elements, one block each
    rows, cols = 64, 128
    ai = rng.integers(-8, 9, size=(rows, cols))
    bi = rng.integers(-8, 9, size=cols)
    a = ai.astype(np.float32)
    b = bi.astype(np.float32)
    r = oracle.cosine_nd("f32", [([rows, cols], [cols, 1], [0, 1], 0, 0)], a.view(np.uint8), b.view(np.uint8))
    assert r["blocks"] == rows and r["pairs"] == rows * cols
    assert r["sum_ab"] == float((ai * bi[None, :]).sum()) and r["sum_bb"] == float(rows * (bi * bi).sum())


def test_nd_segments_sharing_a_result_concatenate_blocks():
    """Several segments of one result: their blocks, in segment order, form
    one tree.  With one block per segment, the result's sums are the pairwise
    tree of the per-segment sums (checked against the tree routine, itself
    pinned above), and exact integer data gives exact totals."""
    rng = np.random.default_rng(9)
    n_seg, blk = 5, 256                               # 256 fp32 elements: one block per segment
    a = rng.standard_normal(n_seg * blk).astype(np.float32)
    b = rng.standard_normal(n_seg * blk).astype(np.float32)
    parts = [([blk], [1], [1], 4 * blk * k, 4 * blk * k) for k in range(n_seg)]
    whole = oracle.cosine_nd("f32", parts, a.view(np.uint8), b.view(np.uint8))
    singles = [oracle.cosine_nd("f32", [p], a.view(np.uint8), b.view(np.uint8)) for p in parts]
    assert whole["blocks"] == n_seg and whole["pairs"] == n_seg * blk
    for f in ("sum_ab", "sum_aa", "sum_bb"):
        assert whole[f] == oracle.pairwise_tree(np.array([s[f] for s in singles]))
    ai = rng.integers(-8, 9, size=n_seg * blk)
    a = ai.astype(np.float32)
    e = oracle.cosine_nd("f32", parts[::-1], a.view(np.uint8), a.view(np.uint8))
    assert e["sum_ab"] == float((ai * ai).sum()) and abs(e["cosine"] - 1.0) <= 2.0 ** -52
    assert oracle.cosine_nd("f32", [], a.view(np.uint8), a.view(np.uint8))["blocks"] == 0
