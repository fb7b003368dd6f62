"""The library's documented order of the cosine sums, as a test-side model.

The cosine term of Eq. 1 (paper section 3.2) fixes no summation order.  The
oracle therefore computes exact sums (oracle.cosine_segment), and the GPU
pass is checked against them within the error bound of its order.  The
library additionally promises an order of its own (include/asmevo.h, at
asmevo_cosine_result), which makes its results reproducible bit for bit
whatever the launch geometry.  This module writes that documented order out
in numpy so that the tests can check the promise; it is not the oracle and
proves nothing about correctness:

  - rows: a segment whose operands are both contiguous is one row; otherwise
    every row is separate (N-D: the walk order below);
  - each row is cut into blocks of 4096 bytes, the last one shorter;
  - in a block, element t belongs to lane (t div (16 / esize)) mod 64, and each
    lane adds its products in increasing t, starting from +0.0;
  - the 64 lane sums combine by an xor butterfly (m = 32, 16, ..., 1);
  - the blocks combine by the left-complete pairwise tree
    P(x[0..n)) = P(x[0..h)) + P(x[h..n)), h the largest power of two below n.

Element values come from the oracle's decode (pinned against numpy and torch
casts); every addition below is one IEEE binary64 addition."""
from __future__ import annotations

import math
from typing import Dict, List, Sequence, Tuple

import numpy as np

import oracle

ESIZE = {"f32": 4, "bf16": 2, "f16": 2, "fp8e4m3": 1, "i32": 4, "i64": 8, "u8": 1}
FLOAT = ("f32", "bf16", "f16", "fp8e4m3")
_PIECE = 1 << 24          # elements per piece of work (bounds the memory of long rows)


def lane_terms(dtype: str) -> int:
    """Products one lane adds in a block: 4 chunks of 16 bytes."""
    return 4 * (16 // ESIZE[dtype])


def perfect_tree(x: np.ndarray) -> float:
    """Pairwise sum of 2^k values, neighbours first, level by level."""
    y = np.asarray(x, dtype=np.float64)
    while y.size > 1:
        y = y[0::2] + y[1::2]
    return float(y[0])


def pairwise_tree(x: Sequence[float]) -> float:
    """The left-complete tree: P(x[0..n)) = P(x[0..h)) + P(x[h..n))."""
    x = np.asarray(x, dtype=np.float64)
    n = x.size
    if n == 0:
        return 0.0
    if n == 1:
        return float(x[0])
    h = 1 << ((n - 1).bit_length() - 1)          # largest power of two below n
    return perfect_tree(x[:h]) + pairwise_tree(x[h:])


_TABLES: Dict[str, Tuple[np.ndarray, np.ndarray]] = {}


def _values(dtype: str, raw: np.ndarray):
    """(finite mask, exact float64 values) of raw elements: the oracle's decode,
    tabulated once over every pattern of the 8- and 16-bit types; binary32 by
    numpy's exact widening."""
    if dtype == "f32":
        with np.errstate(invalid="ignore"):      # NaN patterns widen to NaN
            v = raw.astype(np.uint32).view(np.float32).astype(np.float64)
        return np.isfinite(v), v
    if dtype not in _TABLES:
        n = 1 << (8 * ESIZE[dtype])
        cls, val = oracle.decode_n(dtype, np.arange(n, dtype=np.uint64))
        _TABLES[dtype] = (cls == 0, val)
    ok, val = _TABLES[dtype]
    idx = raw.astype(np.intp)
    return ok[idx], val[idx]


def rows_block_sums(dtype: str, ra: np.ndarray, rb: np.ndarray) -> Tuple[np.ndarray, int]:
    """[rows * blocks_per_row, 3] sums (ab, aa, bb), row-major, of rows of equal
    length given the raw elements of both operands ([rows, length] arrays),
    and the number of pairs with both values finite."""
    R, n = ra.shape
    per_block = 4096 // ESIZE[dtype]
    if R == 1 and n > _PIECE:                    # one long row: whole blocks at a time
        step = _PIECE // per_block * per_block
        parts = [_block_sums(dtype, ra[:, k:k + step], rb[:, k:k + step]) for k in range(0, n, step)]
    elif R > 1 and R * n > _PIECE:
        step = max(1, _PIECE // max(n, 1))
        parts = [_block_sums(dtype, ra[k:k + step], rb[k:k + step]) for k in range(0, R, step)]
    else:
        parts = [_block_sums(dtype, ra, rb)]
    return np.concatenate([p[0] for p in parts]), sum(p[1] for p in parts)


def _block_sums(dtype: str, ra: np.ndarray, rb: np.ndarray) -> np.ndarray:
    es = ESIZE[dtype]
    epc, per_block = 16 // es, 4096 // es
    R, n = ra.shape
    nb = -(-n // per_block)
    if R == 0 or nb == 0:
        return np.zeros((0, 3)), 0
    fa, A = _values(dtype, ra)
    fb, B = _values(dtype, rb)
    ok = fa & fb
    A = np.where(ok, A, 0.0)                     # an excluded or missing product adds +0.0: no change
    B = np.where(ok, B, 0.0)
    terms = np.zeros((3, R, nb * per_block))
    terms[0, :, :n] = A * B
    terms[1, :, :n] = A * A
    terms[2, :, :n] = B * B
    # element of a block = ((j * 64 + lane) * epc + e): order the terms (j, e, ..., lane)
    t = np.ascontiguousarray(terms.reshape(3, R * nb, 4, 64, epc).transpose(2, 4, 0, 1, 3))
    lanes = np.zeros((3, R * nb, 64))
    for j in range(4):
        for e in range(epc):
            lanes += t[j, e]
    idx = np.arange(64)
    for m in (32, 16, 8, 4, 2, 1):
        lanes = lanes + lanes[:, :, idx ^ m]
    return lanes[:, :, 0].T, int(np.count_nonzero(ok))


def _finish(blocks: np.ndarray, pairs: int) -> Dict:
    ab = pairwise_tree(blocks[:, 0]) if blocks.size else 0.0
    aa = pairwise_tree(blocks[:, 1]) if blocks.size else 0.0
    bb = pairwise_tree(blocks[:, 2]) if blocks.size else 0.0
    if aa == 0.0 and bb == 0.0:
        c = 1.0
    elif aa == 0.0 or bb == 0.0:
        c = 0.0
    else:
        c = ab / (math.sqrt(aa) * math.sqrt(bb))
    return {"sum_ab": ab, "sum_aa": aa, "sum_bb": bb, "cosine": c, "pairs": pairs, "blocks": blocks.shape[0]}


def _undefined() -> Dict:
    return {"sum_ab": 0.0, "sum_aa": 0.0, "sum_bb": 0.0, "cosine": math.nan, "pairs": 0, "blocks": 0}


def _strided(buf: np.ndarray, off: int, es: int, shape: Sequence[int], strides: Sequence[int]) -> np.ndarray:
    """Raw elements (as uint64) of the view with this shape and these element
    strides, starting at byte `off` of buf."""
    b = np.ascontiguousarray(buf).view(np.uint8).reshape(-1)
    shape = [int(n) for n in shape]
    if any(n == 0 for n in shape):
        return np.zeros(shape, dtype=np.uint64)
    view = np.lib.stride_tricks.as_strided(b[off:], shape=shape + [es], strides=[int(x) * es for x in strides] + [1],
                                           writeable=False)
    raw = np.ascontiguousarray(view).view("<u%d" % es)[..., 0]
    return raw.astype(np.uint64)


def cosine_2d(dtype: str, rows: int, cols: int, sa: int, sb: int, a: np.ndarray, b: np.ndarray,
              a_off: int = 0, b_off: int = 0) -> Dict:
    """A 2-D segment in the documented order (offsets in bytes of a and b)."""
    if dtype not in FLOAT:
        return _undefined()
    es = ESIZE[dtype]
    if rows <= 0 or cols <= 0:
        return _finish(np.zeros((0, 3)), 0)
    if rows == 1 or (sa == cols and sb == cols):
        ra = _strided(a, a_off, es, [1, rows * cols], [0, 1])
        rb = _strided(b, b_off, es, [1, rows * cols], [0, 1])
    else:
        ra = _strided(a, a_off, es, [rows, cols], [sa, 1])
        rb = _strided(b, b_off, es, [rows, cols], [sb, 1])
    return _finish(*rows_block_sums(dtype, ra, rb))


def walk(shape: Sequence[int], sa: Sequence[int], sb: Sequence[int]) -> List[Tuple[int, int, int]]:
    """The documented walk of an N-D segment: dimensions of extent > 1 ordered
    by decreasing stride of a (0 first), ties by decreasing stride of b, a
    stable order; then, from the innermost, a dimension stepping exactly over
    the next-inner one in both operands merges into it.  Returns (n, sa, sb),
    outermost first (one unit dimension if nothing is left)."""
    key = lambda v: math.inf if v == 0 else v
    dims = [(n, x, y) for n, x, y in zip(shape, sa, sb) if n > 1]
    dims = sorted(dims, key=lambda d: (-key(d[1]), -key(d[2])))   # sorted() is stable
    merged: List[List[int]] = []
    for n, x, y in reversed(dims):
        if merged and x == merged[-1][0] * merged[-1][1] and y == merged[-1][0] * merged[-1][2]:
            merged[-1][0] *= n
        else:
            merged.append([n, x, y])
    merged.reverse()
    return [tuple(m) for m in merged] or [(1, 1, 1)]


def cosine_nd(dtype: str, parts: Sequence, a: np.ndarray, b: np.ndarray) -> Dict:
    """One result over N-D segments (shape, stride_a, stride_b, a_off, b_off),
    in segment order, in the documented walk order."""
    if not parts:
        return {"sum_ab": 0.0, "sum_aa": 0.0, "sum_bb": 0.0, "cosine": 1.0, "pairs": 0, "blocks": 0}
    if dtype not in FLOAT:
        return _undefined()
    es = ESIZE[dtype]
    blocks, pairs = [], 0
    for shape, sa, sb, a_off, b_off in parts:
        if any(n == 0 for n in shape):
            continue
        w = walk(shape, sa, sb)                  # rows: the outer dimensions, last fastest
        dims = [d[0] for d in w]
        ra = _strided(a, a_off, es, dims, [d[1] for d in w]).reshape(-1, dims[-1])
        rb = _strided(b, b_off, es, dims, [d[2] for d in w]).reshape(-1, dims[-1])
        sums, p = rows_block_sums(dtype, ra, rb)
        blocks.append(sums)
        pairs += p
    return _finish(np.concatenate(blocks) if blocks else np.zeros((0, 3)), pairs)
