"""Exhaustive GPU parity of the comparison over every (a, b) pair of 16-bit
values: all 2^32 bf16 x bf16 and fp16 x fp16 pairs, under the tolerance rule
with both NaN policies and in bitwise mode.  Segment v compares the table of
all 65536 patterns (a) against pattern v broadcast (b, an N-D segment with
stride 0), so its result summarises the 65536 pairs (a, v): counts, first
index, max abs and max rel must equal the CPU oracle's, field for field.
Then the same invariants on the GPU as on the CPU: splitting a segment adds
counts and takes minima / maxima; swapping a and b with rtol = 0 keeps the
counts.  Last, every pair of 256 patterns per float type (all 65536 fp8
pairs; the special values and seeded bits of fp32, bf16 and fp16) through
the 2-D diff, in whole tiles and in short padded rows."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
import paper_2608_20711_amd as lib
from gpu_helpers import THREADS, assert_results_equal, log
from paper_2608_20711_amd.state import SEG_RESULT_DTYPE

pytestmark = pytest.mark.gpu

N = 1 << 16


def _gpu_nd(segs, n_results):
    res = torch.empty(n_results * SEG_RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    size = lib.diff_nd_workspace_bytes(len(segs))
    ws = torch.empty(size, dtype=torch.uint8, device="cuda")
    lib.diff_segments_nd(lib.descriptor_array(segs), res.data_ptr(), n_results, ws.data_ptr(), size)
    torch.cuda.synchronize()
    raw = res.cpu().numpy().view(SEG_RESULT_DTYPE)
    return [{f: raw[f][k].item() for f in SEG_RESULT_DTYPE.names} for k in range(n_results)]


@pytest.mark.parametrize("dtype,mode,policy,atol,rtol", [
    ("bf16", "tolerance", "equal", 1e-2, 1.6e-2),
    ("bf16", "tolerance", "strict", 0.0, 0.0),
    ("f16", "tolerance", "equal", 1e-3, 1e-3),
    ("f16", "tolerance", "strict", 6e-8, 2.0 ** -11),
    ("f16", "bitwise", "equal", 0.0, 0.0),
])
def test_every_16_bit_pair(dtype, mode, policy, atol, rtol):
    table = np.arange(N, dtype=np.uint16)
    t_dev = torch.from_numpy(table.view(np.uint8).copy()).cuda()
    base = t_dev.data_ptr()
    code = lib.DTYPE_CODE[dtype]
    segs = [lib.segment_nd(base, base + 2 * v, code, lib.MODE_CODE[mode], lib.NAN_CODE[policy], [N], [1], [0],
                           atol, rtol, v, v * N) for v in range(N)]
    log(f"exhaustive {dtype} {mode} {policy}: {N} segments x {N} pairs on the GPU")
    got = _gpu_nd(segs, N)
    raw = table.view(np.uint8)

    def one(v):
        return oracle.diff_segment_nd(dtype, mode, policy, [N], [1], [0], atol, rtol, raw, raw, 0, 2 * v, v * N)

    with ThreadPoolExecutor(THREADS) as ex:
        want = list(ex.map(one, range(N), chunksize=256))
    assert_results_equal(got, want, f"{dtype} {mode} {policy} pairs")
    total = sum(r["mismatches"] for r in want)
    log(f"exhaustive {dtype} {mode} {policy}: {total} mismatching pairs of 2^32, all fields equal")
    assert 0 < total < N * N


def test_split_and_swap_invariants_on_the_gpu():
    rng = np.random.default_rng(31)
    n = 1_000_003
    b = rng.standard_normal(n).astype(np.float32)
    a = (b + rng.standard_normal(n).astype(np.float32) * 1e-4).astype(np.float32)
    a[rng.choice(n, 50, replace=False)] = np.nan
    a_d = torch.from_numpy(a.view(np.uint8).copy()).cuda()
    b_d = torch.from_numpy(b.view(np.uint8).copy()).cuda()
    A, B = a_d.data_ptr(), b_d.data_ptr()
    f32, tol, eq = lib.F32, lib.TOLERANCE, lib.NAN_EQUAL
    whole = lib.segment_nd(A, B, f32, tol, eq, [n], [1], [1], 1e-4, 1e-4, 0, 0)
    cut = 123_457
    # two halves sharing result 1, with the second half's index base
    first = lib.segment_nd(A, B, f32, tol, eq, [cut], [1], [1], 1e-4, 1e-4, 1, 0)
    second = lib.segment_nd(A + 4 * cut, B + 4 * cut, f32, tol, eq, [n - cut], [1], [1], 1e-4, 1e-4, 1, cut)
    # swapped operands with rtol = 0
    s_ab = lib.segment_nd(A, B, f32, tol, eq, [n], [1], [1], 1e-4, 0.0, 2, 0)
    s_ba = lib.segment_nd(B, A, f32, tol, eq, [n], [1], [1], 1e-4, 0.0, 3, 0)
    r = _gpu_nd([whole, first, second, s_ab, s_ba], 4)
    assert r[0] == r[1]
    assert r[2]["mismatches"] == r[3]["mismatches"] and r[2]["first_mismatch"] == r[3]["first_mismatch"]
    assert r[2]["max_abs"] == r[3]["max_abs"]
    want = oracle.diff_segment("f32", "tolerance", "equal", 1, n, n, n, 1e-4, 1e-4, a.view(np.uint8),
                               b.view(np.uint8))
    assert_results_equal([r[0]], [want], "whole")


def _patterns(dtype):
    """256 element patterns per dtype: every fp8 e4m3 byte; for the wider
    types the special values of the format (signed zeros, the smallest and
    largest subnormals and normals, the largest finite values, infinities,
    quiet and signalling NaNs with payloads and either sign), neighbours of 1
    one and two units in the last place apart, and seeded random bits."""
    if dtype == "fp8e4m3":
        return np.arange(256, dtype=np.uint8)
    ut = {"f32": np.uint32, "bf16": np.uint16, "f16": np.uint16}[dtype]
    sign = {"f32": 0x80000000, "bf16": 0x8000, "f16": 0x8000}[dtype]
    one = {"f32": 0x3F800000, "bf16": 0x3F80, "f16": 0x3C00}[dtype]
    inf = {"f32": 0x7F800000, "bf16": 0x7F80, "f16": 0x7C00}[dtype]
    mant = {"f32": 0x7FFFFF, "bf16": 0x7F, "f16": 0x3FF}[dtype]
    special = [0, 1, 2, mant, mant + 1, mant + 2, inf - 1, inf - 2, inf, inf + 1, inf | (mant >> 1) + 1,
               inf | mant, inf | 0x5, one, one + 1, one + 2, one - 1, one - 2, one + 0x10, one + 3]
    special += [v ^ sign for v in special]
    rng = np.random.default_rng(0x5EED + len(dtype))
    bits = 8 * np.dtype(ut).itemsize
    rand = rng.integers(0, 1 << bits, size=256 - len(special), dtype=np.uint64)
    return np.array(special + [int(r) for r in rand], dtype=ut).view(np.uint8)


@pytest.mark.parametrize("dtype,mode,policy,atol,rtol", [
    ("fp8e4m3", "tolerance", "equal", 0.125, 0.125),
    ("fp8e4m3", "tolerance", "strict", 0.0, 0.0),
    ("fp8e4m3", "tolerance", "strict", 0.125, 0.125),
    ("fp8e4m3", "bitwise", "equal", 0.0, 0.0),
    ("f32", "tolerance", "equal", 1e-5, 1e-5),
    ("f32", "tolerance", "strict", 0.0, 2.0 ** -23),
    ("bf16", "tolerance", "equal", 1e-2, 1.6e-2),
    ("f16", "tolerance", "strict", 1e-3, 1e-3),
    ("f32", "bitwise", "equal", 0.0, 0.0),
])
def test_all_pairs_of_256_patterns_through_the_2d_diff(dtype, mode, policy, atol, rtol):
    """Every pair of 256 element patterns (all 256 for fp8 e4m3) through
    asmevo_diff_segments, in whole tiles and in short padded rows (the
    row-tiled and the narrow walks).  Segment v compares the 256 patterns,
    repeated to 16 KiB, against pattern v; the rows layout holds the same
    elements as rows of 256 at a pitch 16 bytes longer, so both layouts give
    the same logical indices and must give the same results, equal to the
    CPU oracle's field for field."""
    from paper_2608_20711_amd.state import SEG_RESULT_DTYPE as RES
    pat = _patterns(dtype)
    es = pat.size // 256
    cols = 256
    reps = 16384 // (cols * es)
    pitch = cols * es + 16
    n = reps * cols
    flat = np.tile(pat, reps)
    rows = np.zeros(reps * pitch, dtype=np.uint8)
    rows.reshape(reps, pitch)[:, :cols * es] = pat
    rows.reshape(reps, pitch)[:, cols * es:] = 0xFF               # pads: never compared
    b_flat = np.concatenate([np.tile(pat[v * es:(v + 1) * es], n) for v in range(256)])
    b_rows = np.concatenate([np.tile(pat[v * es:(v + 1) * es], reps * pitch // es) for v in range(256)])
    code, m, p = lib.DTYPE_CODE[dtype], lib.MODE_CODE[mode], lib.NAN_CODE[policy]
    out = {}
    for name, a_h, b_h, r, c, s in (("tiles", flat, b_flat, 1, n, n),
                                    ("rows", rows, b_rows, reps, cols, pitch // es)):
        a_d = torch.from_numpy(a_h).cuda()
        b_d = torch.from_numpy(b_h).cuda()
        step = b_h.size // 256
        segs = [lib.Segment(a_d.data_ptr(), b_d.data_ptr() + v * step, code, m, p, 0, r, c, s, s, atol, rtol)
                for v in range(256)]
        res = torch.empty(256 * RES.itemsize, dtype=torch.uint8, device="cuda")
        ws_size = lib.workspace_bytes(256)
        ws = torch.empty(ws_size, dtype=torch.uint8, device="cuda")
        log(f"{dtype} pattern pairs {mode} {policy} {atol}: {name} layout, 256 segments")
        lib.diff_segments(segs, res.data_ptr(), ws.data_ptr(), ws_size)
        torch.cuda.synchronize()
        raw = res.cpu().numpy().view(RES)
        got = [{f: raw[f][k].item() for f in RES.names} for k in range(256)]
        want = [oracle.diff_segment(dtype, mode, policy, r, c, s, s, atol, rtol, a_h, b_h, 0, v * step)
                for v in range(256)]
        assert_results_equal(got, want, f"{dtype} {mode} {policy} {name}")
        out[name] = got
    assert_results_equal(out["rows"], out["tiles"], f"{dtype} layouts")
    assert sum(r["mismatches"] for r in out["tiles"]) > 0
