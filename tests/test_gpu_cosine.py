"""GPU parity of the cosine term of Eq. 1 (c = cos(K'(x), O(x)) per buffer):
the HIP diff+cosine pass against the CPU oracle's exact sums, within the
error bound of the library's documented summation order (pair counts
exactly), and bit for bit against a model of that order (reproducibility),
on the workloads and on odd layouts.  The diff results of the same pass must
equal those of the plain diff."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_20711_amd as lib
import workloads
from gpu_helpers import (THREADS, assert_cosine, cosine_expected, cosine_workload_expected, log,
                         run_gpu)
from paper_2608_20711_amd.state import COS_RESULT_DTYPE, SEG_RESULT_DTYPE
from workloads import ESIZE

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", list(workloads.ALL))
def test_cosine_reduced_workloads(name):
    w = workloads.ALL[name](small=True)
    st = run_gpu(w)
    plain = st.seg_results()
    st.diff_cosine()
    got = st.cos_results()
    assert st.seg_results() == plain                 # same diff results from the fused pass
    cand, ref = st.arena_host("cand"), st.arena_host("ref")
    assert_cosine(got, *cosine_workload_expected(w, cand, ref), f"{name} cosine")


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["single_fp32", "padded_bf16", "decode_state", "int_lowp"])
def test_cosine_full_size(name):
    w = workloads.ALL[name]()
    log(f"[cosine full] {name}")
    st = run_gpu(w)
    plain = st.seg_results()
    st.diff_cosine()
    got = st.cos_results()
    assert st.seg_results() == plain
    cand, ref = st.arena_host("cand"), st.arena_host("ref")
    assert_cosine(got, *cosine_workload_expected(w, cand, ref), f"{name} cosine")
    for r, c in zip(got, w.compares):
        if w.allocs[c.alloc].dtype in workloads.FLOAT_DTYPES:
            assert r["cosine"] > 0.99


def _cos_gpu(specs, a_d, b_d):
    segs = [lib.Segment(a_d.data_ptr() + s["a_off"], b_d.data_ptr() + s["b_off"], lib.DTYPE_CODE[s["dtype"]],
                        lib.BITWISE, 0, 0, s["rows"], s["cols"], s["sa"], s["sb"], 0.0, 0.0) for s in specs]
    for s in specs:
        for off, st, buf in ((s["a_off"], s["sa"], a_d), (s["b_off"], s["sb"], b_d)):
            ext = 0 if s["rows"] == 0 or s["cols"] == 0 else ((s["rows"] - 1) * st + s["cols"]) * ESIZE[s["dtype"]]
            assert off + ext <= buf.numel(), s
    n = len(segs)
    res = torch.empty(n * SEG_RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    cres = torch.empty(n * COS_RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    size = lib.diff_cosine_workspace_bytes(segs)
    ws = torch.empty(size, dtype=torch.uint8, device="cuda")
    lib.diff_cosine(segs, res.data_ptr(), cres.data_ptr(), ws.data_ptr(), size)
    torch.cuda.synchronize()
    raw = cres.cpu().numpy().view(COS_RESULT_DTYPE)
    return [{f: raw[f][k].item() for f in COS_RESULT_DTYPE.names} for k in range(n)]


def _check(got, specs, a_h, b_h, what):
    exp = [cosine_expected(s["dtype"], s["rows"], s["cols"], s["sa"], s["sb"], a_h, b_h, s["a_off"], s["b_off"])
           for s in specs]
    assert_cosine(got, [e[0] for e in exp], [e[1] for e in exp], [s["dtype"] for s in specs], what)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16", "fp8e4m3", "i32"])
def test_cosine_layouts_and_specials(dtype):
    rng = np.random.default_rng(17)
    es = ESIZE[dtype]
    nbytes = 2 << 20
    n = nbytes // es
    raw = rng.integers(0, 1 << (8 * es), size=2 * n, dtype=np.uint64)
    if dtype in ("f32", "bf16", "f16", "fp8e4m3"):
        # mostly ordinary values, a sprinkling of every special pattern
        vals = (rng.standard_normal(2 * n) * 3).astype(np.float32)
        if dtype == "f32":
            raw = vals.view(np.uint32).astype(np.uint64)
        elif dtype == "bf16":
            raw = (vals.view(np.uint32) >> 16).astype(np.uint64)
        elif dtype == "f16":
            raw = vals.astype(np.float16).view(np.uint16).astype(np.uint64)
        else:
            raw = raw & 0x7F
            raw[raw == 0x7F] = 0x3C
        k = rng.integers(0, 2 * n, size=2 * n // 200)
        raw[k] = rng.integers(0, 1 << (8 * es), size=k.size, dtype=np.uint64)   # any pattern, NaN/Inf included
    npt = {1: np.uint8, 2: np.uint16, 4: np.uint32}[es]
    a_h = raw[:n].astype(npt).view(np.uint8).copy()
    b_h = raw[n:].astype(npt).view(np.uint8).copy()
    a_d, b_d = torch.from_numpy(a_h).cuda(), torch.from_numpy(b_h).cuda()
    spec = lambda rows, cols, sa, sb, ao=0, bo=0: dict(dtype=dtype, rows=rows, cols=cols, sa=sa, sb=sb,
                                                     a_off=ao, b_off=bo)
    specs = [spec(1, n, n, n), spec(1, n - 5, n, n, es, 3 * es), spec(1, 4096 // es * 7 + 3, 0, 0),
             spec(3, 1000, 1000, 1000), spec(41, 2000, 2048, 2048), spec(77, 1001, 1003, 1009, 0, es),
             spec(300, 10, 13, 11), spec(1, 1, 1, 1, 7 * es, 9 * es), spec(0, 5, 5, 5)]
    for s in specs:
        s["sa"] = max(s["sa"], s["cols"])
        s["sb"] = max(s["sb"], s["cols"])
    got = _cos_gpu(specs, a_d, b_d)
    _check(got, specs, a_h, b_h, f"{dtype} cosine layouts")


def test_cosine_every_fp8_and_f16_value():
    """Single-block segments over every fp8 pattern and every fp16 pattern
    (the GPU's element conversions against the oracle's decode)."""
    a8 = np.arange(256, dtype=np.uint8)
    b8 = np.roll(a8, 37).copy()
    a16 = np.arange(1 << 16, dtype=np.uint16)
    b16 = np.roll(a16, 1001).copy()
    for dtype, a_h, b_h in (("fp8e4m3", a8, b8), ("f16", a16.view(np.uint8), b16.view(np.uint8))):
        es = ESIZE[dtype]
        n = a_h.size // es
        a_d, b_d = torch.from_numpy(a_h.copy()).cuda(), torch.from_numpy(b_h.copy()).cuda()
        per = 64 if dtype == "f16" else 16
        specs = [dict(dtype=dtype, rows=1, cols=per, sa=per, sb=per, a_off=i * es, b_off=i * es)
                 for i in range(0, n, per)]
        got = _cos_gpu(specs, a_d, b_d)
        _check(got, specs, a_h, b_h, f"{dtype} every value")


@pytest.mark.timeout(300)
def test_cosine_tree_levels_with_leftovers():
    """Segments whose block counts leave entries at every level of the block
    tree: 65536 + 5 * 256 + 3 blocks (one level-2 group, five level-1
    groups, three single blocks), 3 * 256 + 255 and 257 blocks, and a 2-D
    segment whose rows end in partial blocks."""
    rng = np.random.default_rng(21)
    n_blocks = 65536 + 5 * 256 + 3
    n1 = n_blocks * 1024                                   # fp32: 1024 values per 4096-byte block
    a = rng.standard_normal(n1 + 8192).astype(np.float32)
    b = (a + rng.standard_normal(a.size).astype(np.float32) * 1e-3).astype(np.float32)
    a_d = torch.from_numpy(a.view(np.uint8).copy()).cuda()
    b_d = torch.from_numpy(b.view(np.uint8).copy()).cuda()
    specs = [dict(dtype="f32", rows=1, cols=n1, sa=n1, sb=n1, a_off=0, b_off=0),
             dict(dtype="f32", rows=1, cols=(3 * 256 + 255) * 1024, sa=1, sb=1, a_off=4096, b_off=4096),
             dict(dtype="f32", rows=1, cols=257 * 1024 - 5, sa=1, sb=1, a_off=64, b_off=128),
             dict(dtype="f32", rows=300, cols=1500, sa=1600, sb=1536, a_off=0, b_off=4)]
    for s in specs:
        s["sa"] = max(s["sa"], s["cols"])
        s["sb"] = max(s["sb"], s["cols"])
    got = _cos_gpu(specs, a_d, b_d)
    _check(got, specs, a.view(np.uint8), b.view(np.uint8), "cosine tree levels")
    assert got[0]["blocks"] == n_blocks


def test_cosine_many_small_segments_mixed_dtypes():
    """Hundreds of segments of 1 element to 9 blocks, of four float dtypes and
    int32, in one call: the four waves of a workgroup take the tiles of one
    range in turn, so most ranges start and end inside segments and most
    segments are shared by several waves.  Sums, cosine and pair counts equal
    the oracle's; the diff results equal the plain diff's."""
    rng = np.random.default_rng(99)
    nbytes = 8 << 20
    vals = (rng.standard_normal(nbytes // 4) * 2).astype(np.float32)
    a_h = vals.view(np.uint8).copy()
    b_h = a_h.copy()
    flip = rng.integers(0, nbytes, size=2000)
    a_h[flip] ^= 0x10
    a_d, b_d = torch.from_numpy(a_h).cuda(), torch.from_numpy(b_h).cuda()
    specs, off = [], 0
    dtypes = ["f32", "bf16", "f16", "fp8e4m3", "i32"]
    for k in range(700):
        dt = dtypes[k % 5]
        es = ESIZE[dt]
        nb = int(rng.choice([es, 4096 - es, 4096, 4096 + es, 3 * 4096 + 16, 9 * 4096, int(rng.integers(1, 40000))]))
        cols = max(1, nb // es)
        if off + cols * es > nbytes:
            off = 0
        specs.append(dict(dtype=dt, rows=1, cols=cols, sa=cols, sb=cols, a_off=off, b_off=off))
        off = (off + cols * es + 15) // 16 * 16
    log(f"[cosine small] {len(specs)} segments")
    got = _cos_gpu(specs, a_d, b_d)
    _check(got, specs, a_h, b_h, "many small segments cosine")


@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8e4m3"])
def test_cosine_every_short_row_width(dtype):
    """Rows of 1 to 32 chunks (plus a partial chunk, and aligned or misaligned
    pitches) are packed several to a wave-load, a lane holding chunks t and
    t + P of its row (2P the power of two at or above the row's chunks) and
    each group of P lanes finishing the butterfly: the cosine of every such
    width, with NaN and Inf among the values, against the oracle's 64-lane
    definition."""
    rng = np.random.default_rng(31)
    es = ESIZE[dtype]
    n = (4 << 20) // es
    vals = (rng.standard_normal(2 * n) * 2).astype(np.float32)
    if dtype == "f32":
        raw = vals.view(np.uint32).astype(np.uint64)
    elif dtype == "bf16":
        raw = (vals.view(np.uint32) >> 16).astype(np.uint64)
    else:
        raw = rng.integers(0, 0x7F, size=2 * n).astype(np.uint64)
    k = rng.integers(0, 2 * n, size=2 * n // 500)
    raw[k] = rng.integers(0, 1 << (8 * es), size=k.size, dtype=np.uint64)     # NaN / Inf among them
    npt = {1: np.uint8, 2: np.uint16, 4: np.uint32}[es]
    a_h = raw[:n].astype(npt).view(np.uint8).copy()
    b_h = raw[n:].astype(npt).view(np.uint8).copy()
    a_d, b_d = torch.from_numpy(a_h).cuda(), torch.from_numpy(b_h).cuda()
    epc = 16 // es
    specs = []
    for chunks in range(1, 33):
        for extra, pad in ((0, 0), (epc // 2, 3), (0, epc)):
            cols = max(1, (chunks - (1 if extra else 0)) * epc + extra)
            pitch = cols + pad
            rows = 37
            if rows * pitch > n:
                continue
            specs.append(dict(dtype=dtype, rows=rows, cols=cols, sa=pitch, sb=pitch, a_off=0, b_off=0))
    got = _cos_gpu(specs, a_d, b_d)
    _check(got, specs, a_h, b_h, f"{dtype} short rows cosine")
    assert all(g["blocks"] == 37 for g, s in zip(got, specs) if s["sa"] > s["cols"])   # padded: a block per row
