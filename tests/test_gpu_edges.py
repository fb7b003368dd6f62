"""GPU parity on edge cases: misaligned and strided operands, ragged rows,
empty segments, every dtype / mode / NaN policy on random bit patterns, every
fp8 pair, per-pair relative errors (single-element segments, so every GPU
division is compared with the CPU's), encoder edge values, overlapping
injections, guard writes, and the fill's distributions on odd geometries."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_20711_amd as lib
from gpu_helpers import (THREADS, assert_bytes_equal, assert_fill_equal, assert_results_equal, log,
                         run_gpu)
from paper_2608_20711_amd.state import SEG_RESULT_DTYPE, DeviceState
from workloads import ESIZE, Alloc, Compare, Injection, Workload

pytestmark = pytest.mark.gpu

_NP = {1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}


def _extent(s, stride):
    if s["rows"] == 0 or s["cols"] == 0:
        return 0
    return ((s["rows"] - 1) * stride + s["cols"]) * ESIZE[s["dtype"]]


def _gpu_diff(seg_specs, a_dev, b_dev, workgroups=0):
    """seg_specs: list of dicts with dtype/mode/policy/rows/cols/sa/sb/atol/rtol/a_off/b_off."""
    segs = []
    for s in seg_specs:
        # every byte a segment names must lie inside the buffers (checked before launch)
        assert s["a_off"] + _extent(s, s["sa"]) <= a_dev.numel(), s
        assert s["b_off"] + _extent(s, s["sb"]) <= b_dev.numel(), s
        segs.append(lib.Segment(a_dev.data_ptr() + s["a_off"], b_dev.data_ptr() + s["b_off"],
                                lib.DTYPE_CODE[s["dtype"]], lib.MODE_CODE[s["mode"]],
                                lib.NAN_CODE[s["policy"]], 0, s["rows"], s["cols"], s["sa"], s["sb"],
                                s["atol"], s["rtol"]))
    n = len(segs)
    res = torch.empty(max(1, n) * SEG_RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    ws_size = lib.workspace_bytes(n)
    ws = torch.empty(ws_size, dtype=torch.uint8, device="cuda")
    lib.diff_segments(segs, res.data_ptr(), ws.data_ptr(), ws_size, workgroups=workgroups)
    torch.cuda.synchronize()
    raw = res.cpu().numpy()[: n * SEG_RESULT_DTYPE.itemsize].view(SEG_RESULT_DTYPE)
    return [{f: raw[f][k].item() for f in SEG_RESULT_DTYPE.names} for k in range(n)]


def _ora_diff(seg_specs, a_host, b_host):
    return [oracle.diff_segment(s["dtype"], s["mode"], s["policy"], s["rows"], s["cols"], s["sa"], s["sb"],
                                s["atol"], s["rtol"], a_host, b_host, s["a_off"], s["b_off"])
            for s in seg_specs]


def _spec(dtype, rows, cols, sa, sb, a_off, b_off, mode="tolerance", policy="equal", atol=1e-3, rtol=1e-3):
    if dtype in ("i32", "i64", "u8"):
        mode = "bitwise"
    return dict(dtype=dtype, mode=mode, policy=policy, rows=rows, cols=cols, sa=sa, sb=sb,
                atol=atol, rtol=rtol, a_off=a_off, b_off=b_off)


def _random_pair(nbytes, dtype, rng, rate=0.02):
    """b: random normal-ish values of dtype (as bytes); a: b with sparse edits."""
    es = ESIZE[dtype]
    n = nbytes // es
    if dtype == "f32":
        b = (rng.standard_normal(n) * 3).astype(np.float32).view(np.uint32)
    elif dtype == "f16":
        b = (rng.standard_normal(n) * 3).astype(np.float16).view(np.uint16)
    elif dtype == "bf16":
        b = ((rng.standard_normal(n) * 3).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    else:
        b = rng.integers(0, 1 << min(63, 8 * es), size=n, dtype=np.uint64).astype(_NP[es])
    a = b.copy()
    k = rng.random(n) < rate
    idx = np.flatnonzero(k)
    kinds = rng.integers(0, 4, size=idx.size)
    for t, i in zip(kinds, idx):
        if t == 0:
            a[i] ^= _NP[es](1) << _NP[es](int(rng.integers(0, 8 * es)))
        elif t == 1:
            a[i] = _NP[es](int(a[i]) + 1 & ((1 << (8 * es)) - 1))
        elif t == 2 and dtype == "f32":
            a[i] = np.uint32(0x7FC00000)
        elif t == 2 and dtype in ("f16",):
            a[i] = np.uint16(0x7E00)
        elif t == 2 and dtype == "bf16":
            a[i] = np.uint16(0x7F80)
        else:
            a[i] = _NP[es](int(rng.integers(0, 1 << min(63, 8 * es))))
    # NaNs in b too, matched and unmatched
    nb = max(1, n // 500)
    pos = rng.integers(0, n, size=nb)
    nan = {"f32": 0x7FC00001, "f16": 0x7E01, "bf16": 0x7FC1, "fp8e4m3": 0x7F}.get(dtype)
    if nan is not None:
        b[pos] = _NP[es](nan)
        a[pos[: nb // 2]] = _NP[es](nan)
    return a.view(np.uint8), b.view(np.uint8)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16", "fp8e4m3", "i32", "i64", "u8"])
def test_random_patterns_all_layouts(dtype):
    rng = np.random.default_rng(hash(dtype) & 0xFFFF)
    es = ESIZE[dtype]
    nbytes = 3 << 20
    a_h, b_h = _random_pair(nbytes, dtype, rng)
    a_h = np.concatenate([a_h, np.zeros(4096, np.uint8)])
    b_h = np.concatenate([b_h, np.zeros(4096, np.uint8)])
    a_d = torch.from_numpy(a_h).cuda()
    b_d = torch.from_numpy(b_h).cuda()
    n = nbytes // es
    specs = []
    for policy in ("equal", "strict"):
        specs.append(_spec(dtype, 1, n, n, n, 0, 0, policy=policy))                      # contiguous, aligned
    specs.append(_spec(dtype, 1, n - 7, n, n, es, 3 * es))                               # misaligned a and b
    specs.append(_spec(dtype, 1, 10_007, 10_007, 10_007, 16, 16))                        # ragged tail
    rows2d = min(999, n // 1024 - 1)
    specs.append(_spec(dtype, rows2d, 1000, 1024, 1024, 0, 0))                           # 2-D, 16-B pitches
    rows3 = min(333, n // 1009 - 1)
    specs.append(_spec(dtype, rows3, 1001, 1003, 1009, 0, es, policy="strict"))          # 2-D ragged, misaligned
    specs.append(_spec(dtype, 4, 3, 5, 3, 32, 64))                                       # tiny 2-D
    specs.append(_spec(dtype, 1, 1, 1, 1, es * 5, es * 9))                               # one element
    specs.append(_spec(dtype, 0, 10, 10, 10, 0, 0))                                      # empty
    specs.append(_spec(dtype, 10, 0, 0, 0, 0, 0))                                        # empty
    if dtype in ("f32", "bf16", "f16", "fp8e4m3"):
        specs.append(_spec(dtype, 1, n, n, n, 0, 0, mode="bitwise"))
        specs.append(_spec(dtype, 1, n, n, n, 0, 0, atol=0.0, rtol=0.0))
        specs.append(_spec(dtype, 1, n, n, n, 0, 0, atol=0.5, rtol=0.0))
    log(f"[random] {dtype}: {len(specs)} segments")
    got = _gpu_diff(specs, a_d, b_d)
    want = _ora_diff(specs, a_h, b_h)
    assert_results_equal(got, want, f"{dtype} random")
    for wg in (1, 5, 333):
        assert _gpu_diff(specs, a_d, b_d, workgroups=wg) == got


@pytest.mark.parametrize("atol,rtol", [(0.125, 0.125), (0.0, 0.0), (1e-3, 0.0), (0.0, 0.5)])
def test_every_fp8_pair(atol, rtol):
    a, b = np.meshgrid(np.arange(256, dtype=np.uint8), np.arange(256, dtype=np.uint8))
    a_h, b_h = a.ravel().copy(), b.ravel().copy()
    a_d, b_d = torch.from_numpy(a_h).cuda(), torch.from_numpy(b_h).cuda()
    specs = [_spec("fp8e4m3", 1, 65536, 65536, 65536, 0, 0, policy=p, atol=atol, rtol=rtol)
             for p in ("equal", "strict")]
    # and one single-element segment per pair for the per-pair maxima (every division)
    specs += [_spec("fp8e4m3", 1, 1, 1, 1, i, i, atol=atol, rtol=rtol) for i in range(0, 65536, 3)]
    assert_results_equal(_gpu_diff(specs, a_d, b_d), _ora_diff(specs, a_h, b_h), "fp8 pairs")


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_per_pair_relative_error_divisions(dtype):
    """Single-element segments make max_abs / max_rel the values of one pair,
    so each GPU fp64 division is compared with the CPU's."""
    rng = np.random.default_rng(31)
    es = ESIZE[dtype]
    n = 60_000
    raw = rng.integers(0, 1 << (8 * es), size=2 * n, dtype=np.uint64).astype(_NP[es])
    a_h, b_h = raw[:n].view(np.uint8).copy(), raw[n:].view(np.uint8).copy()
    a_d, b_d = torch.from_numpy(a_h).cuda(), torch.from_numpy(b_h).cuda()
    specs = [_spec(dtype, 1, 1, 1, 1, i * es, i * es, atol=1e-3, rtol=1e-2) for i in range(n)]
    assert_results_equal(_gpu_diff(specs, a_d, b_d), _ora_diff(specs, a_h, b_h), f"{dtype} divisions")


def test_zero_segments_and_argument_errors():
    res = torch.zeros(64, dtype=torch.uint8, device="cuda")
    ws = torch.empty(4096, dtype=torch.uint8, device="cuda")
    lib.diff_segments([], res.data_ptr(), ws.data_ptr(), 4096)
    torch.cuda.synchronize()
    assert int(res.sum()) == 0           # nothing written for n = 0
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_segments([lib.Segment(16, 16, lib.F32, lib.TOLERANCE, 0, 0, 1, 8, 4, 8, 0.0, 0.0)],
                          res.data_ptr(), ws.data_ptr(), 4096)
    assert e.value.status == lib.E_INVALID
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_segments([lib.Segment(16, 16, lib.F32, 0, 0, 0, 1, 8, 8, 8, 0.0, 0.0)],
                          res.data_ptr(), ws.data_ptr(), 8)
    assert e.value.status == lib.E_WORKSPACE


# ------------------------------------------------------------------ fills
def _fill_parity(w, variants=(0, 1, 2)):
    """Fill parity for each variant, and guard-check parity on each fill."""
    from paper_2608_20711_amd.state import DeviceState
    st = DeviceState(w)
    P = oracle.Prepared(w)
    for v in variants:
        st.fill("cand", v)
        st.guard()
        torch.cuda.synchronize()
        cand = P.fill_arena(v, THREADS)
        assert_fill_equal(w, st.arena_host("cand"), cand, f"{w.name} variant {v}")
        assert_results_equal(st.guard_results(), oracle.guard_workload(w, cand), f"{w.name} guards {v}")
    return st


def test_fill_encoder_edge_values():
    vals = [0.0, -0.0, 1.0, -1.5, 1e-45, -1e-45, 1.17549435e-38, 5.9e-8, 2.0 ** -24, 2.0 ** -25,
            3 * 2.0 ** -26, 2.0 ** -25 * 1.0000001, 6.1e-5, 65504.0, 65519.0, 65520.0, 1e5, 3.4e38,
            448.0, 464.0, 465.0, 480.0, 1000.0, -464.0, 2.0 ** -9, 2.0 ** -10, 3 * 2.0 ** -11,
            0.0068359375, 0.001953125 * 1.5, 1.0 / 3.0, -2.0 / 3.0, 255.99, 256.0, 3.0e-39]
    allocs = []
    for dt in ("f32", "bf16", "f16", "fp8e4m3"):
        for sat in (False, True):
            if sat and dt != "fp8e4m3":
                continue
            for v in vals:
                allocs.append(Alloc(len(allocs), dt, 1, 24, 24, 0, 0, "const", p0=v, saturate=sat))
    w = Workload("encoder_edges", "", 77, allocs, [], [])
    _fill_parity(w, variants=(0,))


def test_fill_geometry_distributions_and_injections():
    allocs = [
        Alloc(0, "f32", 7, 33, 40, 24, 40, "normal", 1.5, 2.0),               # 2-D, pads, odd guards
        Alloc(1, "bf16", 1, 1001, 1001, 6, 13, "normal", 0.0, 8.0),
        Alloc(2, "f16", 13, 17, 21, 2, 3, "normal", -1.0, 0.5),
        Alloc(3, "fp8e4m3", 3, 333, 340, 5, 7, "normal", 0.0, 100.0, saturate=True),
        Alloc(4, "fp8e4m3", 1, 4099, 4099, 0, 0, "normal", 0.0, 100.0, saturate=False),
        Alloc(5, "i32", 5, 99, 100, 16, 16, "uniform_int", i0=-1000, i1=1 << 20),
        Alloc(6, "i64", 9, 7, 8, 8, 24, "uniform_int", i0=5, i1=(1 << 32) + 5),
        Alloc(7, "u8", 1, 777, 777, 3, 5, "bits"),
        Alloc(8, "f32", 3, 5, 5, 0, 0, "uniform_int", i0=-3, i1=3),
        Alloc(9, "i64", 1, 100, 100, 8, 8, "bits"),
        Alloc(10, "f16", 0, 5, 5, 10, 10, "normal"),                              # empty data, guards only
        Alloc(11, "bf16", 2, 2, 2, 0, 0, "const", p0=2.5),
        Alloc(12, "i32", 4, 4, 4, 0, 0, "const", i0=-7),
    ]
    inj = [
        Injection(0, "flip_bit", arg=-1, rate=0.05),
        Injection(0, "step_within", sides="both", rate=0.03, atol=1e-3, rtol=1e-3),
        Injection(0, "set_beyond", index=5, atol=1e-3, rtol=1e-3),
        Injection(0, "set_nan", index=5),                                         # overrides the line above
        Injection(0, "set_inf", arg=1, index=200),
        Injection(0, "guard_write_lo", arg=3, index=7),
        Injection(0, "guard_write_hi", sides="both", arg=40, index=0),
        Injection(1, "flip_bit", arg=0, rate=0.5),
        Injection(1, "flip_bit", arg=15, rate=0.5),
        Injection(1, "set_inf", sides="both", index=1000),
        Injection(2, "step_within", index=0, atol=1e-3, rtol=1e-3),
        Injection(2, "set_beyond", index=200, atol=1e-3, rtol=1e-3),
        Injection(3, "set_beyond", index=7, atol=0.125, rtol=0.125),
        Injection(3, "step_within", rate=0.01),
        Injection(3, "set_nan", sides="both", index=998),
        Injection(4, "flip_bit", arg=-1, rate=0.001),
        Injection(5, "flip_bit", arg=31, index=494),
        Injection(6, "flip_bit", arg=-1, rate=0.2),
        Injection(6, "flip_bit", arg=63, index=62),
        Injection(7, "flip_bit", arg=-1, rate=1.0),
        Injection(9, "guard_write_hi", arg=8, index=0),
        Injection(11, "set_nan", index=3),
    ]
    w = Workload("geometry", "", 0xFEEDFACE, allocs, inj, [])
    st = _fill_parity(w, variants=(0, 1, 7, 65535))
    g = st.guard_results()
    assert g[0]["bad_lo"] == 3 and g[0]["first_bad_lo"] == 7 and g[0]["bad_hi"] == 40
    assert g[9]["bad_hi"] == 8 and g[9]["first_bad_hi"] == 0


@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8e4m3", "i64"])
def test_every_narrow_row_width(dtype):
    """Rows under half a tile (1 to 127 chunks of 16 bytes, plus partial
    chunks) take the narrow path, where a lane divides its chunk index by the
    row's chunks once per tile and steps its other chunks 64 apart: every such
    width, with 16-byte and odd pitches, as 2-D segments and as N-D views,
    equals the oracle field for field, for several grid sizes."""
    rng = np.random.default_rng(0x5EED + ESIZE[dtype])
    es = ESIZE[dtype]
    nbytes = 6 << 20
    a_h, b_h = _random_pair(nbytes, dtype, rng, rate=0.01)
    a_d = torch.from_numpy(a_h).cuda()
    b_d = torch.from_numpy(b_h).cuda()
    epc = 16 // es
    specs, nd = [], []
    off = 0
    for chunks in list(range(1, 128)) + [129]:
        for extra in (0, 1) if epc > 1 else (0,):            # whole chunks, or one element more
            cols = chunks * epc + extra
            pitch = cols + (epc if chunks % 3 else 1)       # 16-byte pitches, or odd ones
            rows = 1 + (37 * chunks) % 11 + (3000 // chunks) % 40
            ext = ((rows - 1) * pitch + cols) * es
            if off + ext + 64 > nbytes:
                off = 0
            specs.append(_spec(dtype, rows, cols, pitch, pitch, off, off))
            nd.append((rows, cols, pitch, off))
            off += ((ext + 4095) // 4096) * 4096 // 3 * 2 // 16 * 16
    log(f"[narrow] {dtype}: {len(specs)} 2-D segments")
    got = _gpu_diff(specs, a_d, b_d)
    want = _ora_diff(specs, a_h, b_h)
    assert_results_equal(got, want, f"{dtype} narrow 2-D")
    for wg in (1, 7, 300):
        assert _gpu_diff(specs, a_d, b_d, workgroups=wg) == got
    # the same rows as N-D views [rows, cols] / [pitch, 1]
    segs = []
    for k, (rows, cols, pitch, o) in enumerate(nd):
        mode = "bitwise" if dtype in ("i32", "i64", "u8") else "tolerance"
        segs.append(lib.segment_nd(a_d.data_ptr() + o, b_d.data_ptr() + o, lib.DTYPE_CODE[dtype],
                                   lib.MODE_CODE[mode], lib.NAN_CODE["equal"], [rows, cols], [pitch, 1],
                                   [pitch, 1], 1e-3, 1e-3, k, 0))
    res = torch.empty(len(segs) * SEG_RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    ws_size = lib.diff_nd_workspace_bytes(len(segs))
    ws = torch.empty(ws_size, dtype=torch.uint8, device="cuda")
    lib.diff_segments_nd(segs, res.data_ptr(), len(segs), ws.data_ptr(), ws_size)
    torch.cuda.synchronize()
    raw = res.cpu().numpy().view(SEG_RESULT_DTYPE)
    got_nd = [{f: raw[f][k].item() for f in SEG_RESULT_DTYPE.names} for k in range(len(segs))]
    assert_results_equal(got_nd, want, f"{dtype} narrow N-D")


def test_fill_element_aligned_bases():
    """Allocations that start at every element-aligned phase of a 16-byte
    block (the fill then goes byte by byte): every allocation byte equals the
    oracle's fill, the bytes between allocations are never written, and the
    guard check and the diff over those allocations match the oracle."""
    specs = []
    for dt in ("f32", "bf16", "f16", "fp8e4m3", "i32", "i64", "u8"):
        es = ESIZE[dt]
        for phase in range(es, 16, es):
            specs.append((dt, phase))
    allocs, offsets, inj = [], [], []
    dists = {"f32": ("normal", {}), "bf16": ("boundary", dict(p0=0.2, p1=3.0)), "f16": ("normal", {}),
             "fp8e4m3": ("normal", dict(p1=50.0)), "i32": ("uniform_int", dict(i0=-9, i1=1000)),
             "i64": ("bits", {}), "u8": ("bits", {})}
    for k, (dt, phase) in enumerate(specs):
        es = ESIZE[dt]
        rows = 1 + k % 4
        cols = 5 + 3 * k % 37
        stride = cols + (k % 3)
        glo = es * (k % 5)
        ghi = 3 * (k % 4)
        dist, kw = dists[dt]
        allocs.append(Alloc(k, dt, rows, cols, stride, glo, ghi, dist, **kw))
        offsets.append(2048 * k + phase)
        inj.append(Injection(k, "flip_bit", arg=-1, rate=0.3))
        if ghi:
            inj.append(Injection(k, "guard_write_hi", arg=1, index=ghi - 1))
    compares = [Compare(k, "tolerance" if a.dtype in ("f32", "bf16", "f16", "fp8e4m3") else "bitwise",
                        "equal", 1e-3, 1e-3) for k, a in enumerate(allocs)]
    w = Workload("phases", "", 0x5EED, allocs, inj, compares, offsets=offsets, arena_bytes=2048 * len(specs))
    assert all(offsets[k] + a.total_bytes <= 2048 * (k + 1) for k, a in enumerate(allocs))
    log(f"[phases] {len(allocs)} allocations")
    st = DeviceState(w)
    st.ref.fill_(0xA5)
    st.cand.fill_(0xA5)
    st.fill("ref", 0)
    st.fill("cand", 3)
    st.diff()
    st.guard()
    torch.cuda.synchronize()
    P = oracle.Prepared(w)
    for side, v in (("ref", 0), ("cand", 3)):
        want = np.full(w.arena_bytes, 0xA5, dtype=np.uint8)
        for k, a in enumerate(allocs):
            want[offsets[k]:offsets[k] + a.total_bytes] = P.fill_alloc(k, v)
        assert_bytes_equal(st.arena_host(side), want, f"phases {side}")
    cand, ref = st.arena_host("cand"), st.arena_host("ref")
    from oracle import diff_workload, guard_workload
    assert_results_equal(st.seg_results(), diff_workload(w, cand, ref), "phases diff")
    assert_results_equal(st.guard_results(), guard_workload(w, cand), "phases guards")
