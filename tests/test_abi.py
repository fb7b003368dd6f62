"""CPU-side checks of the C ABI: the shared library loads, exports every
function include/asmevo.h declares, the ctypes structures of the binding have
the header's layout (checked by compiling the header with gcc), and argument
errors are reported before anything touches the GPU."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2608_20711_amd as lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "asmevo.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(asmevo_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    L = lib.lib()
    declared = _declared_functions()
    assert declared == sorted(lib.EXPORTED)
    for name in declared:
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", lib.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    for name in declared:
        assert re.search(rf"\bT {name}\b", out), f"{name} not exported"


def test_struct_layouts_match_header(tmp_path):
    src = tmp_path / "layout.c"
    fields = {
        "asmevo_alloc": lib.Alloc, "asmevo_injection": lib.Injection, "asmevo_segment": lib.Segment,
        "asmevo_segment_result": lib.SegmentResult, "asmevo_guard_result": lib.GuardResult,
        "asmevo_cosine_result": lib.CosineResult, "asmevo_region": lib.Region,
        "asmevo_segment_nd": lib.SegmentND, "asmevo_plan": lib.Plan,
    }
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "asmevo.h"', "int main(void) {"]
    for cname, cls in fields.items():
        lines.append(f'  printf("{cname} %zu\\n", sizeof({cname}));')
        for f, _ in cls._fields_:
            lines.append(f'  printf("{cname}.{f} %zu\\n", offsetof({cname}, {f}));')
    lines += ["  return 0;", "}"]
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Werror", "-I", os.path.dirname(HEADER), str(src), "-o",
                    str(exe)], check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True,
                                                 check=True).stdout.splitlines())
    for cname, cls in fields.items():
        assert int(got[cname]) == ctypes.sizeof(cls), cname
        for f, _ in cls._fields_:
            assert int(got[f"{cname}.{f}"]) == getattr(cls, f).offset, f"{cname}.{f}"
    assert ctypes.sizeof(lib.SegmentResult) == 56
    assert ctypes.sizeof(lib.GuardResult) == 48
    assert ctypes.sizeof(lib.SegmentND) == 256


def test_version_status_strings_workspace():
    L = lib.lib()
    assert L.asmevo_abi_version() == 2
    for st in (lib.OK, lib.E_INVALID, lib.E_UNSUPPORTED, lib.E_WORKSPACE, lib.E_HIP):
        assert L.asmevo_status_string(st)
    assert lib.workspace_bytes(4096, 0) >= 4096 * 128
    assert lib.workspace_bytes(0, 0) > 0


def _seg(**kw):
    d = dict(a=0x10000, b=0x20000, dtype=lib.F32, mode=lib.TOLERANCE, nan_policy=0, reserved=0,
             rows=1, cols=8, stride_a=8, stride_b=8, atol=0.0, rtol=0.0)
    d.update(kw)
    return lib.Segment(**d)


@pytest.mark.parametrize("bad", [
    dict(dtype=99), dict(mode=7), dict(nan_policy=3), dict(rows=-1), dict(cols=-2),
    dict(stride_a=4), dict(stride_b=7), dict(a=0), dict(b=0), dict(a=0x10001), dict(b=0x20002),
    dict(dtype=lib.I32, mode=lib.TOLERANCE), dict(atol=-1.0), dict(rtol=float("nan")),
    dict(atol=float("inf")),
])
def test_diff_argument_errors_before_any_device_work(bad):
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_segments([_seg(**bad)], 0x40000, 0x50000, 1 << 20, stream=0)
    assert e.value.status == lib.E_INVALID


def test_diff_null_results_and_workspace():
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_segments([_seg()], 0, 0x50000, 1 << 20, stream=0)
    assert e.value.status == lib.E_INVALID
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_segments([_seg()], 0x40000, 0x50000, 16, stream=0)
    assert e.value.status == lib.E_WORKSPACE
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_segments([_seg()], 0x40000, 0, 1 << 20, stream=0)
    assert e.value.status == lib.E_WORKSPACE


def _alloc(**kw):
    d = dict(base=0x100000, rows=1, cols=64, stride=64, guard_lo=16, guard_hi=16, dtype=lib.F32,
             alloc_id=0, dist=lib.DIST_NORMAL, flags=0, p0=0.0, p1=1.0, i0=0, i1=0)
    d.update(kw)
    return lib.Alloc(**d)


def _inj(**kw):
    d = dict(alloc=0, kind=lib.INJ_FLIP_BIT, sides=0, arg=0, index=0, atol=0.0, rtol=0.0)
    d.update(kw)
    return lib.Injection(**d)


@pytest.mark.parametrize("allocs,inj,status", [
    ([_alloc(base=0x100002)], [], lib.E_INVALID),                         # not element-aligned (f32)
    ([_alloc(base=0)], [], lib.E_INVALID),
    ([_alloc(dtype=0)], [], lib.E_INVALID),
    ([_alloc(stride=10)], [], lib.E_INVALID),
    ([_alloc(guard_lo=6)], [], lib.E_INVALID),                            # not a multiple of 4
    ([_alloc(dist=9)], [], lib.E_INVALID),
    ([_alloc(dtype=lib.I32)], [], lib.E_INVALID),                         # normal on an integer dtype
    ([_alloc(dist=lib.DIST_UNIFORM_INT, i0=5, i1=5)], [], lib.E_INVALID),
    ([_alloc(dist=lib.DIST_UNIFORM_INT, i0=0, i1=(1 << 32) + 1)], [], lib.E_INVALID),
    ([_alloc(p1=float("inf"))], [], lib.E_INVALID),
    ([_alloc(flags=2)], [], lib.E_INVALID),
    ([_alloc(), _alloc(base=0x100100, alloc_id=1)], [], lib.E_INVALID),   # overlapping allocations
    ([_alloc()], [_inj(alloc=1)], lib.E_INVALID),
    ([_alloc()], [_inj(kind=9)], lib.E_INVALID),
    ([_alloc()], [_inj(index=64)], lib.E_INVALID),
    ([_alloc()], [_inj(arg=32)], lib.E_INVALID),
    ([_alloc()], [_inj(kind=lib.INJ_GUARD_WRITE_LO, index=10, arg=7)], lib.E_INVALID),
    ([_alloc()], [_inj(kind=lib.INJ_GUARD_WRITE_HI | lib.INJ_RATE, index=1)], lib.E_INVALID),
    ([_alloc()], [_inj(kind=lib.INJ_FLIP_BIT | lib.INJ_RATE, index=(1 << 32) + 1)], lib.E_INVALID),
    ([_alloc(dtype=lib.I32, dist=lib.DIST_UNIFORM_INT, i1=9)], [_inj(kind=lib.INJ_SET_NAN)], lib.E_INVALID),
    ([_alloc(dtype=lib.FP8_E4M3)], [_inj(kind=lib.INJ_SET_INF)], lib.E_UNSUPPORTED),
    ([_alloc()], [_inj(kind=lib.INJ_SET_BEYOND, atol=-1.0)], lib.E_INVALID),
    ([_alloc()], [_inj(sides=2)], lib.E_INVALID),
    ([_alloc()], [_inj(kind=lib.INJ_FLIP_BIT | lib.INJ_RATE, index=10)] * 17, lib.E_UNSUPPORTED),
    ([_alloc(dist=lib.DIST_BOUNDARY, p0=1.5)], [], lib.E_INVALID),        # rate above 1
    ([_alloc(dist=lib.DIST_BOUNDARY, p0=float("nan"))], [], lib.E_INVALID),
    ([_alloc(dist=lib.DIST_BOUNDARY, p0=0.1, p1=float("inf"))], [], lib.E_INVALID),
    ([_alloc()], [_inj(kind=lib.INJ_PAD_WRITE, index=0, arg=1)], lib.E_INVALID),   # one row: no padding
    ([_alloc(rows=3, cols=10, stride=12)], [_inj(kind=lib.INJ_PAD_WRITE, index=36, arg=1)],
     lib.E_INVALID),                                                      # a data byte of row 0
    ([_alloc(rows=3, cols=10, stride=12)], [_inj(kind=lib.INJ_PAD_WRITE, index=40, arg=9)],
     lib.E_INVALID),                                                      # runs into row 1
    ([_alloc(rows=3, cols=10, stride=12)], [_inj(kind=lib.INJ_PAD_WRITE, index=2 * 48 + 40, arg=1)],
     lib.E_INVALID),                                                      # the last row has no padding
    ([_alloc(rows=3, cols=10, stride=12)], [_inj(kind=lib.INJ_PAD_WRITE | lib.INJ_RATE, index=40, arg=1)],
     lib.E_INVALID),
])
def test_fill_argument_errors_before_any_device_work(allocs, inj, status):
    with pytest.raises(lib.AsmevoError) as e:
        lib.fill_guarded(allocs, inj, 1, 1, 0x900000, 1 << 20, stream=0)
    assert e.value.status == status


def test_fill_variant_range_and_workspace():
    with pytest.raises(lib.AsmevoError) as e:
        lib.fill_guarded([_alloc()], [], 1, 1 << 16, 0x900000, 1 << 20, stream=0)
    assert e.value.status == lib.E_INVALID
    with pytest.raises(lib.AsmevoError) as e:
        lib.fill_guarded([_alloc()], [], 1, 0, 0x900000, 8, stream=0)
    assert e.value.status == lib.E_WORKSPACE


def test_guard_argument_errors():
    with pytest.raises(lib.AsmevoError) as e:
        lib.guard_check([_alloc(stride=3)], 1, 0x40000, 0x50000, 1 << 20, stream=0)
    assert e.value.status == lib.E_INVALID
    with pytest.raises(lib.AsmevoError) as e:
        lib.guard_check([_alloc()], 1, 0, 0x50000, 1 << 20, stream=0)
    assert e.value.status == lib.E_INVALID
    with pytest.raises(lib.AsmevoError) as e:
        lib.guard_check([_alloc()], 1, 0x40000, 0x50000, 4, stream=0)
    assert e.value.status == lib.E_WORKSPACE


def test_cosine_workspace_and_errors():
    L = lib.lib()
    segs = (lib.Segment * 2)(_seg(), _seg(rows=3, cols=1000, stride_a=1024, stride_b=1024))
    need = L.asmevo_diff_cosine_workspace_bytes(segs, 2)
    # descriptors + counters + a 32-byte record per 4096-byte block (1 + 3 blocks)
    assert need >= 2 * 128 + 2 * 8 + 4 * 32
    bad = (lib.Segment * 1)(_seg(dtype=99))
    assert L.asmevo_diff_cosine_workspace_bytes(bad, 1) == 0
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_cosine([_seg()], 0x40000, 0x48000, 0x50000, 16, stream=0)
    assert e.value.status == lib.E_WORKSPACE
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_cosine([_seg()], 0x40000, 0, 0x50000, 1 << 20, stream=0)
    assert e.value.status == lib.E_INVALID


@pytest.mark.parametrize("regions", [
    [(0x1000, 0, 16)],                                   # null source
    [(0x1000, 0x2000, 1 << 53)],                         # too large
    [(0x1000, 0x1008, 64)],                              # source and destination overlap
    [(0x1000, 0x9000, 64), (0x1020, 0xA000, 64)],        # destinations overlap
    [(0x1000, 0x9000, 64), (0x9000, 0xB000, 64)],        # a destination overlaps another source
])
def test_copy_regions_argument_errors(regions):
    with pytest.raises(lib.AsmevoError) as e:
        lib.copy_regions([lib.Region(d, s, n) for d, s, n in regions], 0x50000, 1 << 20, stream=0)
    assert e.value.status == lib.E_INVALID


def test_copy_regions_workspace():
    with pytest.raises(lib.AsmevoError) as e:
        lib.copy_regions([lib.Region(0x1000, 0x9000, 64)], 0x50000, 8, stream=0)
    assert e.value.status == lib.E_WORKSPACE


def test_diff_cosine_nd_argument_errors():
    """Segments of one result must be consecutive and of one element type;
    both are checked before anything is enqueued."""
    def seg(result, dtype=lib.F32, a=0x10000):
        return _seg_nd(a=a, b=a + 0x100000, dtype=dtype, result=result)
    L = lib.lib()
    for segs, n_res, status in (
            ([seg(0), seg(1), seg(0)], 2, lib.E_UNSUPPORTED),                 # result 0 not consecutive
            ([seg(0), seg(0, dtype=lib.F16)], 1, lib.E_UNSUPPORTED),          # two element types
            ([seg(1)], 1, lib.E_INVALID),                                      # result slot out of range
            ([seg(0)], -1, lib.E_INVALID)):
        arr = lib.descriptor_array(segs)
        assert lib.diff_cosine_nd_workspace_bytes(arr, n_res) == 0
        assert L.asmevo_diff_cosine_nd(arr, len(segs), 0x1000, n_res, 0x2000, 0x3000, 1 << 30, None) == status
    arr = lib.descriptor_array([seg(0), seg(0), seg(1)])
    assert lib.diff_cosine_nd_workspace_bytes(arr, 2) > 0
    assert L.asmevo_diff_cosine_nd(arr, 3, 0x1000, 2, 0x2000, 0x3000, 8, None) == lib.E_WORKSPACE


def test_va_argument_errors():
    L = lib.lib()
    out = ctypes.c_uint64(0)
    assert L.asmevo_va_alloc(0, 0, ctypes.byref(out)) == lib.E_INVALID          # zero bytes
    assert L.asmevo_va_alloc(0, 1 << 21, None) == lib.E_INVALID                 # no output
    assert L.asmevo_va_free(0x7000_0000_0000) == lib.E_INVALID                  # not a live range
    assert out.value == 0
    assert lib.va_granularity() >= 0
    with pytest.raises(lib.AsmevoError) as e:
        lib.va_free(0x1000)
    assert e.value.status == lib.E_INVALID


def _seg_nd(shape=(4, 8), sa=(8, 1), sb=(8, 1), **kw):
    d = dict(a=0x10000, b=0x20000, dtype=lib.F32, mode=lib.TOLERANCE, nan_policy=0, shape=shape,
             stride_a=sa, stride_b=sb)
    d.update(kw)
    return lib.segment_nd(**d)


@pytest.mark.parametrize("seg,n_results", [
    (_seg_nd(dtype=99), 1), (_seg_nd(mode=5), 1), (_seg_nd(nan_policy=2), 1),
    (_seg_nd(result=1), 1),                                       # result slot out of range
    (_seg_nd(shape=(4, -1), sa=(8, 1), sb=(8, 1)), 1),
    (_seg_nd(sa=(8, -1)), 1),
    (_seg_nd(index_base=-5), 1),
    (_seg_nd(a=0x10002), 1),                                      # misaligned
    (_seg_nd(b=0), 1),
    (_seg_nd(shape=(1 << 40, 1 << 20), sa=(1 << 20, 1), sb=(1 << 20, 1)), 1),   # beyond 2^52 bytes
    (_seg_nd(dtype=lib.U8, mode=lib.TOLERANCE), 1),
    (_seg_nd(atol=-1.0), 1),
])
def test_diff_nd_argument_errors(seg, n_results):
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_segments_nd([seg], 0x40000, n_results, 0x50000, 1 << 20, stream=0)
    assert e.value.status == lib.E_INVALID


def test_diff_nd_ndim_and_workspace():
    seg = _seg_nd()
    seg.ndim = 9
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_segments_nd([seg], 0x40000, 1, 0x50000, 1 << 20, stream=0)
    assert e.value.status == lib.E_INVALID
    need = lib.diff_nd_workspace_bytes(3)
    assert need >= 3 * (128 + 200)
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_segments_nd([_seg_nd()] * 3, 0x40000, 1, 0x50000, 3 * 128, stream=0)
    assert e.value.status == lib.E_WORKSPACE
    with pytest.raises(lib.AsmevoError) as e:
        lib.diff_segments_nd([_seg_nd()], 0, 1, 0x50000, need, stream=0)
    assert e.value.status == lib.E_INVALID


def test_noalloc_diff_argument_errors():
    """The allocation-free diff validates before touching the GPU: more
    segments than its static table holds, a null result pointer, a negative
    count and malformed segments are refused."""
    L = lib.lib()
    n = lib.NOALLOC_MAX_SEGMENTS + 1
    arr = (lib.Segment * n)(*[_seg()] * n)
    assert L.asmevo_diff_segments_noalloc(arr, n, 0x1000, None) == lib.E_CAPACITY
    assert L.asmevo_diff_segments_noalloc(arr, 1, None, None) == lib.E_INVALID
    assert L.asmevo_diff_segments_noalloc(arr, -1, 0x1000, None) == lib.E_INVALID
    bad = (lib.Segment * 1)(_seg(stride_a=1, cols=5))
    assert L.asmevo_diff_segments_noalloc(bad, 1, 0x1000, None) == lib.E_INVALID
    assert L.asmevo_diff_segments_noalloc(arr, 0, 0x1000, None) == lib.OK
    assert b"static" in L.asmevo_status_string(lib.E_CAPACITY)


def test_plan_argument_errors_before_any_device_work():
    """Plans validate like the unplanned calls, before anything is enqueued;
    a planned launch refuses a null or mismatched plan."""
    L = lib.lib()
    plan = lib.Plan()
    bad = (lib.Segment * 1)(_seg(stride_a=1, cols=5))
    assert L.asmevo_plan_diff(bad, 1, 0x40000, 1 << 20, None, ctypes.byref(plan)) == lib.E_INVALID
    good = (lib.Segment * 1)(_seg())
    assert L.asmevo_plan_diff(good, 1, 0x40000, 1 << 20, None, None) == lib.E_INVALID
    assert L.asmevo_plan_diff(good, 1, 0x40000, 8, None, ctypes.byref(plan)) == lib.E_WORKSPACE
    assert L.asmevo_plan_diff(good, 1, None, 1 << 20, None, ctypes.byref(plan)) == lib.E_WORKSPACE
    allocs = (lib.Alloc * 1)(_alloc(stride=10))
    assert L.asmevo_plan_guard(allocs, 1, 0x40000, 1 << 20, None, ctypes.byref(plan)) == lib.E_INVALID
    assert L.asmevo_diff_planned(None, 0x1000, None) == lib.E_INVALID
    p = lib.Plan(0x40000, 4, 1, 1, lib.PLAN_GUARD, 256)
    assert L.asmevo_diff_planned(ctypes.byref(p), 0x1000, None) == lib.E_INVALID       # a guard plan
    p = lib.Plan(0x40000, 4, 1, 1, lib.PLAN_DIFF, 256)
    assert L.asmevo_guard_planned(ctypes.byref(p), 1, 0x1000, None) == lib.E_INVALID   # a diff plan
    assert L.asmevo_diff_planned(ctypes.byref(p), None, None) == lib.E_INVALID
    empty = lib.Plan(0, 0, 0, 0, lib.PLAN_DIFF, 0)
    assert L.asmevo_diff_planned(ctypes.byref(empty), None, None) == lib.OK
    assert L.asmevo_plan_bytes(4096) >= 4096 * (128 + 328) and L.asmevo_plan_bytes(100) >= 300 * 64
    nd = (lib.SegmentND * 1)(_seg_nd(index_base=-5))
    assert L.asmevo_plan_diff_nd(nd, 1, 1, 0x40000, 1 << 20, None, ctypes.byref(plan)) == lib.E_INVALID
    nd = (lib.SegmentND * 1)(_seg_nd())
    assert L.asmevo_plan_diff_nd(nd, 1, 1, 0x40000, 8, None, ctypes.byref(plan)) == lib.E_WORKSPACE
    p = lib.Plan(0x40000, 4, 1, 0, lib.PLAN_DIFF_ND, 256)
    assert L.asmevo_diff_planned(ctypes.byref(p), None, None) == lib.OK               # no results: nothing to do
    p = lib.Plan(0x40000, 4, 1, 2, lib.PLAN_DIFF_ND, 256)
    assert L.asmevo_diff_planned(ctypes.byref(p), None, None) == lib.E_INVALID
    p = lib.Plan(0x40000, 4, 1, 1, 9, 256)
    assert L.asmevo_diff_planned(ctypes.byref(p), 0x1000, None) == lib.E_INVALID      # unknown kind


def test_workspace_must_be_256_byte_aligned():
    """Workspaces start on a 256-byte boundary (kernels keep 64-bit atomic
    counters there): a misaligned one is refused before anything is enqueued."""
    L = lib.lib()
    segs = (lib.Segment * 1)(_seg())
    assert L.asmevo_diff_segments(segs, 1, 0x1000, 0x40008, 1 << 20, None) == lib.E_INVALID
    plan = lib.Plan()
    assert L.asmevo_plan_diff(segs, 1, 0x40010, 1 << 20, None, ctypes.byref(plan)) == lib.E_INVALID
    allocs = (lib.Alloc * 1)(_alloc())
    assert L.asmevo_plan_guard(allocs, 1, 0x40104, 1 << 20, None, ctypes.byref(plan)) == lib.E_INVALID
    assert L.asmevo_guard_check(allocs, 1, 7, 0x1000, 0x40040, 1 << 20, None) == lib.E_INVALID
    assert L.asmevo_diff_cosine(segs, 1, 0x1000, 0x2000, 0x40080, 1 << 20, None) == lib.E_INVALID
