"""MI355X differential-oracle library: thin Python binding over libasmevo.so.

The binding only marshals arguments (ctypes structures mirroring
include/asmevo.h, device addresses from torch tensors, the current HIP
stream); every step of the fill, comparison and guard check runs in the HIP
kernels of the shared library.  Importing fails loudly if the library has
not been built (`python -m paper_2608_20711_amd.build` or
`__graft_entry__.build()`): there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

PKG = os.path.dirname(os.path.abspath(__file__))
# ASMEVO_LIBRARY may point at another build of the same library (tuning runs)
LIB_PATH = os.environ.get("ASMEVO_LIBRARY") or os.path.join(PKG, "libasmevo.so")

# codes of include/asmevo.h
OK, E_INVALID, E_UNSUPPORTED, E_WORKSPACE, E_HIP, E_CAPACITY = 0, -1, -2, -3, -4, -5
NOALLOC_MAX_SEGMENTS = 4096
F32, BF16, F16, FP8_E4M3, I32, I64, U8 = 1, 2, 3, 4, 5, 6, 7
BITWISE, TOLERANCE = 0, 1
NAN_EQUAL, NAN_STRICT = 0, 1
DIST_NORMAL, DIST_UNIFORM_INT, DIST_BITS, DIST_CONST, DIST_BOUNDARY = 0, 1, 2, 3, 4
FILL_SATURATE = 1
INJ_FLIP_BIT, INJ_STEP_WITHIN, INJ_SET_BEYOND, INJ_SET_NAN, INJ_SET_INF = 1, 2, 3, 4, 5
INJ_GUARD_WRITE_LO, INJ_GUARD_WRITE_HI, INJ_PAD_WRITE = 6, 7, 8
INJ_RATE = 0x100
SIDE_CANDIDATE, SIDE_BOTH = 0, 1

DTYPE_CODE = {"f32": F32, "bf16": BF16, "f16": F16, "fp8e4m3": FP8_E4M3, "i32": I32, "i64": I64, "u8": U8}
MODE_CODE = {"bitwise": BITWISE, "tolerance": TOLERANCE}
NAN_CODE = {"equal": NAN_EQUAL, "strict": NAN_STRICT}
DIST_CODE = {"normal": DIST_NORMAL, "uniform_int": DIST_UNIFORM_INT, "bits": DIST_BITS, "const": DIST_CONST,
             "boundary": DIST_BOUNDARY}
KIND_CODE = {"flip_bit": INJ_FLIP_BIT, "step_within": INJ_STEP_WITHIN, "set_beyond": INJ_SET_BEYOND,
             "set_nan": INJ_SET_NAN, "set_inf": INJ_SET_INF, "guard_write_lo": INJ_GUARD_WRITE_LO,
             "guard_write_hi": INJ_GUARD_WRITE_HI, "pad_write": INJ_PAD_WRITE}
SIDE_CODE = {"candidate": SIDE_CANDIDATE, "both": SIDE_BOTH}


class Alloc(ctypes.Structure):
    _fields_ = [("base", ctypes.c_uint64), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("stride", ctypes.c_int64), ("guard_lo", ctypes.c_int64), ("guard_hi", ctypes.c_int64),
                ("dtype", ctypes.c_uint32), ("alloc_id", ctypes.c_uint32),
                ("dist", ctypes.c_uint32), ("flags", ctypes.c_uint32),
                ("p0", ctypes.c_double), ("p1", ctypes.c_double),
                ("i0", ctypes.c_int64), ("i1", ctypes.c_int64)]


class Injection(ctypes.Structure):
    _fields_ = [("alloc", ctypes.c_uint32), ("kind", ctypes.c_uint32), ("sides", ctypes.c_uint32),
                ("arg", ctypes.c_uint32), ("index", ctypes.c_int64),
                ("atol", ctypes.c_double), ("rtol", ctypes.c_double)]


class Segment(ctypes.Structure):
    _fields_ = [("a", ctypes.c_uint64), ("b", ctypes.c_uint64),
                ("dtype", ctypes.c_uint32), ("mode", ctypes.c_uint32),
                ("nan_policy", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("stride_a", ctypes.c_int64), ("stride_b", ctypes.c_int64),
                ("atol", ctypes.c_double), ("rtol", ctypes.c_double)]


MAX_DIMS = 8


class SegmentND(ctypes.Structure):
    _fields_ = [("a", ctypes.c_uint64), ("b", ctypes.c_uint64),
                ("dtype", ctypes.c_uint32), ("mode", ctypes.c_uint32),
                ("nan_policy", ctypes.c_uint32), ("ndim", ctypes.c_uint32),
                ("result", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("index_base", ctypes.c_int64),
                ("shape", ctypes.c_int64 * MAX_DIMS),
                ("stride_a", ctypes.c_int64 * MAX_DIMS), ("stride_b", ctypes.c_int64 * MAX_DIMS),
                ("atol", ctypes.c_double), ("rtol", ctypes.c_double)]


def segment_nd(a: int, b: int, dtype: int, mode: int, nan_policy: int, shape: Sequence[int],
               stride_a: Sequence[int], stride_b: Sequence[int], atol: float = 0.0, rtol: float = 0.0,
               result: int = 0, index_base: int = 0) -> SegmentND:
    nd = len(shape)
    if nd > MAX_DIMS or len(stride_a) != nd or len(stride_b) != nd:
        raise ValueError("shape and strides must have the same length, at most 8")
    arr = ctypes.c_int64 * MAX_DIMS
    return SegmentND(a, b, dtype, mode, nan_policy, nd, result, 0, index_base, arr(*shape), arr(*stride_a),
                     arr(*stride_b), atol, rtol)


class SegmentResult(ctypes.Structure):
    _fields_ = [("mismatches", ctypes.c_uint64), ("first_mismatch", ctypes.c_int64),
                ("bitwise_mismatches", ctypes.c_uint64), ("first_bitwise", ctypes.c_int64),
                ("nonfinite_mismatches", ctypes.c_uint64),
                ("max_abs", ctypes.c_double), ("max_rel", ctypes.c_double)]


class CosineResult(ctypes.Structure):
    _fields_ = [("sum_ab", ctypes.c_double), ("sum_aa", ctypes.c_double), ("sum_bb", ctypes.c_double),
                ("cosine", ctypes.c_double), ("pairs", ctypes.c_uint64), ("blocks", ctypes.c_uint64)]


class Region(ctypes.Structure):
    _fields_ = [("dst", ctypes.c_uint64), ("src", ctypes.c_uint64), ("bytes", ctypes.c_uint64)]


class GuardResult(ctypes.Structure):
    _fields_ = [("bad_lo", ctypes.c_uint64), ("bad_hi", ctypes.c_uint64),
                ("first_bad_lo", ctypes.c_int64), ("first_bad_hi", ctypes.c_int64),
                ("bad_pad", ctypes.c_uint64), ("first_bad_pad", ctypes.c_int64)]


class Plan(ctypes.Structure):
    _fields_ = [("table", ctypes.c_uint64), ("units", ctypes.c_uint64), ("n", ctypes.c_int32),
                ("n_results", ctypes.c_int32), ("kind", ctypes.c_int32), ("workgroups", ctypes.c_int32)]


PLAN_DIFF, PLAN_GUARD, PLAN_DIFF_ND = 1, 2, 3


class Kernel(ctypes.Structure):
    _fields_ = [("module", ctypes.c_uint64), ("function", ctypes.c_uint64), ("num_regs", ctypes.c_int32),
                ("shared_bytes", ctypes.c_int32), ("max_threads", ctypes.c_int32), ("local_bytes", ctypes.c_int32)]


SEGMENT_RESULT_FIELDS = [f for f, _ in SegmentResult._fields_]
GUARD_RESULT_FIELDS = [f for f, _ in GuardResult._fields_]

EXPORTED = ["asmevo_fill_guarded", "asmevo_diff_segments", "asmevo_diff_segments_ex",
            "asmevo_diff_cosine", "asmevo_diff_cosine_workspace_bytes", "asmevo_copy_regions",
            "asmevo_guard_check", "asmevo_workspace_bytes", "asmevo_status_string",
            "asmevo_abi_version", "asmevo_last_hip_error", "asmevo_diff_segments_nd",
            "asmevo_diff_nd_workspace_bytes", "asmevo_kernel_load", "asmevo_kernel_unload",
            "asmevo_kernel_launch", "asmevo_kernel_time", "asmevo_va_granularity", "asmevo_va_alloc",
            "asmevo_va_free", "asmevo_diff_cosine_nd", "asmevo_diff_cosine_nd_workspace_bytes",
            "asmevo_diff_segments_noalloc", "asmevo_plan_bytes", "asmevo_plan_diff", "asmevo_diff_planned",
            "asmevo_plan_guard", "asmevo_guard_planned", "asmevo_plan_diff_nd"]


class AsmevoError(RuntimeError):
    def __init__(self, status: int, call: str):
        self.status = status
        msg = _lib().asmevo_status_string(status).decode()
        if status == E_HIP:
            msg += f" (hipError {_lib().asmevo_last_hip_error()})"
        super().__init__(f"{call}: {msg} [{status}]")


_handle: Optional[ctypes.CDLL] = None


def _lib() -> ctypes.CDLL:
    global _handle
    if _handle is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it first (python -m paper_2608_20711_amd.build)")
        # torch first: it loads the HIP runtime its tensors and streams live
        # in, and the library must then run on that same runtime (loaded the
        # other way round, torch found no GPU in a fresh process)
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        vp, P = ctypes.c_void_p, ctypes.POINTER
        L.asmevo_fill_guarded.argtypes = [P(Alloc), ctypes.c_int32, P(Injection), ctypes.c_int64,
                                          ctypes.c_uint64, ctypes.c_uint32, vp, ctypes.c_size_t, vp]
        L.asmevo_fill_guarded.restype = ctypes.c_int32
        L.asmevo_diff_segments.argtypes = [P(Segment), ctypes.c_int32, vp, vp, ctypes.c_size_t, vp]
        L.asmevo_diff_segments.restype = ctypes.c_int32
        L.asmevo_diff_segments_ex.argtypes = [P(Segment), ctypes.c_int32, vp, vp, ctypes.c_size_t, vp,
                                              ctypes.c_int32]
        L.asmevo_diff_segments_ex.restype = ctypes.c_int32
        L.asmevo_diff_segments_noalloc.argtypes = [P(Segment), ctypes.c_int32, vp, vp]
        L.asmevo_diff_segments_noalloc.restype = ctypes.c_int32
        L.asmevo_plan_bytes.argtypes = [ctypes.c_int32]
        L.asmevo_plan_bytes.restype = ctypes.c_size_t
        L.asmevo_plan_diff.argtypes = [P(Segment), ctypes.c_int32, vp, ctypes.c_size_t, vp, P(Plan)]
        L.asmevo_plan_diff.restype = ctypes.c_int32
        L.asmevo_plan_diff_nd.argtypes = [P(SegmentND), ctypes.c_int32, ctypes.c_int32, vp, ctypes.c_size_t, vp,
                                          P(Plan)]
        L.asmevo_plan_diff_nd.restype = ctypes.c_int32
        L.asmevo_diff_planned.argtypes = [P(Plan), vp, vp]
        L.asmevo_diff_planned.restype = ctypes.c_int32
        L.asmevo_plan_guard.argtypes = [P(Alloc), ctypes.c_int32, vp, ctypes.c_size_t, vp, P(Plan)]
        L.asmevo_plan_guard.restype = ctypes.c_int32
        L.asmevo_guard_planned.argtypes = [P(Plan), ctypes.c_uint64, vp, vp]
        L.asmevo_guard_planned.restype = ctypes.c_int32
        L.asmevo_diff_cosine.argtypes = [P(Segment), ctypes.c_int32, vp, vp, vp, ctypes.c_size_t, vp]
        L.asmevo_diff_cosine.restype = ctypes.c_int32
        L.asmevo_diff_segments_nd.argtypes = [P(SegmentND), ctypes.c_int32, vp, ctypes.c_int32, vp,
                                              ctypes.c_size_t, vp]
        L.asmevo_diff_segments_nd.restype = ctypes.c_int32
        L.asmevo_diff_nd_workspace_bytes.argtypes = [ctypes.c_int32]
        L.asmevo_diff_nd_workspace_bytes.restype = ctypes.c_size_t
        L.asmevo_diff_cosine_workspace_bytes.argtypes = [P(Segment), ctypes.c_int32]
        L.asmevo_diff_cosine_workspace_bytes.restype = ctypes.c_size_t
        L.asmevo_copy_regions.argtypes = [P(Region), ctypes.c_int32, vp, ctypes.c_size_t, vp]
        L.asmevo_copy_regions.restype = ctypes.c_int32
        L.asmevo_guard_check.argtypes = [P(Alloc), ctypes.c_int32, ctypes.c_uint64, vp, vp,
                                         ctypes.c_size_t, vp]
        L.asmevo_guard_check.restype = ctypes.c_int32
        L.asmevo_workspace_bytes.argtypes = [ctypes.c_int32, ctypes.c_int64]
        L.asmevo_workspace_bytes.restype = ctypes.c_size_t
        L.asmevo_kernel_load.argtypes = [ctypes.c_char_p, ctypes.c_size_t, ctypes.c_char_p, P(Kernel)]
        L.asmevo_kernel_load.restype = ctypes.c_int32
        L.asmevo_kernel_unload.argtypes = [P(Kernel)]
        L.asmevo_kernel_unload.restype = ctypes.c_int32
        u3 = ctypes.c_uint32 * 3
        L.asmevo_kernel_launch.argtypes = [P(Kernel), u3, u3, ctypes.c_uint32, P(ctypes.c_void_p), vp]
        L.asmevo_kernel_launch.restype = ctypes.c_int32
        L.asmevo_kernel_time.argtypes = [P(Kernel), u3, u3, ctypes.c_uint32, P(ctypes.c_void_p), ctypes.c_int32,
                                         ctypes.c_int32, P(ctypes.c_float), vp]
        L.asmevo_kernel_time.restype = ctypes.c_int32
        L.asmevo_status_string.argtypes = [ctypes.c_int32]
        L.asmevo_status_string.restype = ctypes.c_char_p
        L.asmevo_abi_version.restype = ctypes.c_int32
        L.asmevo_last_hip_error.restype = ctypes.c_int32
        L.asmevo_diff_cosine_nd.argtypes = [P(SegmentND), ctypes.c_int32, vp, ctypes.c_int32, vp, vp,
                                            ctypes.c_size_t, vp]
        L.asmevo_diff_cosine_nd.restype = ctypes.c_int32
        L.asmevo_diff_cosine_nd_workspace_bytes.argtypes = [P(SegmentND), ctypes.c_int32, ctypes.c_int32]
        L.asmevo_diff_cosine_nd_workspace_bytes.restype = ctypes.c_size_t
        L.asmevo_va_granularity.argtypes = []
        L.asmevo_va_granularity.restype = ctypes.c_size_t
        L.asmevo_va_alloc.argtypes = [ctypes.c_uint64, ctypes.c_uint64, P(ctypes.c_uint64)]
        L.asmevo_va_alloc.restype = ctypes.c_int32
        L.asmevo_va_free.argtypes = [ctypes.c_uint64]
        L.asmevo_va_free.restype = ctypes.c_int32
        _handle = L
    return _handle


def lib() -> ctypes.CDLL:
    return _lib()


def _array(cls, items: Sequence):
    """A ctypes array of `cls` holding `items`; an array of `cls` built once by
    the caller (see descriptor_array) is passed through unchanged."""
    if isinstance(items, ctypes.Array) and items._type_ is cls:
        return items
    arr = (cls * max(1, len(items)))()
    for k, it in enumerate(items):
        arr[k] = it
    return arr


def descriptor_array(items: Sequence):
    """Packs descriptors (all of one struct type) into a ctypes array once, for
    callers that issue the same call many times."""
    if not items:
        raise ValueError("no descriptors")
    return _array(type(items[0]), items)


def _check(status: int, call: str):
    if status != OK:
        raise AsmevoError(status, call)


def workspace_bytes(n_descs: int, n_inj: int = 0) -> int:
    return int(_lib().asmevo_workspace_bytes(n_descs, n_inj))


def _stream_handle(stream) -> Optional[int]:
    """A torch stream / raw handle / None -> hipStream_t as an int (None = default)."""
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream or None
    if hasattr(stream, "cuda_stream"):
        return stream.cuda_stream or None
    return int(stream) or None


def fill_guarded(allocs: Sequence[Alloc], injections: Sequence[Injection], seed: int, variant: int,
                 workspace_ptr: int, workspace_size: int, stream=None) -> None:
    a = _array(Alloc, allocs)
    j = _array(Injection, injections)
    _check(_lib().asmevo_fill_guarded(a, len(allocs), j, len(injections), seed, variant,
                                      workspace_ptr, workspace_size, _stream_handle(stream)),
           "asmevo_fill_guarded")


def diff_segments(segments: Sequence[Segment], results_ptr: int, workspace_ptr: int,
                  workspace_size: int, stream=None, workgroups: int = 0) -> None:
    s = _array(Segment, segments)
    _check(_lib().asmevo_diff_segments_ex(s, len(segments), results_ptr, workspace_ptr,
                                          workspace_size, _stream_handle(stream), workgroups),
           "asmevo_diff_segments")


def diff_segments_noalloc(segments: Sequence[Segment], results_ptr: int, stream=None) -> None:
    """asmevo_diff_segments without a workspace (its table in the library's static device array)."""
    s = _array(Segment, segments)
    _check(_lib().asmevo_diff_segments_noalloc(s, len(segments), results_ptr, _stream_handle(stream)),
           "asmevo_diff_segments_noalloc")


def plan_bytes(n_descs: int) -> int:
    return int(_lib().asmevo_plan_bytes(n_descs))


def plan_diff(segments: Sequence[Segment], workspace_ptr: int, workspace_size: int, stream=None) -> Plan:
    """Stages the segments' descriptor table once (asmevo_plan_diff)."""
    plan = Plan()
    s = _array(Segment, segments)
    _check(_lib().asmevo_plan_diff(s, len(segments), workspace_ptr, workspace_size, _stream_handle(stream),
                                   ctypes.byref(plan)), "asmevo_plan_diff")
    return plan


def plan_diff_nd(segments: Sequence[SegmentND], n_results: int, workspace_ptr: int, workspace_size: int,
                 stream=None) -> Plan:
    """Stages N-D segments' descriptor table once (asmevo_plan_diff_nd)."""
    plan = Plan()
    s = _array(SegmentND, segments)
    _check(_lib().asmevo_plan_diff_nd(s, len(segments), n_results, workspace_ptr, workspace_size,
                                      _stream_handle(stream), ctypes.byref(plan)), "asmevo_plan_diff_nd")
    return plan


def diff_planned(plan: Plan, results_ptr: int, stream=None) -> None:
    _check(_lib().asmevo_diff_planned(ctypes.byref(plan), results_ptr, _stream_handle(stream)),
           "asmevo_diff_planned")


def plan_guard(allocs: Sequence[Alloc], workspace_ptr: int, workspace_size: int, stream=None) -> Plan:
    """Stages the guard regions of the allocations once (asmevo_plan_guard)."""
    plan = Plan()
    a = _array(Alloc, allocs)
    _check(_lib().asmevo_plan_guard(a, len(allocs), workspace_ptr, workspace_size, _stream_handle(stream),
                                    ctypes.byref(plan)), "asmevo_plan_guard")
    return plan


def guard_planned(plan: Plan, seed: int, results_ptr: int, stream=None) -> None:
    _check(_lib().asmevo_guard_planned(ctypes.byref(plan), seed, results_ptr, _stream_handle(stream)),
           "asmevo_guard_planned")


def diff_nd_workspace_bytes(n: int) -> int:
    return int(_lib().asmevo_diff_nd_workspace_bytes(n))


def diff_segments_nd(segments: Sequence[SegmentND], results_ptr: int, n_results: int, workspace_ptr: int,
                     workspace_size: int, stream=None) -> None:
    s = _array(SegmentND, segments)
    _check(_lib().asmevo_diff_segments_nd(s, len(segments), results_ptr, n_results, workspace_ptr,
                                          workspace_size, _stream_handle(stream)),
           "asmevo_diff_segments_nd")


def diff_cosine_workspace_bytes(segments: Sequence[Segment]) -> int:
    s = _array(Segment, segments)
    return int(_lib().asmevo_diff_cosine_workspace_bytes(s, len(segments)))


def diff_cosine(segments: Sequence[Segment], results_ptr: int, cos_results_ptr: int, workspace_ptr: int,
                workspace_size: int, stream=None) -> None:
    s = _array(Segment, segments)
    _check(_lib().asmevo_diff_cosine(s, len(segments), results_ptr, cos_results_ptr, workspace_ptr,
                                     workspace_size, _stream_handle(stream)),
           "asmevo_diff_cosine")


def copy_regions(regions: Sequence[Region], workspace_ptr: int, workspace_size: int, stream=None) -> None:
    r = _array(Region, regions)
    _check(_lib().asmevo_copy_regions(r, len(regions), workspace_ptr, workspace_size, _stream_handle(stream)),
           "asmevo_copy_regions")


def diff_cosine_nd_workspace_bytes(segments: Sequence[SegmentND], n_results: int) -> int:
    s = _array(SegmentND, segments)
    return int(_lib().asmevo_diff_cosine_nd_workspace_bytes(s, len(segments), n_results))


def diff_cosine_nd(segments: Sequence[SegmentND], results_ptr: int, n_results: int, cos_results_ptr: int,
                   workspace_ptr: int, workspace_size: int, stream=None) -> None:
    s = _array(SegmentND, segments)
    _check(_lib().asmevo_diff_cosine_nd(s, len(segments), results_ptr, n_results, cos_results_ptr, workspace_ptr,
                                        workspace_size, _stream_handle(stream)), "asmevo_diff_cosine_nd")


def va_granularity() -> int:
    """Size and address granularity of va_alloc on the current device (0: unsupported)."""
    return int(_lib().asmevo_va_granularity())


def va_alloc(nbytes: int, addr: int = 0) -> int:
    """Device memory mapped at `addr` (0: anywhere); returns its address."""
    out = ctypes.c_uint64(0)
    _check(_lib().asmevo_va_alloc(addr, nbytes, ctypes.byref(out)), "asmevo_va_alloc")
    return int(out.value)


def va_free(addr: int) -> None:
    _check(_lib().asmevo_va_free(addr), "asmevo_va_free")


def guard_check(allocs: Sequence[Alloc], seed: int, results_ptr: int, workspace_ptr: int,
                workspace_size: int, stream=None) -> None:
    a = _array(Alloc, allocs)
    _check(_lib().asmevo_guard_check(a, len(allocs), seed, results_ptr, workspace_ptr,
                                     workspace_size, _stream_handle(stream)),
           "asmevo_guard_check")


# --------------------------------------------------------------------------
# code objects under test
# --------------------------------------------------------------------------

def kernel_load(image: bytes, name: str) -> Kernel:
    k = Kernel()
    _check(_lib().asmevo_kernel_load(image, len(image), name.encode(), ctypes.byref(k)), "asmevo_kernel_load")
    return k


def kernel_unload(k: Kernel) -> None:
    _check(_lib().asmevo_kernel_unload(ctypes.byref(k)), "asmevo_kernel_unload")


class KernelArgs:
    """Explicit kernel arguments as ctypes values, kept alive with the
    pointer array the runtime reads."""

    def __init__(self, values: Sequence):
        self.values = list(values)
        self.params = (ctypes.c_void_p * max(1, len(self.values)))(
            *[ctypes.cast(ctypes.pointer(v), ctypes.c_void_p) for v in self.values])


def kernel_launch(k: Kernel, grid, block, args: KernelArgs, lds_bytes: int = 0, stream=None) -> None:
    u3 = ctypes.c_uint32 * 3
    _check(_lib().asmevo_kernel_launch(ctypes.byref(k), u3(*grid), u3(*block), lds_bytes, args.params,
                                       _stream_handle(stream)), "asmevo_kernel_launch")


def kernel_time(k: Kernel, grid, block, args: KernelArgs, warmup: int, reps: int, lds_bytes: int = 0,
                stream=None) -> List[float]:
    u3 = ctypes.c_uint32 * 3
    ms = (ctypes.c_float * reps)()
    _check(_lib().asmevo_kernel_time(ctypes.byref(k), u3(*grid), u3(*block), lds_bytes, args.params, warmup, reps,
                                     ms, _stream_handle(stream)), "asmevo_kernel_time")
    return [float(v) for v in ms]
