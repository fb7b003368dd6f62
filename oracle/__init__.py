"""CPU oracle for the differential-oracle hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow C implementation (ref_oracle.c, built with gcc, fp64, no
fast-math, contraction off) of what the GPU library computes: the guarded
seeded fill, the element-wise comparison of a candidate state against the
reference state (paper section 3.2, Eq. 1 and iota; section 3.4 Tier-1/Tier-2
checks), and the canary-guard check.  It shares no code with the GPU library
and neither imports the other.  Only tests/, the smoke entry point and the
bench's cpu_baseline leg may use it; the product path never does.

This binding only marshals arguments (ctypes); every computation happens in
ref_oracle.c.  ctypes releases the GIL during each call, so callers may run
independent calls from a thread pool.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ref_oracle.c")
_SO = os.environ.get("REF_ORACLE_LIBRARY") or os.path.join(_HERE, "libref_oracle.so")

# codes of ref_oracle.h
DTYPE = {"f32": 1, "bf16": 2, "f16": 3, "fp8e4m3": 4, "i32": 5, "i64": 6, "u8": 7}
ESIZE = {1: 4, 2: 2, 3: 2, 4: 1, 5: 4, 6: 8, 7: 1}
MODE = {"bitwise": 0, "tolerance": 1}
NAN_POLICY = {"equal": 0, "strict": 1}
DIST = {"normal": 0, "uniform_int": 1, "bits": 2, "const": 3, "boundary": 4}
KIND = {"flip_bit": 1, "step_within": 2, "set_beyond": 3, "set_nan": 4, "set_inf": 5,
        "guard_write_lo": 6, "guard_write_hi": 7, "pad_write": 8}
RATE = 0x100
SIDES = {"candidate": 0, "both": 1}


def build() -> str:
    """Compile the oracle with gcc (always recompiles)."""
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
           "-ffp-contract=off", "-fno-fast-math", "-o", _SO + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_SO + ".tmp", _SO)
    return _SO


class RefAlloc(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("alloc_id", ctypes.c_uint32),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64), ("stride", ctypes.c_int64),
                ("guard_lo", ctypes.c_int64), ("guard_hi", ctypes.c_int64),
                ("dist", ctypes.c_int32), ("saturate", ctypes.c_int32),
                ("p0", ctypes.c_double), ("p1", ctypes.c_double),
                ("i0", ctypes.c_int64), ("i1", ctypes.c_int64)]


class RefInj(ctypes.Structure):
    _fields_ = [("alloc", ctypes.c_uint32), ("kind", ctypes.c_uint32),
                ("sides", ctypes.c_uint32), ("arg", ctypes.c_uint32),
                ("index", ctypes.c_int64), ("atol", ctypes.c_double), ("rtol", ctypes.c_double)]


class RefSeg(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("nan_policy", ctypes.c_int32), ("pad_", ctypes.c_int32),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("stride_a", ctypes.c_int64), ("stride_b", ctypes.c_int64),
                ("atol", ctypes.c_double), ("rtol", ctypes.c_double)]


MAX_DIMS = 8


class RefSegND(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("nan_policy", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("index_base", ctypes.c_int64),
                ("shape", ctypes.c_int64 * MAX_DIMS),
                ("stride_a", ctypes.c_int64 * MAX_DIMS), ("stride_b", ctypes.c_int64 * MAX_DIMS),
                ("atol", ctypes.c_double), ("rtol", ctypes.c_double)]


class RefSegResult(ctypes.Structure):
    _fields_ = [("mismatches", ctypes.c_uint64), ("first_mismatch", ctypes.c_int64),
                ("bitwise_mismatches", ctypes.c_uint64), ("first_bitwise", ctypes.c_int64),
                ("nonfinite_mismatches", ctypes.c_uint64),
                ("max_abs", ctypes.c_double), ("max_rel", ctypes.c_double)]

    def as_dict(self) -> Dict:
        return {f: getattr(self, f) for f, _ in self._fields_}


class RefCosResult(ctypes.Structure):
    _fields_ = [("sum_ab", ctypes.c_double), ("sum_aa", ctypes.c_double), ("sum_bb", ctypes.c_double),
                ("cosine", ctypes.c_double), ("pairs", ctypes.c_uint64), ("sum_abs_ab", ctypes.c_double)]

    def as_dict(self) -> Dict:
        return {f: getattr(self, f) for f, _ in self._fields_}


class RefRegion(ctypes.Structure):
    _fields_ = [("dst", ctypes.c_void_p), ("src", ctypes.c_void_p), ("bytes", ctypes.c_int64)]


class RefGuardResult(ctypes.Structure):
    _fields_ = [("bad_lo", ctypes.c_uint64), ("bad_hi", ctypes.c_uint64),
                ("first_bad_lo", ctypes.c_int64), ("first_bad_hi", ctypes.c_int64),
                ("bad_pad", ctypes.c_uint64), ("first_bad_pad", ctypes.c_int64)]

    def as_dict(self) -> Dict:
        return {f: getattr(self, f) for f, _ in self._fields_}


_lib_handle: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    global _lib_handle
    if _lib_handle is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        P = ctypes.POINTER
        vp = ctypes.c_void_p
        L.ref_philox4x32_10.argtypes = [vp, vp, vp]
        L.ref_esize.argtypes = [ctypes.c_int32]
        L.ref_decode.argtypes = [ctypes.c_int32, ctypes.c_uint64, P(ctypes.c_double)]
        L.ref_encode_f32.argtypes = [ctypes.c_int32, ctypes.c_float, ctypes.c_int]
        L.ref_encode_f32.restype = ctypes.c_uint64
        L.ref_log_u.argtypes = [ctypes.c_uint32]
        L.ref_log_u.restype = ctypes.c_double
        L.ref_normal.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_int]
        L.ref_normal.restype = ctypes.c_double
        L.ref_element.argtypes = [P(RefAlloc), ctypes.c_int32, P(RefInj), ctypes.c_int64,
                                  ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64]
        L.ref_element.restype = ctypes.c_uint64
        L.ref_canary_byte.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int, ctypes.c_int64]
        L.ref_canary_byte.restype = ctypes.c_uint8
        L.ref_fill_range.argtypes = [P(RefAlloc), ctypes.c_int32, P(RefInj), ctypes.c_int64,
                                     ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64,
                                     ctypes.c_int64, vp]
        L.ref_diff_segment.argtypes = [P(RefSeg), vp, vp, P(RefSegResult)]
        L.ref_diff_segment_nd.argtypes = [P(RefSegND), vp, vp, P(RefSegResult)]
        L.ref_cosine_segment.argtypes = [P(RefSeg), vp, vp, P(RefCosResult)]
        L.ref_cosine_nd.argtypes = [P(RefSegND), ctypes.c_int32, vp, vp, P(RefCosResult)]
        L.ref_exact_sum.argtypes = [vp, ctypes.c_int64]
        L.ref_exact_sum.restype = ctypes.c_double
        L.ref_copy_regions.argtypes = [P(RefRegion), ctypes.c_int64]
        L.ref_guard_check.argtypes = [ctypes.c_uint64, ctypes.c_uint32, vp, ctypes.c_int64,
                                      vp, ctypes.c_int64, P(RefGuardResult)]
        L.ref_pad_check.argtypes = [P(RefAlloc), ctypes.c_uint64, vp, P(RefGuardResult)]
        L.ref_decode_n.argtypes = [ctypes.c_int32, vp, ctypes.c_int64, vp, vp]
        L.ref_encode_f32_n.argtypes = [ctypes.c_int32, vp, ctypes.c_int64, ctypes.c_int, vp]
        L.ref_log_u_n.argtypes = [vp, ctypes.c_int64, vp]
        L.ref_sincos_turns_n.argtypes = [vp, ctypes.c_int64, vp, vp]
        L.ref_normal_n.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int, vp]
        L.ref_philox_n.argtypes = [vp, vp, ctypes.c_int64, vp]
        L.ref_compare_pair_n.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_double,
                                         ctypes.c_double, vp, vp, ctypes.c_int64, vp, vp, vp]
        _lib_handle = L
    return _lib_handle


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


# --------------------------------------------------------------------------
# scalar / bulk primitives (pinned by tests/test_oracle_*.py)
# --------------------------------------------------------------------------

def philox(ctr: Sequence[int], key: Sequence[int]) -> List[int]:
    c = np.array(ctr, dtype=np.uint32)
    k = np.array(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().ref_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return [int(v) for v in out]


def philox_n(ctr: np.ndarray, key: np.ndarray) -> np.ndarray:
    ctr = np.ascontiguousarray(ctr, dtype=np.uint32).reshape(-1, 4)
    key = np.ascontiguousarray(key, dtype=np.uint32).reshape(-1, 2)
    out = np.zeros_like(ctr)
    lib().ref_philox_n(_ptr(ctr), _ptr(key), ctr.shape[0], _ptr(out))
    return out


def decode_n(dtype: str, raw: np.ndarray):
    raw = np.ascontiguousarray(raw, dtype=np.uint64)
    cls = np.zeros(raw.shape, dtype=np.int32)
    val = np.zeros(raw.shape, dtype=np.float64)
    lib().ref_decode_n(DTYPE[dtype], _ptr(raw), raw.size, _ptr(cls), _ptr(val))
    return cls, val


def _out(out, shape, dtype):
    """A caller's output array (contiguous, of the right type and size), or a new one."""
    if out is None:
        return np.zeros(shape, dtype=dtype)
    assert out.dtype == dtype and out.flags.c_contiguous and out.shape == shape
    return out


def encode_f32_n(dtype: str, x: np.ndarray, saturate: bool = False, out=None) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = _out(out, x.shape, np.uint64)
    lib().ref_encode_f32_n(DTYPE[dtype], _ptr(x), x.size, int(saturate), _ptr(out))
    return out


def log_u_n(x: np.ndarray, out=None) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.uint32)
    out = _out(out, x.shape, np.float64)
    lib().ref_log_u_n(_ptr(x), x.size, _ptr(out))
    return out


def sincos_turns_n(x: np.ndarray, c=None, s=None):
    x = np.ascontiguousarray(x, dtype=np.uint32)
    c = _out(c, x.shape, np.float64)
    s = _out(s, x.shape, np.float64)
    lib().ref_sincos_turns_n(_ptr(x), x.size, _ptr(c), _ptr(s))
    return c, s


def normal_n(xa: np.ndarray, xb: np.ndarray, which: int, out=None) -> np.ndarray:
    xa = np.ascontiguousarray(xa, dtype=np.uint32)
    xb = np.ascontiguousarray(xb, dtype=np.uint32)
    out = _out(out, xa.shape, np.float64)
    lib().ref_normal_n(_ptr(xa), _ptr(xb), xa.size, which, _ptr(out))
    return out


def compare_pair_n(dtype: str, mode: str, nan_policy: str, atol: float, rtol: float,
                   ra: np.ndarray, rb: np.ndarray, flags=None, max_abs=None, max_rel=None):
    """Each pair compared on its own: (flags, max_abs, max_rel) with flags bit 0
    a bitwise difference, bit 1 a mismatch, bit 2 a non-finite mismatch."""
    ra = np.ascontiguousarray(ra, dtype=np.uint64)
    rb = np.ascontiguousarray(rb, dtype=np.uint64)
    assert ra.shape == rb.shape
    flags = _out(flags, ra.shape, np.uint8)
    max_abs = _out(max_abs, ra.shape, np.float64)
    max_rel = _out(max_rel, ra.shape, np.float64)
    lib().ref_compare_pair_n(DTYPE[dtype], MODE[mode], NAN_POLICY[nan_policy], atol, rtol, _ptr(ra), _ptr(rb),
                             ra.size, _ptr(flags), _ptr(max_abs), _ptr(max_rel))
    return flags, max_abs, max_rel


def canary_byte(seed: int, alloc_id: int, side: int, p: int) -> int:
    return int(lib().ref_canary_byte(seed, alloc_id, side, p))


# --------------------------------------------------------------------------
# workload-level helpers (workloads.Workload -> oracle structs)
# --------------------------------------------------------------------------

def ref_allocs(w) -> ctypes.Array:
    arr = (RefAlloc * max(1, len(w.allocs)))()
    for k, a in enumerate(w.allocs):
        arr[k] = RefAlloc(DTYPE[a.dtype], a.alloc_id, a.rows, a.cols, a.stride, a.guard_lo,
                          a.guard_hi, DIST[a.dist], int(a.saturate), a.p0, a.p1, a.i0, a.i1)
    return arr


def ref_injections(w) -> ctypes.Array:
    from workloads import rate_threshold
    arr = (RefInj * max(1, len(w.injections)))()
    for t, j in enumerate(w.injections):
        kind = KIND[j.kind]
        index = j.index
        if j.rate is not None:
            kind |= RATE
            index = rate_threshold(j.rate)
        arg = j.arg & 0xFFFFFFFF
        arr[t] = RefInj(j.alloc, kind, SIDES[j.sides], arg, index, j.atol, j.rtol)
    return arr


class Prepared:
    """Oracle structs of one workload, built once."""

    def __init__(self, w):
        self.w = w
        self.allocs = ref_allocs(w)
        self.inj = ref_injections(w)
        self.n_inj = len(w.injections)

    def element(self, k: int, variant: int, i: int) -> int:
        return int(lib().ref_element(self.allocs, k, self.inj, self.n_inj, self.w.seed, variant, i))

    def fill_range(self, k: int, variant: int, off: int, nbytes: int) -> np.ndarray:
        out = np.empty(nbytes, dtype=np.uint8)
        rc = lib().ref_fill_range(self.allocs, k, self.inj, self.n_inj, self.w.seed, variant,
                                  off, nbytes, _ptr(out) if nbytes else None)
        if rc != 0:
            raise ValueError("oracle fill rejected the range")
        return out

    def fill_alloc(self, k: int, variant: int, threads: int = 1) -> np.ndarray:
        total = self.w.allocs[k].total_bytes
        if threads <= 1 or total < (1 << 20):
            return self.fill_range(k, variant, 0, total)
        from concurrent.futures import ThreadPoolExecutor
        step = -(-total // (threads * 4))
        step = -(-step // 16) * 16
        parts = [(o, min(step, total - o)) for o in range(0, total, step)]
        with ThreadPoolExecutor(threads) as ex:
            chunks = list(ex.map(lambda p: self.fill_range(k, variant, p[0], p[1]), parts))
        return np.concatenate(chunks)

    def fill_arena(self, variant: int, threads: int = 1) -> np.ndarray:
        arena = np.zeros(self.w.arena_bytes, dtype=np.uint8)
        for k, a in enumerate(self.w.allocs):
            o = self.w.offsets[k]
            arena[o:o + a.total_bytes] = self.fill_alloc(k, variant, threads)
        return arena


def diff_segment(dtype: str, mode: str, nan_policy: str, rows: int, cols: int,
                 stride_a: int, stride_b: int, atol: float, rtol: float,
                 a: np.ndarray, b: np.ndarray, a_off: int = 0, b_off: int = 0) -> Dict:
    """a, b: uint8 arrays; a_off/b_off: byte offset of element (0,0)."""
    seg = RefSeg(DTYPE[dtype], MODE[mode], NAN_POLICY[nan_policy], 0, rows, cols, stride_a,
                 stride_b, atol, rtol)
    res = RefSegResult()
    a = np.ascontiguousarray(a).view(np.uint8)
    b = np.ascontiguousarray(b).view(np.uint8)
    rc = lib().ref_diff_segment(ctypes.byref(seg), _ptr(a) + a_off, _ptr(b) + b_off, ctypes.byref(res))
    if rc != 0:
        raise ValueError("oracle diff rejected the segment")
    return res.as_dict()


def diff_segment_nd(dtype: str, mode: str, nan_policy: str, shape: Sequence[int],
                    stride_a: Sequence[int], stride_b: Sequence[int], atol: float, rtol: float,
                    a: np.ndarray, b: np.ndarray, a_off: int = 0, b_off: int = 0,
                    index_base: int = 0) -> Dict:
    """N-dimensional segment: shape and strides (in elements) of both
    operands; a, b: uint8 arrays with element (0, ..., 0) at a_off / b_off."""
    nd = len(shape)
    assert nd <= MAX_DIMS and len(stride_a) == nd and len(stride_b) == nd
    seg = RefSegND(DTYPE[dtype], MODE[mode], NAN_POLICY[nan_policy], nd, index_base,
                   (ctypes.c_int64 * MAX_DIMS)(*shape), (ctypes.c_int64 * MAX_DIMS)(*stride_a),
                   (ctypes.c_int64 * MAX_DIMS)(*stride_b), atol, rtol)
    res = RefSegResult()
    a = np.ascontiguousarray(a).view(np.uint8)
    b = np.ascontiguousarray(b).view(np.uint8)
    rc = lib().ref_diff_segment_nd(ctypes.byref(seg), _ptr(a) + a_off, _ptr(b) + b_off, ctypes.byref(res))
    if rc != 0:
        raise ValueError("oracle diff rejected the segment")
    return res.as_dict()


def merge_results(parts: Sequence[Dict]) -> Dict:
    """One result for several segments that share it: counts add, first
    indices take the lowest (ignoring -1), maxima take the largest."""
    out = {"mismatches": 0, "first_mismatch": -1, "bitwise_mismatches": 0, "first_bitwise": -1,
           "nonfinite_mismatches": 0, "max_abs": 0.0, "max_rel": 0.0}
    for r in parts:
        for f in ("mismatches", "bitwise_mismatches", "nonfinite_mismatches"):
            out[f] += r[f]
        for f in ("first_mismatch", "first_bitwise"):
            if r[f] >= 0 and (out[f] < 0 or r[f] < out[f]):
                out[f] = r[f]
        for f in ("max_abs", "max_rel"):
            out[f] = max(out[f], r[f])
    return out


def cosine_segment(dtype: str, rows: int, cols: int, stride_a: int, stride_b: int,
                   a: np.ndarray, b: np.ndarray, a_off: int = 0, b_off: int = 0) -> Dict:
    """Cosine term of Eq. 1 from the exact sums, each rounded once (see
    ref_oracle.h); also sum_abs_ab, the scale of other orders' error bounds."""
    seg = RefSeg(DTYPE[dtype], MODE["bitwise"], 0, 0, rows, cols, stride_a, stride_b, 0.0, 0.0)
    res = RefCosResult()
    a = np.ascontiguousarray(a).view(np.uint8)
    b = np.ascontiguousarray(b).view(np.uint8)
    rc = lib().ref_cosine_segment(ctypes.byref(seg), _ptr(a) + a_off, _ptr(b) + b_off, ctypes.byref(res))
    if rc != 0:
        raise ValueError("oracle cosine rejected the segment")
    return res.as_dict()


def cosine_nd(dtype: str, parts: Sequence, a: np.ndarray, b: np.ndarray) -> Dict:
    """Cosine term of one result over the elements of N-D segments, from the
    exact sums (see ref_oracle.h).  parts: (shape, stride_a, stride_b, a_off, b_off) per
    segment, in segment order; strides in elements, offsets in bytes of the
    uint8 arrays a and b."""
    n = len(parts)
    segs = (RefSegND * max(n, 1))()
    a = np.ascontiguousarray(a).view(np.uint8)
    b = np.ascontiguousarray(b).view(np.uint8)
    pa = (ctypes.c_void_p * max(n, 1))()
    pb = (ctypes.c_void_p * max(n, 1))()
    for k, (shape, sa, sb, a_off, b_off) in enumerate(parts):
        nd = len(shape)
        assert nd <= MAX_DIMS and len(sa) == nd and len(sb) == nd
        segs[k] = RefSegND(DTYPE[dtype], MODE["bitwise"], 0, nd, 0, (ctypes.c_int64 * MAX_DIMS)(*shape),
                           (ctypes.c_int64 * MAX_DIMS)(*sa), (ctypes.c_int64 * MAX_DIMS)(*sb), 0.0, 0.0)
        pa[k] = _ptr(a) + a_off
        pb[k] = _ptr(b) + b_off
    res = RefCosResult()
    rc = lib().ref_cosine_nd(segs, n, pa, pb, ctypes.byref(res))
    if rc != 0:
        raise ValueError("oracle N-D cosine rejected the segments")
    return res.as_dict()


def exact_sum(x: np.ndarray) -> float:
    """The float64 values of x summed exactly, rounded once to nearest (ties to even)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    return float(lib().ref_exact_sum(_ptr(x) if x.size else None, x.size))


def cosine_workload(w, cand: np.ndarray, ref: np.ndarray, threads: int = 1) -> List[Dict]:
    def one(c):
        a = w.allocs[c.alloc]
        off = w.data_offset(c.alloc)
        return cosine_segment(a.dtype, a.rows, a.cols, a.stride, a.stride, cand, ref, off, off)
    if threads <= 1:
        return [one(c) for c in w.compares]
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(threads) as ex:
        return list(ex.map(one, w.compares))


def diff_workload(w, cand: np.ndarray, ref: np.ndarray, threads: int = 1) -> List[Dict]:
    """Compares every Compare entry of `w`; cand/ref are whole arenas (uint8)."""
    def one(c):
        a = w.allocs[c.alloc]
        off = w.data_offset(c.alloc)
        return diff_segment(a.dtype, c.mode, c.nan_policy, a.rows, a.cols, a.stride, a.stride,
                            c.atol, c.rtol, cand, ref, off, off)
    if threads <= 1:
        return [one(c) for c in w.compares]
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(threads) as ex:
        return list(ex.map(one, w.compares))


def copy_regions(buf: np.ndarray, regions) -> None:
    """regions: (dst_offset, src_offset, bytes) inside the uint8 array `buf`, copied in order."""
    arr = (RefRegion * max(1, len(regions)))()
    base = _ptr(buf)
    for k, (d, s_, n) in enumerate(regions):
        assert 0 <= d and d + n <= buf.size and 0 <= s_ and s_ + n <= buf.size
        arr[k] = RefRegion(base + d, base + s_, n)
    lib().ref_copy_regions(arr, len(regions))


def guard_check(seed: int, alloc_id: int, lo: np.ndarray, hi: np.ndarray) -> Dict:
    lo = np.ascontiguousarray(lo, dtype=np.uint8)
    hi = np.ascontiguousarray(hi, dtype=np.uint8)
    res = RefGuardResult()
    lib().ref_guard_check(seed, alloc_id, _ptr(lo) if lo.size else None, lo.size,
                          _ptr(hi) if hi.size else None, hi.size, ctypes.byref(res))
    return res.as_dict()


def pad_check(w, k: int, data: np.ndarray) -> Dict:
    """Row-pad check of allocation k of workload w; `data` is its data region."""
    data = np.ascontiguousarray(data, dtype=np.uint8)
    assert data.size == w.allocs[k].data_bytes
    res = RefGuardResult()
    allocs = ref_allocs(w)
    rc = lib().ref_pad_check(ctypes.byref(allocs[k]), w.seed, _ptr(data) if data.size else None,
                             ctypes.byref(res))
    if rc != 0:
        raise ValueError("oracle pad check rejected the allocation")
    return {"bad_pad": res.bad_pad, "first_bad_pad": res.first_bad_pad}


def pad_check_alloc(seed: int, alloc_id: int, dtype: str, rows: int, cols: int, stride: int,
                    data: np.ndarray) -> Dict:
    """Row-pad check of one allocation given by its geometry; `data` is its data region."""
    data = np.ascontiguousarray(data, dtype=np.uint8)
    a = RefAlloc(DTYPE[dtype], alloc_id, rows, cols, stride, 0, 0, 0, 0, 0.0, 0.0, 0, 0)
    res = RefGuardResult()
    if lib().ref_pad_check(ctypes.byref(a), seed, _ptr(data) if data.size else None, ctypes.byref(res)) != 0:
        raise ValueError("oracle pad check rejected the allocation")
    return {"bad_pad": res.bad_pad, "first_bad_pad": res.first_bad_pad}


def guard_workload(w, arena: np.ndarray) -> List[Dict]:
    """Guard and row-pad check of every allocation of w in `arena`."""
    out = []
    for k, a in enumerate(w.allocs):
        o = w.offsets[k]
        lo = arena[o:o + a.guard_lo]
        h0 = o + a.guard_lo + a.data_bytes
        hi = arena[h0:h0 + a.guard_hi]
        r = guard_check(w.seed, a.alloc_id, lo, hi)
        r.update(pad_check(w, k, arena[o + a.guard_lo:h0]))
        out.append(r)
    return out
