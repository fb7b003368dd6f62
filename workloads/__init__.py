"""Seeded synthetic workloads shared by the tests, the bench and the smoke check.

This module only describes inputs: buffer shapes, dtypes, guard sizes, value
distributions, which elements a candidate perturbs, and which buffers are
compared with which tolerance.  It holds none of the differential oracle's
arithmetic (no Philox, no codecs, no comparisons); the GPU library and the CPU
oracle each turn these descriptions into their own descriptor structs.

The five workloads mirror the situations the paper's oracle faces (section
3.4): a Tier-1 synthetic buffer with canary guards and an out-of-bounds write,
a padded GEMM-like output, a captured decode dispatch with mixed dtypes
(Tier-2: no guards, integer buffers byte-exact), integer and fp8 outputs, and a
many-buffer candidate sweep.  Index lists are drawn with numpy's PCG64 from the
workload seed, so both sides receive the same list.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

# element types: name -> bytes per element
ESIZE = {"f32": 4, "bf16": 2, "f16": 2, "fp8e4m3": 1, "i32": 4, "i64": 8, "u8": 1}
FLOAT_DTYPES = ("f32", "bf16", "f16", "fp8e4m3")

# tolerances per dtype used by the many-buffer sweep (the other workloads
# state their own)
SWEEP_TOL = {"f32": (1e-5, 1e-5), "bf16": (1e-2, 1.6e-2), "f16": (1e-3, 1e-3),
             "fp8e4m3": (0.125, 0.125)}

ARENA_ALIGN = 256


def workload_seed(n: int) -> int:
    return 0xA5E0000000000000 | n


def rate_threshold(rate: float) -> int:
    """Bernoulli selection threshold T on a 32-bit uniform (selected iff x < T)
    for a rate 0 <= r <= 1: T = floor(r * 2^32 + 1/2), 2^32 for r = 1 -- the
    rule the library applies to the rate of its BOUNDARY distribution.  Both
    the library's binding and the oracle's take a RATE rule's T from here."""
    if not 0.0 <= rate <= 1.0:
        raise ValueError(f"rate {rate} outside [0, 1]")
    if rate == 1.0:
        return 1 << 32
    return int(math.floor(rate * 4294967296.0 + 0.5))   # rate * 2^32 is exact; so is + 1/2 below 2^52


@dataclass(frozen=True)
class Alloc:
    """One guarded allocation: [guard_lo][rows x stride elements][guard_hi].

    The last row carries no padding, so the data region is
    ((rows - 1) * stride + cols) elements long.
    """
    alloc_id: int
    dtype: str
    rows: int
    cols: int
    stride: int
    guard_lo: int = 0
    guard_hi: int = 0
    dist: str = "normal"          # normal | uniform_int | bits | const | boundary
    p0: float = 0.0               # normal: mean; const: value; boundary: rate of boundary patterns
    p1: float = 1.0               # normal, boundary: standard deviation
    i0: int = 0                   # uniform_int: [i0, i1)
    i1: int = 0
    saturate: bool = False        # fp8: clamp to +-448 before rounding

    @property
    def esize(self) -> int:
        return ESIZE[self.dtype]

    @property
    def n_elements(self) -> int:
        return self.rows * self.cols

    @property
    def data_bytes(self) -> int:
        if self.rows <= 0 or self.cols <= 0:
            return 0
        return ((self.rows - 1) * self.stride + self.cols) * self.esize

    @property
    def total_bytes(self) -> int:
        return self.guard_lo + self.data_bytes + self.guard_hi


@dataclass(frozen=True)
class Injection:
    """A perturbation of the candidate state (or of both states, sides='both').

    kind: flip_bit | step_within | set_beyond | set_nan | set_inf |
          guard_write_lo | guard_write_hi.
    index: element index (logical row-major), or byte offset within a guard.
    arg: bit index (-1 = random bit) | infinity sign (0 +, 1 -) | guard byte count.
    rate: if set, a Bernoulli rule over every element instead of one index.
    """
    alloc: int
    kind: str
    sides: str = "candidate"
    arg: int = 0
    index: int = 0
    atol: float = 0.0
    rtol: float = 0.0
    rate: Optional[float] = None


@dataclass(frozen=True)
class Compare:
    """One compared buffer pair (candidate vs reference) of allocation `alloc`."""
    alloc: int
    mode: str = "tolerance"       # tolerance | bitwise
    nan_policy: str = "equal"     # equal | strict
    atol: float = 0.0
    rtol: float = 0.0


@dataclass
class Workload:
    name: str
    description: str
    seed: int
    allocs: List[Alloc]
    injections: List[Injection]
    compares: List[Compare]
    offsets: List[int] = field(default_factory=list)   # byte offset of each alloc in its arena
    arena_bytes: int = 0

    def __post_init__(self):
        if not self.offsets:
            off = 0
            offs = []
            for a in self.allocs:
                offs.append(off)
                off += -(-a.total_bytes // ARENA_ALIGN) * ARENA_ALIGN
            self.offsets = offs
            self.arena_bytes = max(off, ARENA_ALIGN)

    def data_offset(self, k: int) -> int:
        return self.offsets[k] + self.allocs[k].guard_lo

    def compared_bytes(self) -> int:
        """2 x logical bytes of every compared pair plus candidate guard bytes."""
        total = 0
        for c in self.compares:
            a = self.allocs[c.alloc]
            total += 2 * a.n_elements * a.esize
        for a in self.allocs:
            total += a.guard_lo + a.guard_hi
        return total


def _distinct(rng: np.random.Generator, n: int, k: int) -> np.ndarray:
    """k distinct indices in [0, n), in draw order."""
    if k > n:
        raise ValueError("more distinct indices than elements")
    picked = []
    seen = set()
    while len(picked) < k:
        for v in rng.integers(0, n, size=2 * k):
            v = int(v)
            if v not in seen:
                seen.add(v)
                picked.append(v)
                if len(picked) == k:
                    break
    return np.array(picked, dtype=np.int64)


# ---------------------------------------------------------------------------
# The five workloads.  `small=True` keeps the structure but shrinks the shapes
# so the CPU oracle can check every element in seconds while still spanning
# many GPU tiles and a ragged tail.
# ---------------------------------------------------------------------------

def single_fp32(small: bool = False) -> Workload:
    """fp32 buffer of 2^20 N(0,1) values, 4 KiB canary guards on each side;
    candidate: 32 perturbations inside atol=rtol=1e-5, 32 beyond, and one
    4-byte out-of-bounds write into a guard."""
    seed = workload_seed(1)
    n = (1 << 20) if not small else (1 << 16) + 37
    tol = 1e-5
    alloc = Alloc(0, "f32", 1, n, n, 4096, 4096, "normal", 0.0, 1.0)
    rng = np.random.default_rng(seed)
    idx = _distinct(rng, n, 64)
    inj = [Injection(0, "step_within", index=int(i), atol=tol, rtol=tol) for i in idx[:32]]
    inj += [Injection(0, "set_beyond", index=int(i), atol=tol, rtol=tol) for i in idx[32:]]
    side = int(rng.integers(0, 2))
    off = int(rng.integers(0, 4096 // 4)) * 4
    inj.append(Injection(0, "guard_write_hi" if side else "guard_write_lo", arg=4, index=off))
    cmp_ = [Compare(0, "tolerance", "equal", tol, tol)]
    return Workload("single_fp32", "fp32 2^20 N(0,1), 4 KiB guards, 32 within + 32 beyond + 1 OOB write",
                    seed, [alloc], inj, cmp_)


def padded_bf16(small: bool = False) -> Workload:
    """bf16 8192x8192 GEMM-like output N(0, 64) with row stride 8320; candidate:
    1% last-bit flips, 50 matched + 50 unmatched NaN, 5 matched + 5 unmatched
    +-Inf; atol=1e-2, rtol=1.6e-2; compared under both NaN policies."""
    seed = workload_seed(2)
    rows, cols, stride = (8192, 8192, 8320) if not small else (301, 1000, 1040)
    alloc = Alloc(0, "bf16", rows, cols, stride, 0, 0, "normal", 0.0, 8.0)
    rng = np.random.default_rng(seed)
    idx = _distinct(rng, rows * cols, 110)
    inj = [Injection(0, "flip_bit", arg=0, rate=0.01)]
    inj += [Injection(0, "set_nan", sides="both", index=int(i)) for i in idx[:50]]
    inj += [Injection(0, "set_nan", index=int(i)) for i in idx[50:100]]
    inj += [Injection(0, "set_inf", sides="both", arg=k % 2, index=int(i)) for k, i in enumerate(idx[100:105])]
    inj += [Injection(0, "set_inf", arg=k % 2, index=int(i)) for k, i in enumerate(idx[105:110])]
    cmp_ = [Compare(0, "tolerance", "equal", 1e-2, 1.6e-2),
            Compare(0, "tolerance", "strict", 1e-2, 1.6e-2)]
    return Workload("padded_bf16", "bf16 8192x8192 stride 8320 N(0,64), 1% bit-0 flips, 110 NaN/Inf",
                    seed, [alloc], inj, cmp_)


def decode_state(small: bool = False) -> Workload:
    """Captured decode-dispatch state: fp16 K and V caches [8192,16,8,128],
    int32 block table [256,512] in [0,8192), fp32 output [256,32,128] N(0,1);
    64 sparse differences per buffer; no guards (state restored in place)."""
    seed = workload_seed(3)
    blocks = 8192 if not small else 67
    tbl_rows = 256 if not small else 19
    out_rows = 256 if not small else 23
    kv_rows = blocks * 16 * 8
    allocs = [
        Alloc(0, "f16", kv_rows, 128, 128, 0, 0, "normal", 0.0, 1.0),
        Alloc(1, "f16", kv_rows, 128, 128, 0, 0, "normal", 0.0, 1.0),
        Alloc(2, "i32", tbl_rows, 512, 512, 0, 0, "uniform_int", i0=0, i1=8192),
        Alloc(3, "f32", out_rows * 32, 128, 128, 0, 0, "normal", 0.0, 1.0),
    ]
    rng = np.random.default_rng(seed)
    tol = 1e-3
    inj = []
    for k in (0, 1, 3):
        idx = _distinct(rng, allocs[k].n_elements, 64)
        inj += [Injection(k, "step_within", index=int(i), atol=tol, rtol=tol) for i in idx[:32]]
        inj += [Injection(k, "set_beyond", index=int(i), atol=tol, rtol=tol) for i in idx[32:]]
    idx = _distinct(rng, allocs[2].n_elements, 64)
    inj += [Injection(2, "flip_bit", arg=-1, index=int(i)) for i in idx]
    cmp_ = [Compare(0, "tolerance", "equal", tol, tol), Compare(1, "tolerance", "equal", tol, tol),
            Compare(2, "bitwise"), Compare(3, "tolerance", "equal", tol, tol)]
    return Workload("decode_state", "fp16 K/V [8192,16,8,128], i32 table [256,512], fp32 out [256,32,128]",
                    seed, allocs, inj, cmp_)


def int_lowp(small: bool = False) -> Workload:
    """int32 top-k indices [65536,8] in [0,2^20), int64 scatter destinations
    2^24 in [0,2^24), fp8 e4m3 2^28 N(0,1) saturated; 16 distinct single-bit
    flips per buffer; fp8 compared bitwise and with atol=rtol=0.125."""
    seed = workload_seed(4)
    topk_rows = 65536 if not small else 5003
    n64 = (1 << 24) if not small else (1 << 14) + 11
    n8 = (1 << 28) if not small else (1 << 18) + 5
    allocs = [
        Alloc(0, "i32", topk_rows, 8, 8, 0, 0, "uniform_int", i0=0, i1=1 << 20),
        Alloc(1, "i64", 1, n64, n64, 0, 0, "uniform_int", i0=0, i1=1 << 24),
        Alloc(2, "fp8e4m3", 1, n8, n8, 0, 0, "normal", 0.0, 1.0, saturate=True),
    ]
    rng = np.random.default_rng(seed)
    inj = []
    for k in range(3):
        idx = _distinct(rng, allocs[k].n_elements, 16)
        inj += [Injection(k, "flip_bit", arg=-1, index=int(i)) for i in idx]
    cmp_ = [Compare(0, "bitwise"), Compare(1, "bitwise"),
            Compare(2, "tolerance", "equal", 0.125, 0.125)]
    return Workload("int_lowp", "i32 top-k [65536,8], i64 2^24, fp8e4m3 2^28; 16 flips each",
                    seed, allocs, inj, cmp_)


def sweep(small: bool = False, n_buffers: int = 4096, total_bytes: int = 64 << 30,
          lo_bytes: int = 4 << 10, hi_bytes: int = 256 << 20) -> Workload:
    """Full candidate-loop sweep: 4096 buffers with log-uniform sizes in
    [4 KiB, 256 MiB] scaled to ~64 GiB per side, dtypes uniform over
    fp32/bf16/fp16/fp8-e4m3/int32, 1 KiB guards on each side, seeded
    1e-6 random-bit flips.  The log-uniform draw over [4 KiB, 256 MiB] has a
    mean of ~24 MB, i.e. ~92 GiB for 4096 buffers, so sizes are scaled to the
    stated total and clamped to the range (the realised total is reported)."""
    seed = workload_seed(5)
    if small:
        n_buffers, total_bytes, lo_bytes, hi_bytes = 48, 24 << 20, 4 << 10, 4 << 20
    rng = np.random.default_rng(seed)
    logs = rng.uniform(math.log(lo_bytes), math.log(hi_bytes), size=n_buffers)
    sizes = np.exp(logs)
    sizes = sizes * (total_bytes / sizes.sum())
    sizes = np.clip(sizes, lo_bytes, hi_bytes)
    dt_names = ("f32", "bf16", "f16", "fp8e4m3", "i32")
    dts = rng.integers(0, len(dt_names), size=n_buffers)
    allocs, inj, cmp_ = [], [], []
    for k in range(n_buffers):
        dt = dt_names[int(dts[k])]
        n = int(sizes[k]) // ESIZE[dt]
        if dt == "i32":
            a = Alloc(k, dt, 1, n, n, 1024, 1024, "uniform_int", i0=0, i1=1 << 31)
            cmp_.append(Compare(k, "bitwise"))
        else:
            a = Alloc(k, dt, 1, n, n, 1024, 1024, "normal", 0.0, 1.0, saturate=(dt == "fp8e4m3"))
            at, rt = SWEEP_TOL[dt]
            cmp_.append(Compare(k, "tolerance", "equal", at, rt))
        allocs.append(a)
        inj.append(Injection(k, "flip_bit", arg=-1, rate=1e-6))
    return Workload("sweep", f"{n_buffers} buffers log-uniform 4KiB-256MiB, ~{total_bytes >> 30} GiB/side, "
                    "mixed dtypes, 1 KiB guards, 1e-6 random-bit flips",
                    seed, allocs, inj, cmp_)


ALL = {"single_fp32": single_fp32, "padded_bf16": padded_bf16, "decode_state": decode_state,
       "int_lowp": int_lowp, "sweep": sweep}
