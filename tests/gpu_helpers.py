"""Shared helpers of the GPU parity tests: run a workload through the HIP
library, run it through the CPU oracle, compare outputs bit for bit."""
import struct
import sys

import numpy as np

import oracle

THREADS = 16


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def run_gpu(w, variant: int = 1, workgroups: int = 0):
    from paper_2608_20711_amd.state import DeviceState
    st = DeviceState(w)
    st.fill("ref", 0)
    st.fill("cand", variant)
    st.diff(workgroups=workgroups)
    st.guard()
    return st


def bits(v) -> int:
    if isinstance(v, float):
        return struct.unpack("<Q", struct.pack("<d", v))[0]
    return int(v)


def assert_results_equal(got, want, what=""):
    assert len(got) == len(want), what
    for k, (g, o) in enumerate(zip(got, want)):
        for f in o:
            assert bits(g[f]) == bits(o[f]), f"{what} entry {k} field {f}: gpu {g[f]!r} oracle {o[f]!r}"


def assert_bytes_equal(got: np.ndarray, want: np.ndarray, what=""):
    if not np.array_equal(got, want):
        bad = np.flatnonzero(got != want)
        raise AssertionError(f"{what}: {bad.size} bytes differ, first at {bad[0]} "
                             f"(gpu {got[bad[0]]:#04x}, oracle {want[bad[0]]:#04x})")


def assert_fill_equal(w, gpu_arena: np.ndarray, ora_arena: np.ndarray, what=""):
    for k, a in enumerate(w.allocs):
        o = w.offsets[k]
        assert_bytes_equal(gpu_arena[o:o + a.total_bytes], ora_arena[o:o + a.total_bytes],
                           f"{what} alloc {k} ({a.dtype} {a.rows}x{a.cols}/{a.stride})")


def fill_windows(w, k, rng, n_random=16, width=4096):
    """Byte windows of allocation k worth checking: both ends, the guards,
    windows around every point injection, and random windows."""
    a = w.allocs[k]
    tot = a.total_bytes
    wins = [(0, min(tot, width)), (max(0, tot - width), min(tot, width))]
    if a.guard_lo:
        wins.append((0, a.guard_lo))
    if a.guard_hi:
        wins.append((a.guard_lo + a.data_bytes, a.guard_hi))
    for j in w.injections:
        if j.alloc != k or j.rate is not None or j.kind.startswith("guard"):
            continue
        r, c = divmod(j.index, a.cols)
        off = a.guard_lo + (r * a.stride + c) * a.esize
        s = max(0, off - 64)
        wins.append((s, min(128, tot - s)))
    for _ in range(n_random):
        if tot > width:
            s = int(rng.integers(0, tot - width))
            wins.append((s, width))
    return [(s, n) for s, n in wins if n > 0]


def check_fill_sampled(w, st, variant_of_side, rng, n_random=16, width=4096):
    P = oracle.Prepared(w)
    for side, variant in variant_of_side.items():
        for k in range(len(w.allocs)):
            for s, n in fill_windows(w, k, rng, n_random, width):
                got = st.alloc_bytes(side, k, s, n)
                want = P.fill_range(k, variant, s, n)
                assert_bytes_equal(got, want, f"{side} alloc {k} bytes [{s}, {s + n})")
