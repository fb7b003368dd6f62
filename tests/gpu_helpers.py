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


# ------------------------------------------------------------ the cosine term
U = 2.0 ** -53


def gamma(k: int) -> float:
    """gamma_k = k u / (1 - k u): the relative error bound of k roundings."""
    return k * U / (1.0 - k * U)


def cosine_depth(dtype: str, blocks: int) -> int:
    """Roundings on one product's path through the library's documented order:
    the lane's run of 4 chunks, 6 butterfly steps, the block tree's depth,
    and one more for the oracle's own rounding of the exact sum."""
    import cosine_order
    return cosine_order.lane_terms(dtype) + 6 + max(1, blocks - 1).bit_length() + 1


def assert_cosine(got, exact, model, dtypes, what=""):
    """The GPU's cosine results against (1) the documented-order model, bit for
    bit on every field (the library's reproducibility promise), and (2) the
    oracle's exact sums, within the error bound of that order: |s - S| <=
    gamma_D * sum|t| for each sum, 2.5 gamma_D + 16u for the cosine (the three
    sums' errors through one division, two square roots and a product), and
    the pair count exactly."""
    import math
    assert len(got) == len(exact) == len(model) == len(dtypes), what
    for k, (g, e, m, dt) in enumerate(zip(got, exact, model, dtypes)):
        for f in m:
            assert bits(g[f]) == bits(m[f]), f"{what} entry {k} field {f}: gpu {g[f]!r} order model {m[f]!r}"
        assert g["pairs"] == e["pairs"], f"{what} entry {k}: pairs gpu {g['pairs']} oracle {e['pairs']}"
        if math.isnan(e["cosine"]):
            assert math.isnan(g["cosine"]) and g["sum_ab"] == g["sum_aa"] == g["sum_bb"] == 0.0, f"{what} {k}"
            continue
        gd = gamma(cosine_depth(dt, g["blocks"]))
        for f, scale in (("sum_ab", e["sum_abs_ab"]), ("sum_aa", e["sum_aa"]), ("sum_bb", e["sum_bb"])):
            assert abs(g[f] - e[f]) <= gd * scale, (
                f"{what} entry {k} {f}: gpu {g[f]!r} exact {e[f]!r} bound {gd * scale!r}")
        if e["sum_aa"] == 0.0 or e["sum_bb"] == 0.0:
            assert g["cosine"] == e["cosine"], f"{what} entry {k} cosine {g['cosine']} vs {e['cosine']}"
        else:
            assert abs(g["cosine"] - e["cosine"]) <= 2.5 * gd + 16 * U, (
                f"{what} entry {k} cosine: gpu {g['cosine']!r} exact {e['cosine']!r}")


def cosine_expected(dtype, rows, cols, sa, sb, a, b, a_off=0, b_off=0):
    """(oracle result from exact sums, documented-order model) of one 2-D segment."""
    import cosine_order
    return (oracle.cosine_segment(dtype, rows, cols, sa, sb, a, b, a_off, b_off),
            cosine_order.cosine_2d(dtype, rows, cols, sa, sb, a, b, a_off, b_off))


def cosine_workload_expected(w, cand, ref, threads=THREADS):
    """Exact oracle results, order-model results and dtypes of every compare of w."""
    from concurrent.futures import ThreadPoolExecutor
    def one(c):
        a = w.allocs[c.alloc]
        off = w.data_offset(c.alloc)
        return cosine_expected(a.dtype, a.rows, a.cols, a.stride, a.stride, cand, ref, off, off)
    with ThreadPoolExecutor(threads) as ex:
        pairs = list(ex.map(one, w.compares))
    return [p[0] for p in pairs], [p[1] for p in pairs], [w.allocs[c.alloc].dtype for c in w.compares]
