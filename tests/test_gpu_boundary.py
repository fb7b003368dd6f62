"""GPU parity of the BOUNDARY fill distribution (boundary values at a rate:
signed zeros, subnormals, +-max, infinities, NaNs, integer extremes) on every
element type and odd geometries, with injections acting on boundary values,
and of the comparison over such data under both NaN policies."""
import numpy as np
import pytest

import oracle
from gpu_helpers import THREADS, assert_fill_equal, assert_results_equal, log, run_gpu
from workloads import Alloc, Compare, Injection, Workload

pytestmark = pytest.mark.gpu

FLOATS = ("f32", "bf16", "f16", "fp8e4m3")


def _boundary_workload(seed=0xB0DA):
    specs = [  # dtype, rows, cols, stride, guard_lo, guard_hi, rate, sigma
        ("f32", 1, 70_001, 70_001, 64, 48, 0.3, 1.0),
        ("bf16", 37, 1001, 1040, 16, 0, 0.05, 8.0),
        ("f16", 5, 9999, 10_003, 0, 32, 1.0, 1.0),
        ("fp8e4m3", 3, 40_000, 40_017, 7, 9, 0.2, 2.0),
        ("i32", 11, 777, 780, 12, 4, 0.5, 1.0),
        ("i64", 1, 20_000, 20_000, 8, 8, 0.25, 1.0),
        ("u8", 7, 3333, 3340, 3, 5, 0.0, 1.0),
    ]
    allocs = [Alloc(40 + k, dt, r, c, s, gl, gh, "boundary", rate, sig, saturate=(dt == "fp8e4m3"))
              for k, (dt, r, c, s, gl, gh, rate, sig) in enumerate(specs)]
    rng = np.random.default_rng(seed)
    inj, cmp_ = [], []
    for k, a in enumerate(allocs):
        inj.append(Injection(k, "flip_bit", arg=-1, rate=0.01))
        if a.dtype in FLOATS:
            inj.append(Injection(k, "step_within", rate=0.005, atol=1e-3, rtol=1e-3))
            inj.append(Injection(k, "set_beyond", rate=0.005, atol=1e-3, rtol=1e-3))
            for i in rng.integers(0, a.n_elements, size=8):
                inj.append(Injection(k, "set_nan", index=int(i)))
            if a.dtype != "fp8e4m3":
                inj.append(Injection(k, "set_inf", arg=1, rate=0.002))
            cmp_.append(Compare(k, "tolerance", "equal", 1e-3, 1e-3))
            cmp_.append(Compare(k, "tolerance", "strict", 1e-3, 1e-3))
        else:
            cmp_.append(Compare(k, "bitwise"))
        if a.guard_hi:
            inj.append(Injection(k, "guard_write_hi", arg=1, index=int(rng.integers(0, a.guard_hi))))
    return Workload("boundary_mix", "boundary values on every dtype", seed, allocs, inj, cmp_)


def test_boundary_fill_diff_guard_parity():
    w = _boundary_workload()
    log(f"boundary_mix: {len(w.allocs)} allocs, {len(w.injections)} injections, arena {w.arena_bytes} B")
    P = oracle.Prepared(w)
    for variant in (1, 3):
        st = run_gpu(w, variant)
        ref = P.fill_arena(0, THREADS)
        cand = P.fill_arena(variant, THREADS)
        assert_fill_equal(w, st.arena_host("ref"), ref, "reference")
        assert_fill_equal(w, st.arena_host("cand"), cand, f"candidate {variant}")
        assert_results_equal(st.seg_results(), oracle.diff_workload(w, cand, ref, THREADS), f"diff v{variant}")
        assert_results_equal(st.guard_results(), oracle.guard_workload(w, cand), f"guard v{variant}")
        res = st.seg_results()
        assert all(r["mismatches"] > 0 for r in res)
