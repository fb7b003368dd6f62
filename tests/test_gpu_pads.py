"""GPU parity of the row-pad canaries (interior guards between the rows of a
strided allocation): pad-write injections on every element size, pads that
are not 16-byte aligned or shorter than a chunk, runs longer than several
chunks, and the guard check's pad counts and first offsets against the
oracle's."""
import numpy as np
import pytest

import oracle
from gpu_helpers import THREADS, assert_fill_equal, assert_results_equal, log, run_gpu
from workloads import Alloc, Injection, Workload

pytestmark = pytest.mark.gpu


def _pad_workload(seed=0x9AD5):
    specs = [  # dtype, rows, cols, stride, guard_lo, guard_hi
        ("f32", 33, 1000, 1003, 16, 16),       # 12-byte pads, unaligned
        ("bf16", 17, 300, 400, 0, 0),          # 200-byte pads: 13 chunks per run
        ("u8", 101, 17, 18, 5, 3),             # 1-byte pads
        ("i64", 9, 5, 40, 8, 8),               # 280-byte pads, pitch 320
        ("fp8e4m3", 65, 4096, 4111, 0, 16),    # 15-byte pads
        ("f16", 2, 64, 72, 32, 0),             # one run
        ("i32", 1, 100, 120, 0, 4),            # one row: no padding at all
        ("f32", 5, 0, 8, 16, 16),              # no columns: no data, no padding
    ]
    allocs = [Alloc(60 + k, dt, r, c, s, gl, gh, "normal" if dt in ("f32", "bf16", "f16", "fp8e4m3") else "bits",
                    saturate=dt == "fp8e4m3")
              for k, (dt, r, c, s, gl, gh) in enumerate(specs)]
    rng = np.random.default_rng(seed)
    inj = []
    for k, a in enumerate(allocs):
        if a.rows < 2 or a.cols == 0 or a.stride == a.cols:
            continue
        pitch, row_data = a.stride * a.esize, a.cols * a.esize
        plen = pitch - row_data
        for _ in range(3):
            r = int(rng.integers(0, a.rows - 1))
            off = int(rng.integers(0, plen))
            n = int(rng.integers(1, plen - off + 1))
            inj.append(Injection(k, "pad_write", arg=n, index=r * pitch + row_data + off))
        # one that both sides carry (reference corrupted too) and a whole run
        inj.append(Injection(k, "pad_write", sides="both", arg=1, index=(a.rows - 2) * pitch + pitch - 1))
        inj.append(Injection(k, "pad_write", arg=plen, index=row_data))
        inj.append(Injection(k, "flip_bit", arg=-1, rate=0.01))
    return Workload("pads", "row-pad canaries", seed, allocs, inj, [])


def test_pad_canaries_fill_and_check_parity():
    w = _pad_workload()
    log(f"pads: {len(w.allocs)} allocs, {len(w.injections)} injections, arena {w.arena_bytes} B")
    P = oracle.Prepared(w)
    for variant in (1, 2):
        st = run_gpu(w, variant)
        ref = P.fill_arena(0, THREADS)
        cand = P.fill_arena(variant, THREADS)
        assert_fill_equal(w, st.arena_host("ref"), ref, "reference")
        assert_fill_equal(w, st.arena_host("cand"), cand, f"candidate {variant}")
        want = oracle.guard_workload(w, cand)
        assert_results_equal(st.guard_results(), want, f"guard v{variant}")
        padded = [k for k, a in enumerate(w.allocs) if a.rows >= 2 and 0 < a.cols < a.stride]
        assert all(want[k]["bad_pad"] > 0 for k in padded)
        assert all(want[k]["bad_pad"] == 0 for k in range(len(w.allocs)) if k not in padded)


def test_pad_check_of_an_intact_state_and_of_the_reference():
    w = _pad_workload(seed=0x9AD6)
    st = run_gpu(w, 1)
    # re-check the reference arena too: only the 'both' pad writes show
    from paper_2608_20711_amd import guard_check
    st.guard_res.zero_()
    guard_check(st.allocs_ref, w.seed, st.guard_res.data_ptr(), st.ws.data_ptr(), st.ws_size)
    got = st.guard_results()
    want = oracle.guard_workload(w, oracle.Prepared(w).fill_arena(0, THREADS))
    assert_results_equal(got, want, "reference guards")
    assert all(g["bad_pad"] in (0, 1) for g in got)
