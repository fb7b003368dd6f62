"""GPU parity on the five seeded workloads: the HIP fill, diff and guard check
against the CPU oracle, bit for bit on every output (fill bytes, counts,
first indices, fp64 maxima, guard counts and offsets).

Reduced sizes check every byte and every result.  Full sizes check every
comparison and guard result against the oracle run on the GPU's own buffers
and every fill byte against the oracle's fill; the 4096-buffer sweep (64 GiB
per side) checks every comparison and guard result the same way, and the
fill bytes of a stratified sample of whole allocations."""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import THREADS, assert_fill_equal, assert_results_equal, log, run_gpu

INTACT = {"bad_lo": 0, "bad_hi": 0, "first_bad_lo": -1, "first_bad_hi": -1, "bad_pad": 0,
          "first_bad_pad": -1}

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", list(workloads.ALL))
def test_reduced_size_everything_bit_exact(name):
    w = workloads.ALL[name](small=True)
    log(f"[reduced] {name}: {len(w.allocs)} allocs, {w.arena_bytes} B per side")
    st = run_gpu(w)
    P = oracle.Prepared(w)
    ref = P.fill_arena(0, THREADS)
    cand = P.fill_arena(1, THREADS)
    assert_fill_equal(w, st.arena_host("ref"), ref, f"{name} reference fill")
    assert_fill_equal(w, st.arena_host("cand"), cand, f"{name} candidate fill")
    assert_results_equal(st.seg_results(), oracle.diff_workload(w, cand, ref, THREADS), f"{name} diff")
    assert_results_equal(st.guard_results(), oracle.guard_workload(w, cand), f"{name} guard")


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["single_fp32", "padded_bf16", "decode_state", "int_lowp"])
def test_full_size_bit_exact(name):
    w = workloads.ALL[name]()
    log(f"[full] {name}: {w.arena_bytes} B per side")
    st = run_gpu(w)
    cand = st.arena_host("cand")
    ref = st.arena_host("ref")
    # every comparison / guard result against the oracle on the same bytes
    assert_results_equal(st.seg_results(), oracle.diff_workload(w, cand, ref, THREADS), f"{name} diff")
    assert_results_equal(st.guard_results(), oracle.guard_workload(w, cand), f"{name} guard")
    # the fills themselves: every byte of every allocation, both sides
    P = oracle.Prepared(w)
    assert_fill_equal(w, ref, P.fill_arena(0, THREADS), f"{name} reference fill")
    assert_fill_equal(w, cand, P.fill_arena(1, THREADS), f"{name} candidate fill")
    del cand, ref


def _fill_sample(w, rng):
    """A stratified sample of the sweep's allocations: for every element type,
    one allocation from each tenth of its size range (sorted by size)."""
    picks = []
    for dt in sorted({a.dtype for a in w.allocs}):
        ks = sorted((k for k, a in enumerate(w.allocs) if a.dtype == dt), key=lambda k: w.allocs[k].total_bytes)
        for part in np.array_split(np.array(ks), 10):
            if part.size:
                picks.append(int(rng.choice(part)))
    return set(picks)


@pytest.mark.timeout(900)
def test_sweep_full_size_every_result_bit_exact():
    """4096 buffers, ~64 GiB per side, in the launch configuration the bench
    times.  Every segment result and every guard result bit-exact against the
    oracle run on the GPU's own buffers (streamed one allocation at a time by
    THREADS workers); every differing element a single-bit flip, their count
    consistent with the 1e-6 rate; whole-allocation fill bytes of both sides
    against the oracle's fill for a stratified sample (every element type x
    every tenth of its size range)."""
    from concurrent.futures import ThreadPoolExecutor
    w = workloads.sweep()
    free, total = torch.cuda.mem_get_info()
    need = 2 * w.arena_bytes + (1 << 30)
    if free < need:
        pytest.skip(f"needs {need >> 30} GiB of free device memory, {free >> 30} GiB free")
    log(f"[sweep] {len(w.allocs)} buffers, {w.arena_bytes / 2**30:.1f} GiB per side")
    st = run_gpu(w)
    res = st.seg_results()
    guards = st.guard_results()
    P = oracle.Prepared(w)
    sample = _fill_sample(w, np.random.default_rng(5))

    def one(k):
        a = w.allocs[k]
        c = w.compares[k]
        cand_k = st.alloc_bytes("cand", k)
        ref_k = st.alloc_bytes("ref", k)
        lo, hi = a.guard_lo, a.guard_lo + a.data_bytes
        d = oracle.diff_segment(a.dtype, c.mode, c.nan_policy, a.rows, a.cols, a.stride, a.stride,
                                c.atol, c.rtol, cand_k, ref_k, lo, lo)
        g = oracle.guard_check(w.seed, a.alloc_id, cand_k[:lo], cand_k[hi:])
        g.update(oracle.pad_check_alloc(w.seed, a.alloc_id, a.dtype, a.rows, a.cols, a.stride, cand_k[lo:hi]))
        # every element whose bytes differ differs in exactly one bit
        diff_at = np.flatnonzero(cand_k[lo:hi] != ref_k[lo:hi])
        elems = np.unique(diff_at // a.esize)
        flips_ok = True
        for e in elems:
            x = cand_k[lo + e * a.esize: lo + (e + 1) * a.esize] ^ ref_k[lo + e * a.esize: lo + (e + 1) * a.esize]
            flips_ok = flips_ok and int(np.unpackbits(x).sum()) == 1
        fills = None
        if k in sample:
            fills = (np.array_equal(cand_k, P.fill_alloc(k, 1, 4)), np.array_equal(ref_k, P.fill_alloc(k, 0, 4)))
        return k, d, g, elems.size, flips_ok, fills

    done = 0
    n_el = sum(a.n_elements for a in w.allocs)
    flips = 0
    with ThreadPoolExecutor(THREADS) as ex:
        for k, d, g, n_diff, flips_ok, fills in ex.map(one, range(len(w.allocs))):
            a = w.allocs[k]
            assert_results_equal([res[k]], [d], f"sweep segment {k} ({a.dtype}, {a.data_bytes} B)")
            assert_results_equal([guards[k]], [g], f"sweep guards {k}")
            assert guards[k] == INTACT
            assert flips_ok, f"sweep segment {k}: a differing element is not a single-bit flip"
            assert n_diff == res[k]["bitwise_mismatches"]
            if fills is not None:
                assert fills == (True, True), f"sweep fill of allocation {k} ({a.dtype}, {a.total_bytes} B)"
            flips += n_diff
            done += 1
            if done % 128 == 0:
                log(f"  {done} of {len(w.allocs)} allocations checked")
    assert abs(flips - 1e-6 * n_el) < 6 * math.sqrt(1e-6 * n_el)
    log(f"[sweep] every result equal; {flips} flips; fills of {len(sample)} whole allocations equal")
    del st
    torch.cuda.empty_cache()


def test_repeats_and_launch_geometry_are_bit_identical():
    """The check is repeated three times per candidate (section 4.1); results
    must not depend on repetition or on the number of workgroups."""
    w = workloads.padded_bf16(small=True)
    st = run_gpu(w)
    base = st.seg_results()
    for rep in range(3):
        st.diff()
        assert st.seg_results() == base
    for wg in (1, 2, 3, 17, 64, 1000, 4096):
        st.diff(workgroups=wg)
        assert st.seg_results() == base, f"workgroups={wg}"
