"""Staged plans (asmevo_plan_diff / asmevo_plan_guard, then the planned
launches): a check planned once and launched for several candidates in a
row -- the state refilled in place between them, as Algorithm 1 checks every
input of every candidate and section 4.1 repeats each check three times --
gives exactly the results of the unplanned calls on the same bytes, and of
the oracle."""
import pytest
import torch

import oracle
import workloads
from gpu_helpers import THREADS, assert_results_equal, log
from paper_2608_20711_amd.state import DeviceState

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,small", [(n, True) for n in workloads.ALL] + [("decode_state", False)])
def test_planned_checks_equal_unplanned(name, small):
    w = workloads.ALL[name](small=small)
    log(f"[plans] {name} small={small}")
    st = DeviceState(w)
    st.fill("ref", 0)
    st.fill("cand", 1)
    st.plan()
    for variant in (1, 2, 3, 2):
        st.fill("cand", variant)
        st.diff_planned()
        st.guard_planned()
        planned = (st.seg_results(), st.guard_results())
        st.diff()
        st.guard()
        assert_results_equal(planned[0], st.seg_results(), f"{name} planned diff, variant {variant}")
        assert_results_equal(planned[1], st.guard_results(), f"{name} planned guard, variant {variant}")
        if small:
            cand, ref = st.arena_host("cand"), st.arena_host("ref")
            assert_results_equal(planned[0], oracle.diff_workload(w, cand, ref, THREADS), f"{name} v{variant}")
            assert_results_equal(planned[1], oracle.guard_workload(w, cand), f"{name} guards v{variant}")
    torch.cuda.synchronize()


def test_planned_nd_block_table_equals_unplanned():
    """A paged cache as N-D segments (one per block, two sequences sharing
    results), planned once and checked after three in-place edits of the
    candidate: results equal asmevo_diff_segments_nd's on the same bytes."""
    import numpy as np
    import paper_2608_20711_amd as lib
    from paper_2608_20711_amd.state import SEG_RESULT_DTYPE
    rng = np.random.default_rng(40)
    n_phys, blk, width = 64, 16, 128
    b = torch.from_numpy(rng.standard_normal((n_phys, blk, width)).astype(np.float16)).cuda()
    a = b.clone()
    order = rng.permutation(n_phys)
    seqs = [order[:30].tolist(), order[30:62].tolist()]
    segs = []
    for r, table in enumerate(seqs):
        for j, p in enumerate(table):
            off = p * blk * width * 2
            segs.append(lib.segment_nd(a.data_ptr() + off, b.data_ptr() + off, lib.F16, lib.TOLERANCE,
                                       lib.NAN_EQUAL, [blk, width], [width, 1], [width, 1], 1e-3, 1e-3, r,
                                       j * blk * width))
    size = lib.plan_bytes(len(segs))
    ws = torch.empty(size, dtype=torch.uint8, device="cuda")
    plan = lib.plan_diff_nd(segs, 2, ws.data_ptr(), size)
    uws_size = lib.diff_nd_workspace_bytes(len(segs))
    uws = torch.empty(uws_size, dtype=torch.uint8, device="cuda")
    got = torch.empty(2 * SEG_RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    want = torch.empty_like(got)
    flat = a.view(-1)
    for step in range(3):
        idx = torch.from_numpy(rng.integers(0, flat.numel(), size=50 * (step + 1))).cuda()
        flat[idx] = flat[idx] + 0.5
        lib.diff_planned(plan, got.data_ptr())
        lib.diff_segments_nd(segs, want.data_ptr(), 2, uws.data_ptr(), uws_size)
        torch.cuda.synchronize()
        g = got.cpu().numpy().view(SEG_RESULT_DTYPE)
        w = want.cpu().numpy().view(SEG_RESULT_DTYPE)
        assert g.tobytes() == w.tobytes(), f"step {step}"
        assert int(w["mismatches"].sum()) > 0
