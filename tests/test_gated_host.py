"""Host side of the gated verification harness (paper section 3.7, Algorithm
1; Eq. 2): the build and static-consistency gates on every candidate (no GPU
needed), the code-object metadata reader, and the commit gate pinned by
hand-computed cases of Eq. 2 with the paper's epsilon = 0.002, k = 0.85,
s_floor = 1.0 (section 4.1)."""
import math
import os

import pytest

from paper_2608_20711_amd.gated import candidates as C
from paper_2608_20711_amd.gated import toolchain

HARNESS_OK = True
try:
    from paper_2608_20711_amd.gated.harness import commit_gate, static_consistent, KERNEL
except ImportError:          # torch missing: not the case in this image
    HARNESS_OK = False


@pytest.fixture(scope="module")
def sources():
    s0 = toolchain.load_assembly(toolchain.K0_SOURCE)
    s1 = toolchain.load_assembly(toolchain.K1_SOURCE)
    return s0, s1


@pytest.fixture(scope="module")
def k0(sources):
    b = toolchain.build(sources[0])
    assert b.ok, b.log
    return b.code_object


def test_k0_metadata(k0):
    assert toolchain.metadata(k0)["amdhsa.target"] == "amdgcn-amd-amdhsa--gfx950"
    assert toolchain.kernel_names(k0) == ["rmsnorm_k0"]
    m = toolchain.kernel_metadata(k0, "rmsnorm_k0")
    # 7 pointers and 3 ints, as the source declares them
    args = [(a[".offset"], a[".size"], a[".value_kind"]) for a in m[".args"]]
    assert args == [(8 * k, 8, "global_buffer") for k in range(7)] + [(56, 4, "by_value"), (60, 4, "by_value"),
                                                                     (64, 4, "by_value")]
    assert m[".kernarg_segment_size"] == 68 and m[".wavefront_size"] == 64
    assert m[".max_flat_workgroup_size"] == 256
    assert m[".group_segment_fixed_size"] == 3 * 256 * 4       # three 256-entry LDS arrays


def test_assembly_round_trip_is_stable(sources, k0):
    """Assembling s(K0) twice gives the same code object (the build is deterministic)."""
    again = toolchain.build(sources[0])
    assert again.ok and again.code_object == k0


@pytest.mark.skipif(not HARNESS_OK, reason="harness import failed")
@pytest.mark.parametrize("cand", C.CANDIDATES, ids=[c.name for c in C.CANDIDATES])
def test_build_and_static_gates(cand, sources, k0):
    s = cand.make(*sources)
    b = toolchain.build(s)
    if cand.expect == "asm_invalid":
        assert not b.ok and b.stage == "assemble" and "error" in b.log
        return
    assert b.ok, b.log
    bad = static_consistent(toolchain.kernel_metadata(b.code_object, KERNEL),
                            toolchain.kernel_metadata(k0, KERNEL))
    if cand.expect == "abi_invalid":
        assert bad, cand.name
    else:
        assert bad == [], (cand.name, bad)
    if cand.name not in ("k0_roundtrip", "k1_vectorized"):
        assert s != sources[0]                  # the edit changed the text


def test_edits_touch_one_line_each(sources):
    s0, s1 = sources
    for name in ("eps_constant", "out_store_shift", "amax_lds_slot"):
        cand = next(c for c in C.CANDIDATES if c.name == name)
        a, b = s0.split("\n"), cand.make(s0, s1).split("\n")
        assert len(a) == len(b)
        assert sum(x != y for x, y in zip(a, b)) == 1, name


@pytest.mark.skipif(not HARNESS_OK, reason="harness import failed")
def test_commit_gate_hand_computed_cases():
    # epsilon dominates: k * cv = 0.85 * 0.001 = 0.00085 < 0.002, bar = 1.002 * s_best
    ok, bar = commit_gate(True, 1.25, 1.0, 0.001)
    assert ok and bar == 1.0 + 0.002
    assert commit_gate(True, 1.0019, 1.0, 0.001) == (False, 1.002)
    # k * cv dominates: cv = 0.04 -> margin 0.034, bar = 1.034 * 1.5 = 1.551
    ok, bar = commit_gate(True, 1.56, 1.5, 0.04)
    assert ok and math.isclose(bar, 1.551, rel_tol=0, abs_tol=1e-12)
    assert not commit_gate(True, 1.55, 1.5, 0.04)[0]
    # the floor: a best below 1 / 1.002 still needs s_hat >= 1
    ok, bar = commit_gate(True, 0.999, 0.9, 0.0)
    assert not ok and bar == 1.0
    assert commit_gate(True, 1.0, 0.9, 0.0) == (True, 1.0)
    # equality commits (>=); failed equivalence never commits
    ok, bar = commit_gate(True, (1.0 + 0.002) * 1.25, 1.25, 0.0)
    assert ok
    assert not commit_gate(False, 10.0, 1.0, 0.0)[0]
    # the margin grows with the measured variation (variance-aware)
    bars = [commit_gate(True, 2.0, 1.0, cv)[1] for cv in (0.0, 0.002, 0.01, 0.1)]
    assert bars == sorted(bars) and bars[0] == bars[1] == 1.002 and bars[-1] == 1.0 + 0.085
