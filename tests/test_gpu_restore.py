"""GPU parity of the Tier-2 state restore (asmevo_copy_regions): random
regions with every address phase against the oracle's byte copy, and a
snapshot -> candidate run -> restore replay whose diff against the reference
repeats the original result."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_20711_amd as lib
import workloads
from gpu_helpers import assert_bytes_equal, assert_results_equal, run_gpu

pytestmark = pytest.mark.gpu


def _copy(regions, buf_dev):
    ws_size = lib.workspace_bytes(max(1, len(regions)))
    ws = torch.empty(ws_size, dtype=torch.uint8, device="cuda")
    base = buf_dev.data_ptr()
    for d, s, n in regions:
        assert 0 <= d and d + n <= buf_dev.numel() and 0 <= s and s + n <= buf_dev.numel()
    lib.copy_regions([lib.Region(base + d, base + s, n) for d, s, n in regions], ws.data_ptr(), ws_size)
    torch.cuda.synchronize()


def test_copy_regions_random_phases_and_sizes():
    rng = np.random.default_rng(21)
    size = 48 << 20
    half = size // 2
    regions, dst = [], half
    for k in range(400):
        n = int(rng.choice([0, 1, 15, 16, 17, 4095, 4096, 4097]) if k < 40 else
                rng.integers(1, 1 << int(rng.integers(1, 18))))
        dst += int(rng.integers(0, 64))
        if dst + n > size:
            break
        src = int(rng.integers(0, half - n))
        regions.append((dst, src, n))
        dst += n
    host = rng.integers(0, 256, size=size, dtype=np.uint8)
    dev = torch.from_numpy(host.copy()).cuda()
    _copy(regions, dev)
    want = host.copy()
    oracle.copy_regions(want, regions)
    assert_bytes_equal(dev.cpu().numpy(), want, "copy_regions")
    # phases: both aligned, same phase, different phases all occurred
    phases = {((d % 16) == (s % 16), d % 16 == 0) for d, s, n in regions if n}
    assert len(phases) >= 3


def test_snapshot_restore_replay():
    w = workloads.sweep(small=True)
    st = run_gpu(w)                       # reference + candidate 1, diffed
    first = st.seg_results()
    before = st.arena_host("cand")
    backup = torch.empty_like(st.cand)
    regions = [(st.w.offsets[k], a.total_bytes) for k, a in enumerate(w.allocs)]
    ws = torch.empty(lib.workspace_bytes(len(regions)), dtype=torch.uint8, device="cuda")
    snap = [lib.Region(backup.data_ptr() + o, st.cand.data_ptr() + o, n) for o, n in regions]
    rest = [lib.Region(st.cand.data_ptr() + o, backup.data_ptr() + o, n) for o, n in regions]
    lib.copy_regions(snap, ws.data_ptr(), ws.numel())
    st.fill("cand", 9)                    # another candidate overwrites the state
    st.diff()
    assert st.seg_results() != first
    lib.copy_regions(rest, ws.data_ptr(), ws.numel())
    st.diff()
    assert_results_equal(st.seg_results(), first, "diff after restore")
    after = st.arena_host("cand")
    for o, n in regions:
        assert_bytes_equal(after[o:o + n], before[o:o + n], f"region at {o}")


def test_va_alloc_in_use_and_again():
    """A range handed out by asmevo_va_alloc cannot be requested while it is
    live, and can be requested again, at the same address, once freed."""
    gran = lib.va_granularity()
    assert gran > 0, "the device has no virtual memory management"
    size = 64 * gran
    a = lib.va_alloc(size)
    assert a % gran == 0
    with pytest.raises(lib.AsmevoError) as e:
        lib.va_alloc(size, a)
    assert e.value.status == lib.E_UNSUPPORTED
    lib.va_free(a)
    assert lib.va_alloc(size, a) == a
    # the range is usable memory: a pattern copied in comes back out
    pattern = torch.from_numpy(np.random.default_rng(5).integers(0, 256, size=size, dtype=np.uint8)).cuda()
    back = torch.empty_like(pattern)
    ws_size = lib.workspace_bytes(1)
    ws = torch.empty(ws_size, dtype=torch.uint8, device="cuda")
    lib.copy_regions([lib.Region(a, pattern.data_ptr(), size)], ws.data_ptr(), ws_size)
    lib.copy_regions([lib.Region(back.data_ptr(), a, size)], ws.data_ptr(), ws_size)
    torch.cuda.synchronize()
    assert torch.equal(back, pattern)
    lib.va_free(a)
    with pytest.raises(lib.AsmevoError):
        lib.va_free(a)

