"""Tier-2 replay of a captured state in another process (section 3.4: the
captured pre-dispatch state holds absolute device pointers, so the replay
needs its memory back at the same addresses).  One child process builds a
state in memory mapped by asmevo_va_alloc at an explicit address, with a
first page of absolute pointers into the state, snapshots it to the host and
exits; a second child maps the same address range, restores the bytes, and
diffs the data each captured pointer points to (used as the segment address)
against the snapshot.

Explicit device addresses were honoured only while no other process held
the device, so this test runs before every other test of a session
(tests/conftest.py moves it to the front whatever the selection or order)
and is skipped when the test process already uses the GPU, or when the
capture process cannot map any of the candidate addresses."""
import json
import os
import subprocess
import sys

import pytest
import torch

import paper_2608_20711_amd as lib

pytestmark = pytest.mark.gpu

_CAPTURE = r"""
import json, sys
import numpy as np
import paper_2608_20711_amd as lib
size, path = int(sys.argv[1]), sys.argv[2]
gran = lib.va_granularity()
size = -(-size // gran) * gran if gran else size
a = None
for hint in (0x4E0000000000, 0x4C0000000000, 0x300000000000):
    try:                                  # an explicit address, away from the runtime's own
        a = lib.va_alloc(size, hint)
        break
    except lib.AsmevoError:
        pass
if a is None:
    print(json.dumps({"addr": None, "size": size}), flush=True)
    sys.exit(0)
import torch
rng = np.random.default_rng(0xADD2)
host = rng.integers(0, 256, size=size, dtype=np.uint8)
ptrs = a + 4096 + 16384 * rng.permutation(256).astype(np.uint64)
host[:4096] = 0
host[:256 * 8] = ptrs.astype(np.uint64).view(np.uint8)   # page 0: absolute pointers into the state
src = torch.from_numpy(host).cuda()
ws_size = lib.workspace_bytes(4)
ws = torch.empty(ws_size, dtype=torch.uint8, device="cuda")
lib.copy_regions([lib.Region(a, src.data_ptr(), size)], ws.data_ptr(), ws_size)
snap = torch.empty_like(src)
lib.copy_regions([lib.Region(snap.data_ptr(), a, size)], ws.data_ptr(), ws_size)
torch.cuda.synchronize()
np.save(path, snap.cpu().numpy())
lib.va_free(a)
print(json.dumps({"addr": a, "size": size}), flush=True)
"""

_REPLAY = r"""
import json, sys
import numpy as np
import paper_2608_20711_amd as lib
addr, size, path = int(sys.argv[1]), int(sys.argv[2]), sys.argv[3]
try:
    got = lib.va_alloc(size, addr)        # the first device allocation of this process
except lib.AsmevoError as e:
    print(json.dumps({"addr": None, "status": e.status}), flush=True)
    sys.exit(0)
import torch
host = np.load(path)
state = torch.from_numpy(host).cuda()
ws_size = lib.workspace_bytes(300)
ws = torch.empty(ws_size, dtype=torch.uint8, device="cuda")
lib.copy_regions([lib.Region(got, state.data_ptr(), size)], ws.data_ptr(), ws_size)
ptrs = host[:4096].view(np.uint64)
segs = [lib.Segment(int(p), state.data_ptr() + int(p) - got, lib.U8, lib.BITWISE, 0, 0, 1, 16384, 16384, 16384,
                    0.0, 0.0) for p in ptrs[:256]]
segs.append(lib.Segment(got + 4096, state.data_ptr() + 4097, lib.U8, lib.BITWISE, 0, 0, 1, 4096, 4096, 4096,
                        0.0, 0.0))        # control: shifted by one byte, must differ
from paper_2608_20711_amd.state import SEG_RESULT_DTYPE as RES
res = torch.empty(len(segs) * RES.itemsize, dtype=torch.uint8, device="cuda")
lib.diff_segments(segs, res.data_ptr(), ws.data_ptr(), ws_size)
torch.cuda.synchronize()
raw = res.cpu().numpy().view(RES)
print(json.dumps({"addr": got, "in_range": bool(((ptrs[:256] >= got) & (ptrs[:256] < got + size)).all()),
                  "mismatches": [int(x) for x in raw["bitwise_mismatches"][:256]],
                  "control": int(raw["bitwise_mismatches"][256])}), flush=True)
lib.va_free(got)
"""


def _child(src, *args):
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = subprocess.run([sys.executable, "-c", src, *map(str, args)], capture_output=True, text=True,
                         timeout=240, cwd=root)
    assert out.returncode == 0, out.stderr[-2000:]
    return json.loads(out.stdout.strip().splitlines()[-1])


def test_state_replayed_at_its_addresses_in_another_process(tmp_path):
    if torch.cuda.is_initialized() or lib._handle is not None:
        pytest.skip("this process already uses the GPU: explicit device addresses are honoured only "
                    "while no other process holds the device")
    path = str(tmp_path / "state.npy")
    cap = _child(_CAPTURE, 4096 + 256 * 16384, path)   # rounded up to the granularity there
    if cap["addr"] is None:
        pytest.skip("no candidate address could be mapped in a fresh process")
    a, size = cap["addr"], cap["size"]
    rec = _child(_REPLAY, a, size, path)
    if rec["addr"] is None:
        pytest.skip(f"the replay process could not map {a:#x} (status {rec['status']}): another process "
                    "may hold the device")
    assert rec["addr"] == a and rec["in_range"]
    assert rec["mismatches"] == [0] * 256
    assert rec["control"] > 0
