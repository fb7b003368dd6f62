"""The allocation-free diff (asmevo_diff_segments_noalloc), for callers that
cannot allocate device memory: its descriptor table lives in the library's
static device array.  Two calls in a row through the C ABI, the second with
fewer and smaller segments, each against asmevo_diff_segments (the entry
point with a workspace) on the same operands, bit for bit on every result
field.  This file runs last in a session (tests/conftest.py)."""
import numpy as np
import pytest
import torch

import paper_2608_20711_amd as lib
from gpu_helpers import assert_results_equal, log
from paper_2608_20711_amd.state import SEG_RESULT_DTYPE

pytestmark = pytest.mark.gpu

_DT = ["f32", "bf16", "f16", "fp8e4m3", "i32", "i64", "u8"]
_ES = {"f32": 4, "bf16": 2, "f16": 2, "fp8e4m3": 1, "i32": 4, "i64": 8, "u8": 1}


def _operands(nbytes, rng):
    b = rng.integers(0, 256, size=nbytes, dtype=np.uint8)
    vals = (rng.standard_normal(nbytes // 4) * 3).astype(np.float32).view(np.uint8)
    b[: vals.size] = np.where(rng.random(vals.size) < 0.9, vals, b[: vals.size])
    a = b.copy()
    k = rng.integers(0, nbytes, size=nbytes // 2000)
    a[k] ^= (1 << rng.integers(0, 8, size=k.size)).astype(np.uint8)
    return torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()


def _segments(a_d, b_d, n, max_bytes, rng):
    nbytes = a_d.numel()
    segs = []
    for k in range(n):
        dt = _DT[k % len(_DT)]
        es = _ES[dt]
        rows = int(rng.choice([1, 1, 3, 17]))
        cols = int(rng.integers(1, max(2, max_bytes // (es * rows))))
        pad = int(rng.choice([0, 0, 1, 9]))
        stride = cols + pad
        ext = ((rows - 1) * stride + cols) * es
        off = int(rng.integers(0, (nbytes - ext) // es)) * es
        assert off + ext <= nbytes
        tol = dt in ("f32", "bf16", "f16", "fp8e4m3")
        segs.append(lib.Segment(a_d.data_ptr() + off, b_d.data_ptr() + off, lib.DTYPE_CODE[dt],
                                lib.TOLERANCE if tol else lib.BITWISE, int(k % 2 and tol), 0, rows, cols,
                                stride, stride, 1e-3 if tol else 0.0, 1e-3 if tol else 0.0))
    return segs


def _results(buf, n):
    raw = buf.cpu().numpy()[: n * SEG_RESULT_DTYPE.itemsize].view(SEG_RESULT_DTYPE)
    return [{f: raw[f][k].item() for f in SEG_RESULT_DTYPE.names} for k in range(n)]


def test_noalloc_diff_equals_workspace_diff_twice():
    rng = np.random.default_rng(0x0A110C)
    a_d, b_d = _operands(64 << 20, rng)
    for n, max_bytes in ((lib.NOALLOC_MAX_SEGMENTS, 96 << 10), (300, 16 << 10)):
        segs = _segments(a_d, b_d, n, max_bytes, rng)
        log(f"[noalloc] {n} segments")
        got = torch.full((n * SEG_RESULT_DTYPE.itemsize,), 0xEE, dtype=torch.uint8, device="cuda")
        want = torch.full_like(got, 0x11)
        lib.diff_segments_noalloc(segs, got.data_ptr())
        ws_size = lib.workspace_bytes(n)
        ws = torch.empty(ws_size, dtype=torch.uint8, device="cuda")
        lib.diff_segments(segs, want.data_ptr(), ws.data_ptr(), ws_size)
        torch.cuda.synchronize()
        g, w = _results(got, n), _results(want, n)
        assert_results_equal(g, w, f"noalloc n={n}")
        assert sum(r["bitwise_mismatches"] for r in w) > 0
