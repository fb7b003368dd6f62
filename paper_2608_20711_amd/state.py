"""Device-resident candidate / reference states of one workload.

Holds the two arenas (torch uint8 tensors in HBM), the workspace and the
result buffers, and turns a workloads.Workload description into the C-ABI
descriptor structs with device addresses.  torch is used only for device
memory and streams; all work runs in libasmevo.so.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np
import torch

from . import (Alloc, DIST_CODE, diff_planned, guard_planned, plan_bytes, plan_diff, plan_guard, DTYPE_CODE, FILL_SATURATE, Injection, KIND_CODE, MODE_CODE,
               NAN_CODE, INJ_RATE, SIDE_CODE, Segment, descriptor_array, diff_cosine,
               diff_cosine_workspace_bytes, diff_segments, fill_guarded, guard_check, workspace_bytes)

SEG_RESULT_DTYPE = np.dtype([("mismatches", "<u8"), ("first_mismatch", "<i8"),
                             ("bitwise_mismatches", "<u8"), ("first_bitwise", "<i8"),
                             ("nonfinite_mismatches", "<u8"), ("max_abs", "<f8"), ("max_rel", "<f8")])
COS_RESULT_DTYPE = np.dtype([("sum_ab", "<f8"), ("sum_aa", "<f8"), ("sum_bb", "<f8"), ("cosine", "<f8"),
                             ("pairs", "<u8"), ("blocks", "<u8")])
GUARD_RESULT_DTYPE = np.dtype([("bad_lo", "<u8"), ("bad_hi", "<u8"),
                               ("first_bad_lo", "<i8"), ("first_bad_hi", "<i8"),
                               ("bad_pad", "<u8"), ("first_bad_pad", "<i8")])


def injection_structs(w) -> List[Injection]:
    from workloads import rate_threshold
    out = []
    for j in w.injections:
        kind = KIND_CODE[j.kind]
        index = j.index
        if j.rate is not None:
            kind |= INJ_RATE
            index = rate_threshold(j.rate)
        out.append(Injection(j.alloc, kind, SIDE_CODE[j.sides], j.arg & 0xFFFFFFFF, index, j.atol, j.rtol))
    return out


def _packed(items: list):
    return descriptor_array(items) if items else items


class DeviceState:
    def __init__(self, w, device: str = "cuda"):
        self.w = w
        self.device = torch.device(device)
        self.ref = torch.empty(w.arena_bytes, dtype=torch.uint8, device=self.device)
        self.cand = torch.empty(w.arena_bytes, dtype=torch.uint8, device=self.device)
        n_desc = max(len(w.allocs), len(w.compares))
        self.ws_size = workspace_bytes(n_desc, len(w.injections))
        self.ws = torch.empty(self.ws_size, dtype=torch.uint8, device=self.device)
        self.seg_res = torch.empty(max(1, len(w.compares)) * SEG_RESULT_DTYPE.itemsize,
                                   dtype=torch.uint8, device=self.device)
        self.guard_res = torch.empty(max(1, len(w.allocs)) * GUARD_RESULT_DTYPE.itemsize,
                                     dtype=torch.uint8, device=self.device)
        # descriptors are packed into ctypes arrays once: every call passes them as they are
        self.inj = _packed(injection_structs(w))
        self.allocs_ref = _packed(self._alloc_structs(self.ref))
        self.allocs_cand = _packed(self._alloc_structs(self.cand))
        self.segments = _packed(self._segment_structs())
        self.cos_ws = None
        self.cos_res = torch.empty(max(1, len(w.compares)) * COS_RESULT_DTYPE.itemsize,
                                   dtype=torch.uint8, device=self.device)

    def arena(self, side: str) -> torch.Tensor:
        return self.cand if side == "cand" else self.ref

    def _alloc_structs(self, arena: torch.Tensor) -> List[Alloc]:
        base = arena.data_ptr()
        out = []
        for k, a in enumerate(self.w.allocs):
            flags = FILL_SATURATE if a.saturate else 0
            out.append(Alloc(base + self.w.offsets[k], a.rows, a.cols, a.stride, a.guard_lo, a.guard_hi,
                             DTYPE_CODE[a.dtype], a.alloc_id, DIST_CODE[a.dist], flags,
                             a.p0, a.p1, a.i0, a.i1))
        return out

    def _segment_structs(self) -> List[Segment]:
        out = []
        for c in self.w.compares:
            a = self.w.allocs[c.alloc]
            off = self.w.data_offset(c.alloc)
            out.append(Segment(self.cand.data_ptr() + off, self.ref.data_ptr() + off,
                               DTYPE_CODE[a.dtype], MODE_CODE[c.mode], NAN_CODE[c.nan_policy], 0,
                               a.rows, a.cols, a.stride, a.stride, c.atol, c.rtol))
        return out

    # ------------------------------------------------------------ the calls
    def fill(self, side: str, variant: int, stream=None) -> None:
        allocs = self.allocs_cand if side == "cand" else self.allocs_ref
        fill_guarded(allocs, self.inj, self.w.seed, variant, self.ws.data_ptr(), self.ws_size, stream)

    def diff(self, stream=None, workgroups: int = 0, segments: Optional[List[Segment]] = None) -> None:
        diff_segments(segments if segments is not None else self.segments, self.seg_res.data_ptr(),
                      self.ws.data_ptr(), self.ws_size, stream, workgroups)

    def diff_cosine(self, stream=None) -> None:
        """The diff plus the cosine term of every float segment, in one pass."""
        if self.cos_ws is None:
            size = diff_cosine_workspace_bytes(self.segments)
            self.cos_ws = torch.empty(max(size, 256), dtype=torch.uint8, device=self.device)
        diff_cosine(self.segments, self.seg_res.data_ptr(), self.cos_res.data_ptr(), self.cos_ws.data_ptr(),
                    self.cos_ws.numel(), stream)

    def cos_results(self) -> List[Dict]:
        torch.cuda.synchronize(self.device)
        n = len(self.w.compares)
        raw = self.cos_res.cpu().numpy()[: n * COS_RESULT_DTYPE.itemsize].view(COS_RESULT_DTYPE)
        return [{f: raw[f][k].item() for f in COS_RESULT_DTYPE.names} for k in range(n)]

    def plan(self, stream=None) -> None:
        """Stages the diff's and the guard check's tables once (repeated checks
        then launch without host planning or uploads)."""
        n = max(len(self.w.compares), len(self.w.allocs))
        size = -(-plan_bytes(n) // 256) * 256        # each plan's workspace starts on a 256-byte boundary
        self.plan_ws = torch.empty(2 * size, dtype=torch.uint8, device=self.device)
        self.diff_plan = plan_diff(self.segments, self.plan_ws.data_ptr(), size, stream)
        self.guard_plan = plan_guard(self.allocs_cand, self.plan_ws.data_ptr() + size, size, stream)

    def diff_planned(self, stream=None) -> None:
        diff_planned(self.diff_plan, self.seg_res.data_ptr(), stream)

    def guard_planned(self, stream=None) -> None:
        guard_planned(self.guard_plan, self.w.seed, self.guard_res.data_ptr(), stream)

    def guard(self, stream=None) -> None:
        guard_check(self.allocs_cand, self.w.seed, self.guard_res.data_ptr(), self.ws.data_ptr(),
                    self.ws_size, stream)

    # ------------------------------------------------------------ results
    def seg_results(self, n: Optional[int] = None) -> List[Dict]:
        torch.cuda.synchronize(self.device)
        n = len(self.w.compares) if n is None else n
        raw = self.seg_res.cpu().numpy()[: n * SEG_RESULT_DTYPE.itemsize].view(SEG_RESULT_DTYPE)
        return [{f: raw[f][k].item() for f in SEG_RESULT_DTYPE.names} for k in range(n)]

    def guard_results(self) -> List[Dict]:
        torch.cuda.synchronize(self.device)
        n = len(self.w.allocs)
        raw = self.guard_res.cpu().numpy()[: n * GUARD_RESULT_DTYPE.itemsize].view(GUARD_RESULT_DTYPE)
        return [{f: raw[f][k].item() for f in GUARD_RESULT_DTYPE.names} for k in range(n)]

    def alloc_bytes(self, side: str, k: int, off: int = 0, nbytes: Optional[int] = None) -> np.ndarray:
        """Bytes [off, off+nbytes) of allocation k (from its first lo-guard byte), copied to host."""
        a = self.w.allocs[k]
        nbytes = a.total_bytes - off if nbytes is None else nbytes
        o = self.w.offsets[k] + off
        return self.arena(side)[o:o + nbytes].cpu().numpy()

    def arena_host(self, side: str) -> np.ndarray:
        return self.arena(side).cpu().numpy()

    def compared_bytes(self) -> int:
        return self.w.compared_bytes()
