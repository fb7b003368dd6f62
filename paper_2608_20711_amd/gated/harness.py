"""GatedEval (AsmEvo section 3.7, Algorithm 1) and the commit gate (Eq. 2)
around a K0 built here from source.

For a candidate s' the harness runs, in this order, stopping at the first
failure:

  1. Assembles(s') and c = Build(s')          -> asm_invalid
  2. StaticConsistent(c) against K0           -> abi_invalid
  3. for every input x in the oracle set X, three times:
       restore the pre-state, launch c, compare the whole post-state with
       O(x) = run(K0, x) (floats within tau and with cosine >= theta, integers
       and inputs bit-exact, guards and row pads intact)
                                              -> divergent / runtime_failure
  4. s_hat(c) = T(K0) / T(c), each the median of R event-timed launches
     after a warm-up, under the same device and launch     -> ok, s_hat

Every data-parallel step (guarded fills, snapshot / restore, the comparison,
the guard check, launches and timing) runs in libasmevo.so; this module is
the host-side controller.  The oracle set is Tier-1 style: seeded guarded
allocations for K0's inputs and outputs (outputs start as random bits, so a
value a candidate fails to write shows up), one launch of K0 per input.
"""
from __future__ import annotations

import os
import statistics
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import torch

from .. import (Alloc, F32, BF16, I32, BITWISE, TOLERANCE, NAN_EQUAL, DIST_NORMAL, DIST_BITS,
                DIST_BOUNDARY, KernelArgs, Region, Segment, copy_regions, diff_cosine,
                diff_cosine_workspace_bytes, fill_guarded, guard_check, kernel_load, kernel_time,
                kernel_launch, kernel_unload, workspace_bytes, AsmevoError)
from . import toolchain

KERNEL = "rmsnorm_k0"
BLOCK = 256
K0_SOURCE, K1_SOURCE = toolchain.K0_SOURCE, toolchain.K1_SOURCE
load_assembly = toolchain.load_assembly


# the paper's settings (section 4.1)
TAU = 1e-3          # Eq. 1: infinity norm of the difference
THETA = 0.9999      # Eq. 1: cosine similarity
REPEATS = 3         # the equivalence check is repeated per candidate
EPSILON, K_CV, S_FLOOR = 0.002, 0.85, 1.0   # Eq. 2

LDS_LIMIT = 160 * 1024          # bytes of LDS per workgroup on gfx950
VGPR_LIMIT = 512                # architected + accumulation VGPRs per wave64 lane
SGPR_LIMIT = 102

OUTCOMES = ("ok", "asm_invalid", "abi_invalid", "divergent", "runtime_failure")


# ---------------------------------------------------------------- outcomes
@dataclass
class Outcome:
    status: str
    reason: str = ""
    speedup: Optional[float] = None
    t_k0_ms: Optional[float] = None
    t_ms: Optional[float] = None
    cv: Optional[float] = None
    checks: List[Dict] = field(default_factory=list)    # per (input, repeat) equivalence records
    static: List[str] = field(default_factory=list)     # failed static checks
    wall_s: Optional[float] = None                      # host wall time of the whole evaluation

    def as_dict(self) -> Dict:
        return {"status": self.status, "reason": self.reason, "speedup": self.speedup, "t_k0_ms": self.t_k0_ms,
                "t_ms": self.t_ms, "cv": self.cv, "static": self.static, "checks": self.checks,
                "wall_s": self.wall_s}


def commit_gate(eq_all: bool, s_c: float, s_best: float, cv: float, eps: float = EPSILON, k: float = K_CV,
                s_floor: float = S_FLOOR) -> Tuple[bool, float]:
    """Eq. 2: m* = (1 + max(eps, k * cv)) * s_hat(K*); commit iff every
    equivalence check passed and s_hat(c) >= max(m*, s_floor).  Returns
    (commit, the threshold max(m*, s_floor))."""
    m_star = (1.0 + max(eps, k * cv)) * s_best
    bar = max(m_star, s_floor)
    return bool(eq_all) and s_c >= bar, bar


# ---------------------------------------------------------------- static checks
def static_consistent(meta_c: Optional[Dict], meta_k0: Dict, block: int = BLOCK) -> List[str]:
    """StaticConsistent(c): the candidate keeps K0's kernel ABI (same name,
    argument list, argument segment and wavefront size) and stays within the
    hardware's resources.  Returns the failed checks (empty if consistent)."""
    if meta_c is None:
        return [f"kernel {KERNEL} not in the code object"]
    bad = []
    for key in (".kernarg_segment_size", ".kernarg_segment_align", ".wavefront_size", ".uses_dynamic_stack"):
        if meta_c.get(key) != meta_k0.get(key):
            bad.append(f"{key}: {meta_c.get(key)} != K0's {meta_k0.get(key)}")
    args_c = [(a.get(".offset"), a.get(".size"), a.get(".value_kind"), a.get(".address_space"))
              for a in meta_c.get(".args", [])]
    args_0 = [(a.get(".offset"), a.get(".size"), a.get(".value_kind"), a.get(".address_space"))
              for a in meta_k0.get(".args", [])]
    if args_c != args_0:
        bad.append(f"arguments {args_c} != K0's {args_0}")
    if meta_c.get(".max_flat_workgroup_size", 0) < block:
        bad.append(f".max_flat_workgroup_size {meta_c.get('.max_flat_workgroup_size')} < launch block {block}")
    if meta_c.get(".group_segment_fixed_size", 0) > LDS_LIMIT:
        bad.append(f".group_segment_fixed_size {meta_c.get('.group_segment_fixed_size')} > {LDS_LIMIT}")
    if meta_c.get(".vgpr_count", 0) + meta_c.get(".agpr_count", 0) > VGPR_LIMIT:
        bad.append("VGPRs beyond the register file")
    if meta_c.get(".sgpr_count", 0) > SGPR_LIMIT + 4:
        bad.append("SGPRs beyond the register file")
    return bad


# ---------------------------------------------------------------- inputs X
@dataclass(frozen=True)
class InputSpec:
    """One evaluated input x: shape, strides, seed, and the value mix of x."""
    name: str
    rows: int
    hidden: int
    in_stride: int
    out_stride: int
    seed: int
    boundary_rate: float = 0.0      # BOUNDARY values in x (NaN / Inf / subnormals / extremes)


DEFAULT_INPUTS = (
    InputSpec("decode_16k_x_4096", 16384, 4096, 4096 + 64, 4096 + 32, 0xA5E0000000000F31),
    InputSpec("odd_1000_x_2304", 1000, 2304, 2304 + 8, 2304 + 4, 0xA5E0000000000F32),
    InputSpec("boundary_512_x_1024", 512, 1024, 1024 + 8, 1024 + 8, 0xA5E0000000000F33, 1e-3),
)

GUARD = 4096
ALIGN = 256


class OracleInput:
    """Device state of one input x: the pre-state P(x) (seeded guarded fill),
    the reference post-state O(x) = run(K0, P(x)), and a work arena where
    candidates run after P(x) is restored in place."""

    # allocation table: name, dtype, rows, cols, stride, dist, p0, p1
    def __init__(self, spec: InputSpec, device: torch.device):
        if spec.hidden % BLOCK or spec.hidden % 8 or spec.in_stride % 8 or spec.out_stride % 4:
            raise ValueError("hidden must be a multiple of 256, strides of 16 bytes")
        if spec.in_stride < spec.hidden or spec.out_stride <= spec.hidden:
            raise ValueError("the output rows need padding")
        self.spec = spec
        r, h = spec.rows, spec.hidden
        xdist = (DIST_BOUNDARY, spec.boundary_rate, 1.0) if spec.boundary_rate else (DIST_NORMAL, 0.0, 1.0)
        self.table = [  # name, dtype, esize, rows, cols, stride, dist, p0, p1, is_input
            ("x", BF16, 2, r, h, spec.in_stride, *xdist, True),
            ("residual", BF16, 2, r, h, spec.in_stride, DIST_NORMAL, 0.0, 0.5, True),
            ("weight", BF16, 2, 1, h, h, DIST_NORMAL, 1.0, 0.1, True),
            ("out", F32, 4, r, h, spec.out_stride, DIST_BITS, 0.0, 0.0, False),
            ("res_out", BF16, 2, r, h, spec.in_stride, DIST_BITS, 0.0, 0.0, False),
            ("rstd", F32, 4, 1, r, r, DIST_BITS, 0.0, 0.0, False),
            ("amax", I32, 4, 1, r, r, DIST_BITS, 0.0, 0.0, False),
        ]
        self.offsets, self.sizes = [], []
        off = 0
        for (_, _, es, rows, cols, stride, *_rest) in self.table:
            size = 2 * GUARD + ((rows - 1) * stride + cols) * es
            self.offsets.append(off)
            self.sizes.append(size)
            off += -(-size // ALIGN) * ALIGN
        self.arena_bytes = off
        self.device = device
        self.pre = torch.empty(off, dtype=torch.uint8, device=device)
        self.ref = torch.empty(off, dtype=torch.uint8, device=device)
        self.work = torch.empty(off, dtype=torch.uint8, device=device)
        n = len(self.table)
        self.ws_size = max(workspace_bytes(n, 0), 4096)
        self.ws = torch.empty(self.ws_size, dtype=torch.uint8, device=device)
        self.seg_res = torch.empty(n * 56, dtype=torch.uint8, device=device)
        self.cos_res = torch.empty(n * 48, dtype=torch.uint8, device=device)
        self.guard_res = torch.empty(n * 48, dtype=torch.uint8, device=device)
        self.cos_ws = None
        fill_guarded(self.allocs(self.pre), [], spec.seed, 0, self.ws.data_ptr(), self.ws_size)

    def allocs(self, arena: torch.Tensor) -> List[Alloc]:
        out = []
        for k, (_, dt, _, rows, cols, stride, dist, p0, p1, _) in enumerate(self.table):
            out.append(Alloc(arena.data_ptr() + self.offsets[k], rows, cols, stride, GUARD, GUARD, dt, 100 + k,
                             dist, 0, p0, p1, 0, 0))
        return out

    def data_ptr(self, arena: torch.Tensor, name: str) -> int:
        k = [t[0] for t in self.table].index(name)
        return arena.data_ptr() + self.offsets[k] + GUARD

    def restore(self, dst: torch.Tensor) -> None:
        """dst <- P(x), every allocation with its guards and pads, in place."""
        regs = [Region(dst.data_ptr() + o, self.pre.data_ptr() + o, n) for o, n in zip(self.offsets, self.sizes)]
        copy_regions(regs, self.ws.data_ptr(), self.ws_size)

    def args(self, arena: torch.Tensor) -> KernelArgs:
        import ctypes
        s = self.spec
        ptrs = [ctypes.c_uint64(self.data_ptr(arena, n)) for n in
                ("x", "residual", "weight", "out", "res_out", "rstd", "amax")]
        return KernelArgs(ptrs + [ctypes.c_int32(s.hidden), ctypes.c_int32(s.in_stride), ctypes.c_int32(s.out_stride)])

    def grid(self) -> Tuple[int, int, int]:
        return (self.spec.rows, 1, 1)

    def segments(self) -> List[Segment]:
        """Whole-state comparison: inputs bit-exact (a candidate must not
        change them), float outputs within tau, the integer output bit-exact."""
        segs = []
        for k, (name, dt, _, rows, cols, stride, _, _, _, is_input) in enumerate(self.table):
            a = self.data_ptr(self.work, name)
            b = self.data_ptr(self.ref, name)
            mode = BITWISE if (is_input or dt == I32) else TOLERANCE
            segs.append(Segment(a, b, dt, mode, NAN_EQUAL, 0, rows, cols, stride, stride,
                                TAU if mode == TOLERANCE else 0.0, 0.0))
        return segs

    def compare(self) -> Dict:
        """Compares the work arena with O(x): diff + cosine per buffer, guards and pads."""
        from ..state import SEG_RESULT_DTYPE, COS_RESULT_DTYPE, GUARD_RESULT_DTYPE
        segs = self.segments()
        if self.cos_ws is None:
            need = diff_cosine_workspace_bytes(segs)
            self.cos_ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        diff_cosine(segs, self.seg_res.data_ptr(), self.cos_res.data_ptr(), self.cos_ws.data_ptr(),
                    self.cos_ws.numel())
        guard_check(self.allocs(self.work), self.spec.seed, self.guard_res.data_ptr(), self.ws.data_ptr(),
                    self.ws_size)
        torch.cuda.synchronize(self.device)
        n = len(self.table)
        seg = self.seg_res.cpu().numpy().view(SEG_RESULT_DTYPE)[:n]
        cos = self.cos_res.cpu().numpy().view(COS_RESULT_DTYPE)[:n]
        grd = self.guard_res.cpu().numpy().view(GUARD_RESULT_DTYPE)[:n]
        buffers, ok = {}, True
        for k, (name, dt, *_rest) in enumerate(self.table):
            is_input = self.table[k][-1]
            tol = not is_input and dt != I32
            rec = {"mismatches": int(seg["mismatches"][k]), "first_mismatch": int(seg["first_mismatch"][k]),
                   "bitwise_mismatches": int(seg["bitwise_mismatches"][k]), "max_abs": float(seg["max_abs"][k]),
                   "guard_bytes_corrupted": int(grd["bad_lo"][k] + grd["bad_hi"][k]),
                   "pad_bytes_corrupted": int(grd["bad_pad"][k])}
            if tol:
                rec["cosine"] = float(cos["cosine"][k])
            good = rec["mismatches"] == 0 and rec["guard_bytes_corrupted"] == 0 and rec["pad_bytes_corrupted"] == 0
            if tol and not (rec["cosine"] >= THETA):
                good = False
            rec["equal"] = good
            ok = ok and good
            buffers[name] = rec
        return {"equal": ok, "buffers": buffers}

    def free(self) -> None:
        del self.pre, self.ref, self.work, self.ws, self.cos_ws


# ---------------------------------------------------------------- the harness
class GatedEval:
    """Holds K0 (built from its source), the oracle set (X, O) acquired by
    running K0 once per input, and evaluates candidates with Algorithm 1."""

    def __init__(self, inputs: Sequence[InputSpec] = DEFAULT_INPUTS, timing_input: int = 0, warmup: int = 5,
                 reps: int = 20, device: str = "cuda"):
        self.device = torch.device(device)
        self.s_k0 = load_assembly(K0_SOURCE)
        self.s_k1 = load_assembly(K1_SOURCE)
        b = toolchain.build(self.s_k0)
        if not b.ok:
            raise RuntimeError("K0 does not build: " + b.log)
        self.k0_image = b.code_object
        self.meta_k0 = toolchain.kernel_metadata(self.k0_image, KERNEL)
        self.k0 = kernel_load(self.k0_image, KERNEL)
        self.warmup, self.reps = warmup, reps
        self.inputs = [OracleInput(s, self.device) for s in inputs]
        self.timing_input = timing_input
        for x in self.inputs:                       # AcquireOracle: O(x) = run(K0, P(x))
            x.restore(x.ref)
            kernel_launch(self.k0, x.grid(), (BLOCK, 1, 1), x.args(x.ref))
        torch.cuda.synchronize(self.device)

    def close(self) -> None:
        kernel_unload(self.k0)
        for x in self.inputs:
            x.free()

    # -------------------------------------------------------- Algorithm 1
    def evaluate(self, s_prime: str) -> Outcome:
        b = toolchain.build(s_prime)
        if not b.ok:
            first = next((l for l in b.log.splitlines() if "error" in l), b.log.strip()[:200])
            return Outcome("asm_invalid", f"{b.stage}: {first}")
        try:
            meta = toolchain.kernel_metadata(b.code_object, KERNEL)
            if toolchain.metadata(b.code_object).get("amdhsa.target") != toolchain.metadata(self.k0_image).get(
                    "amdhsa.target"):
                return Outcome("abi_invalid", "code object target differs from K0's", static=["amdhsa.target"])
        except ValueError as e:
            return Outcome("abi_invalid", str(e))
        bad = static_consistent(meta, self.meta_k0)
        if bad:
            return Outcome("abi_invalid", bad[0], static=bad)
        try:
            c = kernel_load(b.code_object, KERNEL)
        except AsmevoError as e:
            return Outcome("runtime_failure", str(e))
        try:
            checks = []
            for x in self.inputs:
                for rep in range(REPEATS):
                    x.restore(x.work)
                    kernel_launch(c, x.grid(), (BLOCK, 1, 1), x.args(x.work))
                    res = x.compare()
                    checks.append({"input": x.spec.name, "repeat": rep, **res})
                    if not res["equal"]:
                        bad_bufs = [n for n, r in res["buffers"].items() if not r["equal"]]
                        return Outcome("divergent", f"{x.spec.name}: " + ", ".join(bad_bufs), checks=checks)
            x = self.inputs[self.timing_input]
            t0 = kernel_time(self.k0, x.grid(), (BLOCK, 1, 1), x.args(x.work), self.warmup, self.reps)
            tc = kernel_time(c, x.grid(), (BLOCK, 1, 1), x.args(x.work), self.warmup, self.reps)
            m0, mc = statistics.median(t0), statistics.median(tc)
            cv = statistics.pstdev(tc) / statistics.fmean(tc)
            return Outcome("ok", "", m0 / mc, m0, mc, cv, checks=checks)
        except AsmevoError as e:
            return Outcome("runtime_failure", str(e))
        finally:
            kernel_unload(c)


# ---------------------------------------------------------------- lineage
@dataclass
class Node:
    id: int
    name: str
    parent: Optional[int]
    speedup: float


def search(harness: GatedEval, candidates) -> Tuple[List[Node], List[Tuple[str, Outcome, bool, Optional[float]]]]:
    """A single-mode pass over fixed candidates (Algorithm 2 without the
    driver): every candidate is evaluated against K0; a candidate that passes
    is committed when Eq. 2 holds against the current best K*.  Returns the
    lineage (committed nodes, K0 first) and (name, outcome, committed, bar)
    per candidate."""
    import time
    lineage = [Node(0, "K0", None, 1.0)]
    best = lineage[0]
    log = []
    for cand in candidates:
        t0 = time.perf_counter()
        out = harness.evaluate(cand.make(harness.s_k0, harness.s_k1))
        out.wall_s = time.perf_counter() - t0
        committed, bar = False, None
        if out.status == "ok":
            committed, bar = commit_gate(True, out.speedup, best.speedup, out.cv)
            if committed:
                node = Node(len(lineage), cand.name, best.id, out.speedup)
                lineage.append(node)
                best = node
        log.append((cand.name, out, committed, bar))
    return lineage, log


def main(argv=None) -> int:
    """Runs the fixed candidates through GatedEval and the commit gate and
    prints one JSON line: per-candidate outcome, speedup, threshold, commit,
    wall time, and the lineage."""
    import argparse
    import json
    import time
    from .candidates import CANDIDATES
    p = argparse.ArgumentParser(description=main.__doc__)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--reps", type=int, default=20)
    args = p.parse_args(argv)
    t0 = time.perf_counter()
    h = GatedEval(warmup=args.warmup, reps=args.reps)
    setup_s = time.perf_counter() - t0
    try:
        lineage, records = search(h, CANDIDATES)
    finally:
        h.close()
    out = {"setup_s": round(setup_s, 3), "inputs": [x.spec.name for x in h.inputs],
           "candidates": [{"name": n, "status": o.status, "reason": o.reason[:160],
                           "speedup": None if o.speedup is None else round(o.speedup, 4),
                           "t_k0_ms": None if o.t_k0_ms is None else round(o.t_k0_ms, 4),
                           "t_ms": None if o.t_ms is None else round(o.t_ms, 4),
                           "cv": None if o.cv is None else round(o.cv, 5),
                           "bar": None if bar is None else round(bar, 5), "committed": c,
                           "equivalence_checks": len(o.checks), "wall_s": round(o.wall_s, 3)}
                          for n, o, c, bar in records],
           "lineage": [{"id": nd.id, "name": nd.name, "parent": nd.parent, "speedup": round(nd.speedup, 4)}
                       for nd in lineage]}
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
