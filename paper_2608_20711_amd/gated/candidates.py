"""Candidate edits of s(K0) for the gated verification harness.

The paper's candidates are edits of a kernel's assembly proposed by a search
driver (section 3.8); the harness accepts any candidate generator (section
3.7).  These fixed candidates stand in for such proposals, one per outcome
the harness distinguishes:

  k0_roundtrip     s(K0) unchanged: equivalent, no speedup, not committed
  k1_vectorized    the assembly of a rewrite with 16-byte loads and
                   cross-lane reductions: equivalent and faster
  sleep_in_loop    an s_sleep in K0's first loop: equivalent, slower
  eps_constant     the normalisation epsilon literal changed: divergent
                   floats beyond the tolerance
  out_store_shift  the output store moved by one element: every row's last
                   value lands in its row padding (the last row's in the
                   guard) and its first value is never written: divergent,
                   with corrupted pads and guard
  amax_lds_slot    the argmax read from the neighbouring LDS slot: divergent
                   integer output
  bad_mnemonic     an unknown instruction: does not assemble
  kernarg_size     the metadata declares a larger argument segment: not
                   ABI-consistent with K0
  renamed_kernel   the kernel symbol renamed: K0's kernel is not in the
                   code object
  lds_overflow     the kernel descriptor claims more LDS than a CU has: not
                   ABI-consistent

Every edit that reaches the GPU keeps each access inside memory the harness
allocated: the shifted store writes 4 bytes past a row into its padding or
into the 4 KiB guard, and the shifted LDS read stays inside the argmax
array."""
from __future__ import annotations

import re
from dataclasses import dataclass
from typing import Callable, List


@dataclass(frozen=True)
class Candidate:
    name: str
    expect: str                     # the outcome this candidate is built to produce
    make: Callable[[str, str], str]  # (s(K0), s(K1)) -> s'


def _one(pattern: str, text: str) -> re.Match:
    ms = list(re.finditer(pattern, text, flags=re.M))
    if len(ms) != 1:
        raise ValueError(f"edit anchor {pattern!r} found {len(ms)} times")
    return ms[0]


def _replace_one(text: str, pattern: str, repl: str) -> str:
    m = _one(pattern, text)
    return text[:m.start()] + m.expand(repl) + text[m.end():]


def eps_constant(s0: str, s1: str) -> str:
    # 1e-5f (0x3727c5ac) -> 0.1f (0x3dcccccd)
    return _replace_one(s0, r"0x3727c5ac", "0x3dcccccd")


def out_store_shift(s0: str, s1: str) -> str:
    # the only vector-address dword store is the output store of the last loop
    return _replace_one(s0, r"^(\s*global_store_dword v\[\d+:\d+\], v\d+, off)$", r"\1 offset:4")


def amax_lds_slot(s0: str, s1: str) -> str:
    # the argmax store is the scalar-base dword store whose data comes from LDS
    lines = s0.split("\n")
    for k, line in enumerate(lines):
        m = re.match(r"^\s*global_store_dword v\d+, (v\d+), s\[\d+:\d+\]$", line)
        if not m:
            continue
        reg = m.group(1)
        for j in range(k - 1, max(-1, k - 12), -1):
            r = re.match(rf"^(\s*ds_read_b32 {reg}, v\d+)$", lines[j])
            if r:
                lines[j] = r.group(1) + " offset:4"
                return "\n".join(lines)
    raise ValueError("argmax store not found")


def sleep_in_loop(s0: str, s1: str) -> str:
    m = re.search(r"^(\.LBB\d+_\d+:\s*; =>This Inner Loop Header.*)$", s0, flags=re.M)
    if not m:
        raise ValueError("no loop header")
    return s0[:m.end()] + "\n\ts_sleep 127" + s0[m.end():]


def bad_mnemonic(s0: str, s1: str) -> str:
    m = _one(r"^rmsnorm_k0:.*$", s0)
    return s0[:m.end()] + "\n\tv_frobnicate_f32 v1, v2, v3" + s0[m.end():]


def kernarg_size(s0: str, s1: str) -> str:
    t = _replace_one(s0, r"^(\s*\.amdhsa_kernarg_size )68$", r"\g<1>72")
    return _replace_one(t, r"^(\s*\.kernarg_segment_size:\s+)68$", r"\g<1>72")


def renamed_kernel(s0: str, s1: str) -> str:
    return re.sub(r"\brmsnorm_k0\b", "rmsnorm_kx", s0)


def lds_overflow(s0: str, s1: str) -> str:
    t = _replace_one(s0, r"^(\s*\.amdhsa_group_segment_fixed_size )3072$", r"\g<1>200000")
    return _replace_one(t, r"^(\s*\.group_segment_fixed_size:\s+)3072$", r"\g<1>200000")


CANDIDATES: List[Candidate] = [
    Candidate("k0_roundtrip", "ok", lambda s0, s1: s0),
    Candidate("k1_vectorized", "ok", lambda s0, s1: s1),
    Candidate("sleep_in_loop", "ok", sleep_in_loop),
    Candidate("eps_constant", "divergent", eps_constant),
    Candidate("out_store_shift", "divergent", out_store_shift),
    Candidate("amax_lds_slot", "divergent", amax_lds_slot),
    Candidate("bad_mnemonic", "asm_invalid", bad_mnemonic),
    Candidate("kernarg_size", "abi_invalid", kernarg_size),
    Candidate("renamed_kernel", "abi_invalid", renamed_kernel),
    Candidate("lds_overflow", "abi_invalid", lds_overflow),
]
