"""Build steps of the gated verification harness (AsmEvo section 3.7,
Algorithm 1: Assembles(s'), c = Build(s'), StaticConsistent(c)).

The kernel under test is compiled here from its own HIP source to gfx950
assembly text, s(K0).  A candidate is assembly text: it is assembled with
the LLVM assembler and linked into a code object with ld.lld, and the code
object's AMDGPU metadata note (msgpack) is read back for the static checks.
Only code objects built here from source are read."""
from __future__ import annotations

import os
import shutil
import struct
import subprocess
import tempfile
from dataclasses import dataclass
from typing import Dict, List, Optional

ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HERE = os.path.dirname(os.path.abspath(__file__))
K0_SOURCE = os.path.join(HERE, "k0_rmsnorm.hip")        # the kernel under test
K1_SOURCE = os.path.join(HERE, "k1_rmsnorm_vec.hip")    # a rewrite, one of the candidates
ARCH = "gfx950"
HIPCC_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-ffp-contract=off",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _tool(name: str) -> str:
    for d in (os.path.join(ROCM, "llvm", "bin"), os.path.join(ROCM, "bin")):
        p = os.path.join(d, name)
        if os.path.exists(p):
            return p
    found = shutil.which(name)
    if not found:
        raise FileNotFoundError(f"{name} not found under {ROCM}")
    return found


def device_assembly(source: str) -> str:
    """gfx950 assembly text of a HIP source file (device code only)."""
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k.s")
        cmd = [_tool("hipcc"), *HIPCC_FLAGS, "-S", "--cuda-device-only", source, "-o", out]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {source}:\n{r.stderr[-4000:]}")
        with open(out) as f:
            return f.read()


def assembly_path(source: str) -> str:
    return os.path.splitext(source)[0] + ".s"


def build_assembly() -> None:
    """s(K0) and s(K1): gfx950 assembly of the two sources, written beside
    them (part of the library build)."""
    for src in (K0_SOURCE, K1_SOURCE):
        text = device_assembly(src)
        tmp = assembly_path(src) + ".tmp"
        with open(tmp, "w") as f:
            f.write(text)
        os.replace(tmp, assembly_path(src))


def load_assembly(source: str) -> str:
    path = assembly_path(source)
    if not os.path.exists(path):
        raise FileNotFoundError(f"{path} is missing: build the library first (__graft_entry__.build())")
    with open(path) as f:
        return f.read()


@dataclass
class BuildResult:
    ok: bool
    stage: str                      # "assemble" or "link" when not ok
    log: str
    code_object: Optional[bytes] = None


def build(asm_text: str) -> BuildResult:
    """Assembles s' and links it into a code object (Assembles and Build)."""
    with tempfile.TemporaryDirectory() as d:
        s_path, o_path, co_path = (os.path.join(d, n) for n in ("k.s", "k.o", "k.hsaco"))
        with open(s_path, "w") as f:
            f.write(asm_text)
        r = subprocess.run([_tool("clang"), "-x", "assembler", "-target", "amdgcn-amd-amdhsa", "-mcpu=" + ARCH,
                            "-c", s_path, "-o", o_path], capture_output=True, text=True)
        if r.returncode != 0:
            return BuildResult(False, "assemble", r.stderr[-4000:])
        r = subprocess.run([_tool("ld.lld"), "-shared", o_path, "-o", co_path], capture_output=True, text=True)
        if r.returncode != 0:
            return BuildResult(False, "link", r.stderr[-4000:])
        with open(co_path, "rb") as f:
            return BuildResult(True, "", "", f.read())


NT_AMDGPU_METADATA = 32


def metadata(code_object: bytes) -> Dict:
    """The AMDGPU metadata map of an ELF64 code object (its NT_AMDGPU_METADATA note)."""
    import msgpack
    b = code_object
    if b[:4] != b"\x7fELF" or b[4] != 2:
        raise ValueError("not an ELF64 code object")
    shoff = struct.unpack_from("<Q", b, 0x28)[0]
    shentsize, shnum = struct.unpack_from("<HH", b, 0x3A)
    for k in range(shnum):
        sh = shoff + k * shentsize
        sh_type = struct.unpack_from("<I", b, sh + 4)[0]
        if sh_type != 7:                                   # SHT_NOTE
            continue
        off, size = struct.unpack_from("<QQ", b, sh + 0x18)
        p, end = off, off + size
        while p + 12 <= end:
            namesz, descsz, ntype = struct.unpack_from("<III", b, p)
            name = b[p + 12:p + 12 + namesz].rstrip(b"\0")
            dp = p + 12 + ((namesz + 3) & ~3)
            desc = b[dp:dp + descsz]
            if name == b"AMDGPU" and ntype == NT_AMDGPU_METADATA:
                return msgpack.unpackb(desc, raw=False)
            p = dp + ((descsz + 3) & ~3)
    raise ValueError("no AMDGPU metadata note")


def kernel_metadata(code_object: bytes, name: str) -> Optional[Dict]:
    for k in metadata(code_object).get("amdhsa.kernels", []):
        if k.get(".name") == name:
            return k
    return None


def kernel_names(code_object: bytes) -> List[str]:
    return [k.get(".name") for k in metadata(code_object).get("amdhsa.kernels", [])]
