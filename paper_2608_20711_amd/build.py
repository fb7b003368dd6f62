"""Builds libasmevo.so (HIP for gfx950) in-tree with hipcc."""
from __future__ import annotations

import glob
import os
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libasmevo.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # every fp operation rounds once, in the order written; denormals kept
    "-ffp-contract=off", "-fno-fast-math", "-fno-gpu-flush-denormals-to-zero",
    # no packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]

# Flags for one source only.  In the fill, machine LICM hoists loop-invariant
# scalar values (among them the fp64 series coefficients, 64-bit literals that
# a gfx9 VOP3 cannot encode, so each lives in a scalar pair) out of the
# Box-Muller loop until the scalar file overflows: 496 SGPRs spilled to VGPR
# lanes and read back inside the loop.  Without it: 268 spills, 62 VGPRs
# instead of 79, and the 64 GiB candidate fill in 157.0 ms instead of 168.7 ms.
PER_SOURCE = {
    "fill.hip": ["-mllvm", "-disable-machine-licm"],
}

PROBE_SRC = os.path.join(ROOT, "read_probe.hip")
PROBE_EXE = os.path.join(ROOT, "read_probe")


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def build(verbose: bool = False, extra=(), out: str = LIB) -> str:
    """Compiles every HIP source (in parallel) and links libasmevo.so, or the
    library `out` (always recompiles)."""
    tmp = out + ".tmp"
    compile_flags = [f for f in FLAGS if f != "-shared"]
    with tempfile.TemporaryDirectory() as objdir:
        jobs, objs = [], []
        for src in sources():
            obj = os.path.join(objdir, os.path.basename(src) + ".o")
            cmd = [HIPCC, *compile_flags, *PER_SOURCE.get(os.path.basename(src), []), *extra,
                   "-I", INCLUDE, "-I", CSRC, "-c", src, "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            jobs.append((cmd, subprocess.Popen(cmd)))
            objs.append(obj)
        failed = [cmd for cmd, proc in jobs if proc.wait() != 0]
        if failed:
            raise subprocess.CalledProcessError(1, failed[0])
        cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build_probe(verbose: bool = False) -> str:
    """Compiles the HBM read-ceiling probe that bench.py reports beside the diff."""
    tmp = PROBE_EXE + ".tmp"
    flags = [f for f in FLAGS if f not in ("-shared", "-fPIC")]
    cmd = [HIPCC, *flags, PROBE_SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, PROBE_EXE)
    return PROBE_EXE


if __name__ == "__main__":
    build(verbose=True, extra=sys.argv[1:])
    build_probe(verbose=True)
