"""Build and ctypes binding of tests/hip/device_pins.hip: test-only kernels
that run the library's per-element device functions (built from its own
headers) so that their outputs can be compared with the CPU oracle."""
import ctypes
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "hip", "device_pins.hip")
SO = os.path.join(HERE, "hip", "libdevice_pins.so")

_lib = None


def build(verbose: bool = False) -> str:
    """Compiles the kernels with the library's own compiler flags (always recompiles)."""
    from paper_2608_20711_amd import build as hip_build
    cmd = [hip_build.HIPCC, *hip_build.FLAGS, "-I", hip_build.INCLUDE, "-I", hip_build.CSRC, SRC, "-o", SO + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(SO + ".tmp", SO)
    return SO


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(SO):
            raise RuntimeError(f"{SO} is not built: run __graft_entry__.build()")
        L = ctypes.CDLL(SO)
        u32, u64, vp, i32, dbl = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int32, ctypes.c_double
        L.pins_encode.argtypes = [u32, u64, vp, vp, vp, vp, vp]
        L.pins_log_u.argtypes = [u32, u64, vp, vp]
        L.pins_sincos.argtypes = [u32, u64, vp, vp, vp]
        L.pins_normal.argtypes = [vp, vp, u64, vp, vp, vp]
        L.pins_pairs.argtypes = [i32, i32, dbl, dbl, vp, vp, u64, vp, vp, vp, vp]
        for f in (L.pins_encode, L.pins_log_u, L.pins_sincos, L.pins_normal, L.pins_pairs):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def check(status: int, what: str) -> None:
    if status != 0:
        raise RuntimeError(f"{what}: status {status}")
