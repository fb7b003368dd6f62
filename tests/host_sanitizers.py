"""Runs the CPU test suite against host code built with AddressSanitizer and
UndefinedBehaviorSanitizer:

    python tests/host_sanitizers.py [extra pytest arguments]

It builds, in a scratch directory, the CPU oracle (clang) and libasmevo.so
with every sanitizer flag passed to the host compilation alone (device code
is built as usual), preloads clang's sanitizer runtime, points the package
and the oracle at those builds (ASMEVO_LIBRARY, REF_ORACLE_LIBRARY) and runs
`pytest tests -m "not gpu"`.  Without a GPU the library's host code runs its
argument validation, planning and error paths; the oracle runs everything.
Any report ends the run with a non-zero status."""
import glob
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)

from paper_2608_20711_amd import build as hip_build  # noqa: E402

CLANG = "/opt/rocm/llvm/bin/clang"
SANITIZE = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined",
            "-fno-omit-frame-pointer", "-g"]


def runtime() -> str:
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not found:
        raise RuntimeError("clang's AddressSanitizer runtime is not installed")
    return found[-1]


def main(argv) -> int:
    out = tempfile.mkdtemp(prefix="asmevo_sanitize_")
    oracle_so = os.path.join(out, "libref_oracle.so")
    subprocess.run([CLANG, "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared", "-ffp-contract=off",
                    "-fno-fast-math", *SANITIZE, "-o", oracle_so, os.path.join(ROOT, "oracle", "ref_oracle.c"),
                    "-lm"], check=True)
    host_only = [x for f in SANITIZE for x in ("-Xarch_host", f)]
    lib_so = hip_build.build(extra=host_only, out=os.path.join(out, "libasmevo.so"))
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": runtime(),
        # Python's own allocations are not freed at exit: leak reports would be noise
        "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=1",
        "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1",
        "ASMEVO_LIBRARY": lib_so,
        "REF_ORACLE_LIBRARY": oracle_so,
    })
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-m", "not gpu", "-q", "-x",
           "-p", "no:cacheprovider", *argv]
    print(" ".join(cmd), flush=True)
    return subprocess.run(cmd, env=env, cwd=ROOT).returncode


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
