"""Build step for the CPU oracle (test infrastructure): compiles oracle.c with gcc.

Plain ``-O2`` without fast-math, so libm's ``exp`` and IEEE fp64 arithmetic are
used as written.  OpenMP spreads independent rows over host threads.

``build(sanitize=True)`` (``python oracle/build.py --sanitize``) compiles it
with clang, AddressSanitizer and UndefinedBehaviorSanitizer instead (the same
runtime as the sanitized HIP library, so both load into one process).
"""
import os
import pathlib
import subprocess

HERE = pathlib.Path(__file__).resolve().parent
SRC = HERE / "oracle.c"
LIB = HERE / "liboracle.so"


def build(verbose: bool = False, sanitize: bool = False) -> pathlib.Path:
    if sanitize:
        clang = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin", "clang")
        cc = [clang, "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-shared-libasan",
              "-fno-omit-frame-pointer"]
    else:
        cc = ["gcc"]
    cmd = [*cc, "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-Werror", str(SRC), "-o", str(LIB) + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    pathlib.Path(str(LIB) + ".tmp").replace(LIB)
    return LIB


if __name__ == "__main__":
    import sys
    print(build(verbose=True, sanitize="--sanitize" in sys.argv[1:]))
