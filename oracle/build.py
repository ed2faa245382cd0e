"""Build step for the CPU oracle (test infrastructure): compiles oracle.c with gcc.

Plain ``-O2`` without fast-math, so libm's ``exp`` and IEEE fp64 arithmetic are
used as written.  OpenMP spreads independent rows over host threads.
"""
import pathlib
import subprocess

HERE = pathlib.Path(__file__).resolve().parent
SRC = HERE / "oracle.c"
LIB = HERE / "liboracle.so"


def build(verbose: bool = False) -> pathlib.Path:
    cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-Werror", str(SRC), "-o", str(LIB) + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    pathlib.Path(str(LIB) + ".tmp").replace(LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
