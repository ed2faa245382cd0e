"""Build step for the HIP library: compiles csrc/ for gfx950 into libfastseq_hip.so.

Every source is compiled with hipcc for gfx950 only.  Packed-fp32 VALU
instructions are disabled for device code (``-packed-fp32-ops``); the host
pass warns that it does not know that feature, which is harmless.

The CPython marshalling module (csrc/pyext.c, plain C) is then compiled with
gcc and linked against the library.
"""
import concurrent.futures
import os
import pathlib
import subprocess
import sysconfig

PKG = pathlib.Path(__file__).resolve().parent
ROOT = PKG.parent
CSRC = PKG / "csrc"
BUILD = PKG / "_build"
LIB = PKG / "libfastseq_hip.so"
EXT = PKG / ("_fastseq_ext" + sysconfig.get_config_var("EXT_SUFFIX"))
SOURCES = ["capi.cpp", "cross_attn.hip", "ngram_block.hip", "beam_select.hip", "cache_reorder.hip", "postproc.cpp"]  # pyext.c is built by build_ext
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          # kernel arguments arrive preloaded in SGPRs: the first wave of a
          # workgroup skips one dependent scalar load before its first
          # address computation
          "-mllvm", "-amdgpu-kernarg-preload-count=16",
          "-Wall", "-Wno-unused-command-line-argument",
          f"-I{ROOT / 'include'}", f"-I{CSRC}"]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def _compile(src: str, verbose: bool) -> pathlib.Path:
    obj = BUILD / (src + ".o")
    cmd = [hipcc(), *COMMON, "-x", "hip", "-c", str(CSRC / src), "-o", str(obj)]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "'-packed-fp32-ops' is not a recognized feature"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip() and verbose:
        print(err, flush=True)
    return obj


def build(verbose: bool = False) -> pathlib.Path:
    BUILD.mkdir(exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = str(LIB) + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-Wl,-soname,libfastseq_hip.so",
           *map(str, objs), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    build_ext(verbose)
    return LIB


def build_ext(verbose: bool = False) -> pathlib.Path:
    """The CPython module that marshals arguments into the C ABI."""
    tmp = str(EXT) + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-Wall", "-Wextra", "-Werror",
           f"-I{sysconfig.get_paths()['include']}", f"-I{ROOT / 'include'}", str(CSRC / "pyext.c"),
           f"-L{PKG}", "-lfastseq_hip", "-Wl,-rpath,$ORIGIN", "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, EXT)
    return EXT


if __name__ == "__main__":
    print(build(verbose=True))
