"""Build step for the HIP library: compiles csrc/ for gfx950 into libfastseq_hip.so.

Every source is compiled with hipcc for gfx950 only.  Packed-fp32 VALU
instructions are disabled for device code (``-packed-fp32-ops``); the host
pass warns that it does not know that feature, which is harmless.

The CPython marshalling module (csrc/pyext.c, plain C) is then compiled with
gcc and linked against the library.

``build(trace=True)`` (``--trace``) compiles every source with FS_TRACE=1: the
attention and selection kernels then write per-workgroup timelines to a
buffer set with fs_trace_set (for measurements of where a launch spends its
time; a plain ``build()`` restores the normal kernels).

``build(sanitize=True)`` (``python -m paper_2106_04718_amd.build --sanitize``)
instruments the host code of every source with AddressSanitizer and
UndefinedBehaviorSanitizer (``-Xarch_host``: device code is built as usual),
links the library against clang's shared sanitizer runtime and builds the
marshalling module with clang and the same sanitizers.  Such a build is for
CPU test runs only (tests/run_sanitized.sh); a plain ``build()`` restores the
normal library.
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


# host-side sanitizer flags: every one behind -Xarch_host, so no device code
# is built with a sanitizer
SANITIZE_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
SANITIZE_LINK = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-shared-libasan"]


def clang() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "llvm", "bin", "clang")


def sanitizer_runtime() -> str:
    """Path of clang's shared AddressSanitizer runtime (to preload into python)."""
    return subprocess.run([clang(), "-print-file-name=libclang_rt.asan-x86_64.so"], check=True,
                          capture_output=True, text=True).stdout.strip()


def _compile(src: str, verbose: bool, sanitize: bool = False, trace: bool = False) -> pathlib.Path:
    obj = BUILD / (src + ".o")
    cmd = [hipcc(), *COMMON, *(SANITIZE_HOST if sanitize else []), *(["-DFS_TRACE=1"] if trace else []),
           "-x", "hip", "-c", str(CSRC / src), "-o", str(obj)]
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


def build(verbose: bool = False, sanitize: bool = False, trace: bool = False) -> pathlib.Path:
    BUILD.mkdir(exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, sanitize, trace), SOURCES))
    tmp = str(LIB) + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-Wl,-soname,libfastseq_hip.so",
           *(SANITIZE_LINK if sanitize else []), *map(str, objs), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    build_ext(verbose, sanitize)
    return LIB


def build_ext(verbose: bool = False, sanitize: bool = False) -> pathlib.Path:
    """The CPython module that marshals arguments into the C ABI."""
    tmp = str(EXT) + ".tmp"
    cc = [clang(), "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-shared-libasan",
          "-fno-omit-frame-pointer"] if sanitize else ["gcc"]
    cmd = [*cc, "-std=c11", "-O2", "-fPIC", "-shared", "-Wall", "-Wextra", "-Werror",
           f"-I{sysconfig.get_paths()['include']}", f"-I{ROOT / 'include'}", str(CSRC / "pyext.c"),
           f"-L{PKG}", "-lfastseq_hip", "-Wl,-rpath,$ORIGIN", "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, EXT)
    return EXT


if __name__ == "__main__":
    import sys
    print(build(verbose=True, sanitize="--sanitize" in sys.argv[1:], trace="--trace" in sys.argv[1:]))
