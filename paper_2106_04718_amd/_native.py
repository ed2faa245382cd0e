"""Bindings of libfastseq_hip.so (the C ABI declared in include/fastseq_hip.h).

Only argument marshalling lives here.  ``lib()`` is a ctypes handle on the
library (every entry point, used for the size queries and the ABI tests);
``ext()`` is the CPython module built from csrc/pyext.c, which the launch
calls go through because it converts arguments in a fraction of ctypes'
time.  Both must have been built (``__graft_entry__.build()`` or
``python -m paper_2106_04718_amd.build``); if either is missing every call
raises -- there is no fallback path.
"""
import ctypes
import pathlib

_HERE = pathlib.Path(__file__).resolve().parent
LIB_PATH = _HERE / "libfastseq_hip.so"

FS_OK = 0
FS_ERR_INVALID_ARG = 1
FS_ERR_UNSUPPORTED = 2
FS_ERR_HIP = 3
FS_F32 = 0
FS_BF16 = 1
FS_TUNE_ATTN_PATH = 1
FS_TUNE_SELECT_SLICES = 2
FS_TUNE_VALIDATE = 3
ATTN_PATHS = {"auto": 0, "split": 1, "whole1": 2, "whole2": 3, "whole4": 4}

# (name, restype, argtypes) for every exported entry point.
_c_int, _c_size, _vp = ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p
SIGNATURES = [
    ("fs_abi_version", _c_int, []),
    ("fs_status_string", ctypes.c_char_p, [_c_int]),
    ("fs_last_error", ctypes.c_char_p, []),
    ("fs_beam_cross_attn_workspace_bytes", _c_size, [_c_int] * 6),
    ("fs_beam_cross_attn", _c_int,
     [_vp, _vp, _vp, _vp, _vp] + [_c_int] * 6 + [_vp, _c_size, _vp]),
    ("fs_beam_prefix_attn_workspace_bytes", _c_size, [_c_int] * 7),
    ("fs_beam_prefix_attn", _c_int,
     [_vp, _vp, _vp, _vp, _vp, _vp, _c_int, _c_int, _vp] + [_c_int] * 6 + [_vp, _c_size, _vp]),
    ("fs_ngram_block", _c_int, [_vp, _c_int, _c_int, _c_int, _c_int, _vp, _c_int, _vp]),
    ("fs_beam_decode_step", _c_int,
     [_vp] * 5 + [_c_int] * 6 + [_vp] + [_c_int] * 3 + [_vp, _c_int, _vp, _c_size, _vp]),
    ("fs_set_tuning", _c_int, [_c_int, _c_int]),
    ("fs_trace_set", _c_int, [_vp, _c_size]),
    ("fs_beam_decode_step_noalloc", _c_int,
     [_vp] * 5 + [_c_int] * 6 + [_vp] + [_c_int] * 3 + [_vp, _c_int, _vp]),
    ("fs_beam_select_workspace_bytes", _c_size, [_c_int] * 4),
    ("fs_beam_select", _c_int,
     [_vp, _vp, _vp, _c_int, _c_int, _c_int, _vp, _vp, _vp] + [_c_int] * 4 + [_vp, _c_size, _vp]),
    ("fs_cache_reorder", _c_int, [_vp, _vp, _vp] + [_c_int] * 7 + [_vp]),
    ("fs_beam_ancestry_step", _c_int, [_vp, _c_int, _vp] + [_c_int] * 3 + [_vp]),
    ("fs_beam_prefix_attn_indirect", _c_int,
     [_vp] * 7 + [_c_int] * 3 + [_vp] + [_c_int] * 6 + [_vp, _c_size, _vp]),
    ("fs_postproc_create", _c_int,
     [ctypes.POINTER(_vp), ctypes.c_char_p, _vp] + [_c_int] * 5 + [ctypes.c_char_p]),
    ("fs_postproc_submit", _c_int, [_vp, _vp, _c_int, _c_int, _c_int, _vp]),
    ("fs_postproc_flush", _c_int, [_vp]),
    ("fs_postproc_output", _c_size, [_vp, _vp, _c_size]),
    ("fs_postproc_busy_seconds", ctypes.c_double, [_vp]),
    ("fs_postproc_destroy", None, [_vp]),
]

_lib = None
_ext = None


class NativeError(RuntimeError):
    """A non-OK status from the library; ``status`` holds the fs_status_t."""

    def __init__(self, status: int, detail: str):
        super().__init__(f"{status_string(status)}: {detail}")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load the in-tree library once; raise if it was never built."""
    global _lib
    if _lib is None:
        if not LIB_PATH.exists():
            raise RuntimeError(
                f"{LIB_PATH} is not built; run __graft_entry__.build() "
                "(no CPU fallback exists for the decode-step kernels)")
        handle = ctypes.CDLL(str(LIB_PATH))
        for name, res, args in SIGNATURES:
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def ext():
    """The CPython marshalling module; raise if it was never built."""
    global _ext
    if _ext is None:
        lib()
        try:
            from . import _fastseq_ext
        except ImportError as e:
            raise RuntimeError("the _fastseq_ext module is not built; run __graft_entry__.build() "
                               "(no CPU fallback exists for the decode-step kernels)") from e
        _ext = _fastseq_ext
    return _ext


def status_string(status: int) -> str:
    return lib().fs_status_string(status).decode()


def last_error() -> str:
    return lib().fs_last_error().decode()


def check_lib(status: int) -> None:
    """Raise on a non-OK status of a call made through lib()."""
    if status != FS_OK:
        raise NativeError(status, last_error())


def check(status: int) -> None:
    """Raise on a non-OK status of a call made through ext()."""
    if status != FS_OK:
        raise NativeError(status, ext().fs_last_error())
