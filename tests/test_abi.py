"""The C ABI loads without a GPU, exports what include/fastseq_hip.h declares,
and rejects invalid arguments on the host before any HIP call.

No test here launches a kernel: every call below fails validation (or is an
empty problem) and returns before touching device memory, so the fake
pointers passed are never dereferenced.
"""
import ctypes
import pathlib
import re

import pytest

from paper_2106_04718_amd import _native as N

ROOT = pathlib.Path(__file__).resolve().parents[1]
FAKE = 1 << 20          # aligned, never dereferenced


def header_functions():
    names = set()
    for h in (ROOT / "include").glob("*.h"):
        text = re.sub(r"/\*.*?\*/", "", h.read_text(), flags=re.S)
        names.update(re.findall(r"\b(fs_[a-z0-9_]+)\s*\(", text))
    return names


def test_library_exports_every_declared_function():
    declared = header_functions()
    assert {"fs_beam_cross_attn", "fs_ngram_block", "fs_beam_cross_attn_workspace_bytes",
            "fs_abi_version", "fs_status_string", "fs_last_error"} <= declared
    lib = ctypes.CDLL(str(N.LIB_PATH))
    for name in declared:
        assert hasattr(lib, name), name
    assert {s[0] for s in N.SIGNATURES} == declared


def test_abi_version_and_status_strings():
    lib = N.lib()
    hdr = (ROOT / "include" / "fastseq_hip.h").read_text()
    assert lib.fs_abi_version() == int(re.search(r"#define FS_ABI_VERSION (\d+)", hdr).group(1))
    assert N.status_string(0) == "FS_OK"
    assert N.status_string(1) == "FS_ERR_INVALID_ARG"
    assert N.status_string(2) == "FS_ERR_UNSUPPORTED"
    assert N.status_string(3) == "FS_ERR_HIP"
    assert N.status_string(99) == "unknown status"


def attn(**kw):
    a = dict(q=FAKE, K=FAKE * 2, V=FAKE * 3, src_len=FAKE * 4, out=FAKE * 5,
             B=2, k=4, H=2, S=64, D=16, dtype=N.FS_F32, ws=FAKE * 6, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    return N.lib().fs_beam_cross_attn(a["q"], a["K"], a["V"], a["src_len"], a["out"], a["B"], a["k"],
                                      a["H"], a["S"], a["D"], a["dtype"], a["ws"], a["ws_bytes"],
                                      a["stream"])


@pytest.mark.parametrize("kw,status,needle", [
    (dict(B=-1), N.FS_ERR_INVALID_ARG, "negative"),
    (dict(S=-5), N.FS_ERR_INVALID_ARG, "negative"),
    (dict(D=48), N.FS_ERR_UNSUPPORTED, "D=48"),
    (dict(D=0), N.FS_ERR_UNSUPPORTED, "D=0"),
    (dict(k=9), N.FS_ERR_UNSUPPORTED, "k=9"),
    (dict(dtype=7), N.FS_ERR_UNSUPPORTED, "dtype"),
    (dict(q=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(K=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(src_len=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(out=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(q=FAKE + 4), N.FS_ERR_INVALID_ARG, "aligned"),
    (dict(V=FAKE * 3 + 8), N.FS_ERR_INVALID_ARG, "aligned"),
    (dict(src_len=FAKE * 4 + 2), N.FS_ERR_INVALID_ARG, "aligned"),
    (dict(out=FAKE), N.FS_ERR_INVALID_ARG, "overlaps"),
    (dict(out=FAKE * 2 + 64), N.FS_ERR_INVALID_ARG, "overlaps"),
    (dict(ws_bytes=16), N.FS_ERR_INVALID_ARG, "workspace"),
    (dict(ws=None), N.FS_ERR_INVALID_ARG, "workspace"),
    (dict(ws=FAKE * 6 + 4), N.FS_ERR_INVALID_ARG, "aligned"),
    (dict(ws=FAKE * 3), N.FS_ERR_INVALID_ARG, "overlaps"),
    (dict(B=1 << 20, H=1 << 12), N.FS_ERR_INVALID_ARG, "too large"),
])
def test_cross_attn_rejects(kw, status, needle):
    assert attn(**kw) == status
    assert needle in N.last_error()


def test_cross_attn_empty_problems_return_ok_without_launch():
    for kw in (dict(B=0), dict(k=0), dict(H=0)):
        assert attn(q=None, K=None, V=None, src_len=None, out=None, ws=None, ws_bytes=0, **kw) == N.FS_OK
        assert N.last_error() == ""


def test_workspace_bytes():
    f = N.lib().fs_beam_cross_attn_workspace_bytes
    assert f(0, 4, 16, 1024, 64, N.FS_BF16) == 0
    # S = 0: one empty chunk column of 4 tiles, and a counter per (b, h)
    assert f(2, 4, 2, 0, 16, N.FS_F32) == 2 * 2 * 4 * 4 * 18 * 8 + 2 * 2 * 8
    assert f(2, 4, 2, 64, 48, N.FS_F32) == 2**64 - 1
    assert f(-1, 4, 2, 64, 16, N.FS_F32) == 2**64 - 1
    # per (b, h, 64-key tile): k * (D + 2) 8-byte tagged partials (tiles of
    # four 256-key chunks at D = 64, bf16), then one 8-byte counter per (b, h)
    # for captured calls
    a = f(32, 4, 16, 1024, 64, N.FS_BF16)
    assert a == 32 * 16 * 16 * 4 * 66 * 8 + 32 * 16 * 8
    assert f(64, 4, 16, 1024, 64, N.FS_BF16) == 2 * a
    assert f(32, 4, 16, 1025, 64, N.FS_BF16) > a
    assert f(32, 4, 16, 1023, 64, N.FS_BF16) == a


def ngram(**kw):
    a = dict(tokens=FAKE, ld=8, rows=4, t=8, n=3, logits=FAKE * 8, V=100, stream=None)
    a.update(kw)
    return N.lib().fs_ngram_block(a["tokens"], a["ld"], a["rows"], a["t"], a["n"], a["logits"],
                                  a["V"], a["stream"])


@pytest.mark.parametrize("kw,status,needle", [
    (dict(n=0), N.FS_ERR_INVALID_ARG, "n=0"),
    (dict(n=-2), N.FS_ERR_INVALID_ARG, "n=-2"),
    (dict(rows=-1), N.FS_ERR_INVALID_ARG, "negative"),
    (dict(t=-1), N.FS_ERR_INVALID_ARG, "negative"),
    (dict(V=-1), N.FS_ERR_INVALID_ARG, "negative"),
    (dict(ld=4), N.FS_ERR_INVALID_ARG, "ld_tokens"),
    (dict(tokens=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(logits=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(tokens=FAKE + 2), N.FS_ERR_INVALID_ARG, "aligned"),
    (dict(logits=FAKE + 64), N.FS_ERR_INVALID_ARG, "overlap"),
])
def test_ngram_rejects(kw, status, needle):
    assert ngram(**kw) == status
    assert needle in N.last_error()


def test_ngram_no_window_returns_ok_without_launch():
    # t < n and rows == 0 have no window; V == 0 leaves nothing writable
    assert ngram(tokens=None, logits=None, t=2, n=3) == N.FS_OK
    assert ngram(tokens=None, logits=None, rows=0) == N.FS_OK
    assert ngram(logits=None, V=0) == N.FS_OK


def test_validation_runs_before_any_hip_call():
    # A rejected call must not initialise HIP (there is no GPU here): the
    # status is the argument error, not FS_ERR_HIP.
    assert attn(D=48) == N.FS_ERR_UNSUPPORTED
    assert ngram(n=0) == N.FS_ERR_INVALID_ARG


def test_marshalling_module_reaches_the_same_library():
    # The launch calls go through the CPython module built from pyext.c; it
    # must bind the very library that ctypes loads (one copy, one
    # thread-local error slot), and pass every argument through unchanged.
    E = N.ext()
    for name in ("fs_beam_cross_attn", "fs_beam_prefix_attn", "fs_ngram_block", "fs_last_error"):
        assert callable(getattr(E, name)), name
    assert E.fs_ngram_block(FAKE, 4, 2, 5, 3, FAKE * 2, 7, None) == N.FS_ERR_INVALID_ARG
    assert "ld_tokens=4 < t=5" in E.fs_last_error()
    assert "ld_tokens=4 < t=5" in N.last_error()
    st = E.fs_beam_cross_attn(FAKE, FAKE * 2, FAKE * 3, FAKE * 4, FAKE * 5, 2, 9, 2, 64, 16, N.FS_F32,
                              FAKE * 6, 1 << 30, None)
    assert st == N.FS_ERR_UNSUPPORTED and "k=9" in E.fs_last_error()
    st = E.fs_beam_prefix_attn(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 3, 4, FAKE, 1, 1, 1, 1, 16, N.FS_F32,
                               FAKE, 1 << 20, None)
    assert st == N.FS_ERR_INVALID_ARG and "t=4 exceeds" in E.fs_last_error()
    with pytest.raises(TypeError):
        E.fs_ngram_block(FAKE, 4, 2)
    with pytest.raises(OverflowError):
        E.fs_ngram_block(FAKE, 1 << 40, 2, 5, 3, FAKE * 2, 7, None)


def select(**kw):
    a = dict(logits=FAKE, bs=FAKE * 64, tokens=FAKE * 128, ld=8, t=8, n=3, os=FAKE * 256, ob=FAKE * 320,
             ot=FAKE * 384, B=2, k=4, V=100, c=8, ws=FAKE * 512, wsb=1 << 20, stream=None)
    a.update(kw)
    return N.lib().fs_beam_select(a["logits"], a["bs"], a["tokens"], a["ld"], a["t"], a["n"], a["os"], a["ob"],
                                  a["ot"], a["B"], a["k"], a["V"], a["c"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status,needle", [
    (dict(c=17), N.FS_ERR_UNSUPPORTED, "c=17"),
    (dict(c=0), N.FS_ERR_UNSUPPORTED, "c=0"),
    (dict(k=17), N.FS_ERR_UNSUPPORTED, "k=17"),
    (dict(k=1, V=3, c=4), N.FS_ERR_INVALID_ARG, "c=4 > k*V"),
    (dict(B=-1), N.FS_ERR_INVALID_ARG, "negative"),
    (dict(n=-1), N.FS_ERR_INVALID_ARG, "n=-1"),
    (dict(ld=4), N.FS_ERR_INVALID_ARG, "ld_tokens"),
    (dict(logits=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(os=FAKE * 256 + 2), N.FS_ERR_INVALID_ARG, "aligned"),
    (dict(wsb=8), N.FS_ERR_INVALID_ARG, "workspace"),
    (dict(ob=FAKE * 256 + 4), N.FS_ERR_INVALID_ARG, "overlap"),
])
def test_select_rejects(kw, status, needle):
    assert select(**kw) == status
    assert needle in N.last_error()


def test_select_workspace_bytes_and_empty_batch():
    f = N.lib().fs_beam_select_workspace_bytes
    assert f(0, 4, 100, 8) == 0
    # one slice per row at V = 100, then one counter per source
    assert f(2, 4, 100, 8) == 2 * 4 * 1 * (2 + 2 * 8) * 8 + 2 * 8
    assert f(2, 17, 100, 8) == ctypes.c_size_t(-1).value
    assert select(B=0, logits=None, bs=None, tokens=None, os=None, ob=None, ot=None, ws=None, wsb=0) == N.FS_OK


def reorder(**kw):
    a = dict(K=FAKE, V=FAKE * 64, parent=FAKE * 128, B=2, k=4, H=2, T=10, t=5, D=16, dtype=N.FS_BF16, stream=None)
    a.update(kw)
    return N.lib().fs_cache_reorder(a["K"], a["V"], a["parent"], a["B"], a["k"], a["H"], a["T"], a["t"], a["D"],
                                    a["dtype"], a["stream"])


@pytest.mark.parametrize("kw,status,needle", [
    (dict(t=11), N.FS_ERR_INVALID_ARG, "t=11 > T=10"),
    (dict(B=-1), N.FS_ERR_INVALID_ARG, "negative"),
    (dict(k=17), N.FS_ERR_UNSUPPORTED, "k=17"),
    (dict(k=0), N.FS_ERR_UNSUPPORTED, "k=0"),
    (dict(dtype=7), N.FS_ERR_UNSUPPORTED, "dtype"),
    (dict(D=3), N.FS_ERR_UNSUPPORTED, "4-byte"),
    (dict(K=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(parent=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(V=FAKE * 64 + 2), N.FS_ERR_INVALID_ARG, "aligned"),
    (dict(V=FAKE + 64), N.FS_ERR_INVALID_ARG, "K overlaps V"),
    (dict(parent=FAKE + 64), N.FS_ERR_INVALID_ARG, "parent overlaps"),
])
def test_reorder_rejects(kw, status, needle):
    assert reorder(**kw) == status
    assert needle in N.last_error()


def test_reorder_nothing_to_move_returns_ok_without_launch():
    assert reorder(K=None, parent=None, t=0) == N.FS_OK
    assert reorder(K=None, parent=None, B=0) == N.FS_OK
    assert reorder(K=None, parent=None, H=0) == N.FS_OK
    # the marshalling module reaches the same entry point
    E = N.ext()
    assert E.fs_cache_reorder(FAKE, FAKE, FAKE * 128, 2, 4, 2, 10, 5, 16, N.FS_BF16, None) == N.FS_ERR_INVALID_ARG
    assert "K overlaps V" in E.fs_last_error()


def ancestry(**kw):
    a = dict(anc=FAKE, ld=10, parent=FAKE * 64, B=2, k=4, t=3, stream=None)
    a.update(kw)
    return N.lib().fs_beam_ancestry_step(a["anc"], a["ld"], a["parent"], a["B"], a["k"], a["t"], a["stream"])


@pytest.mark.parametrize("kw,status,needle", [
    (dict(t=10), N.FS_ERR_INVALID_ARG, "column t=10"),
    (dict(B=-1), N.FS_ERR_INVALID_ARG, "negative"),
    (dict(k=17), N.FS_ERR_UNSUPPORTED, "k=17"),
    (dict(anc=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(parent=FAKE * 64 + 2), N.FS_ERR_INVALID_ARG, "aligned"),
    (dict(parent=FAKE + 8), N.FS_ERR_INVALID_ARG, "overlaps"),
])
def test_ancestry_rejects(kw, status, needle):
    assert ancestry(**kw) == status
    assert needle in N.last_error()
    assert ancestry(B=0, anc=None, parent=None) == N.FS_OK


def indirect(**kw):
    a = dict(q=FAKE, Kp=FAKE * 2, Vp=FAKE * 3, plen=FAKE * 4, Kt=FAKE * 5, Vt=FAKE * 6, anc=FAKE * 7, ld=8,
             T=8, t=5, out=FAKE * 9, B=2, k=4, H=2, N=16, D=64, dtype=N.FS_BF16, ws=FAKE * 10, wsb=1 << 24,
             stream=None)
    a.update(kw)
    return N.lib().fs_beam_prefix_attn_indirect(a["q"], a["Kp"], a["Vp"], a["plen"], a["Kt"], a["Vt"], a["anc"],
                                                a["ld"], a["T"], a["t"], a["out"], a["B"], a["k"], a["H"], a["N"],
                                                a["D"], a["dtype"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status,needle", [
    (dict(anc=None), N.FS_ERR_INVALID_ARG, "null ancestry table"),
    (dict(ld=4), N.FS_ERR_INVALID_ARG, "ld_anc=4 < t=5"),
    (dict(anc=FAKE * 7 + 2), N.FS_ERR_INVALID_ARG, "anc must be 4-byte aligned"),
    (dict(anc=FAKE * 9 + 16), N.FS_ERR_INVALID_ARG, "out overlaps the ancestry table"),
    (dict(t=9), N.FS_ERR_INVALID_ARG, "exceeds"),
    (dict(D=48), N.FS_ERR_UNSUPPORTED, "D=48"),
])
def test_indirect_prefix_attn_rejects(kw, status, needle):
    assert indirect(**kw) == status
    assert needle in N.last_error()


def test_indirect_prefix_attn_needs_no_table_without_generated_tokens():
    # t == 0 reads no table: a null anc passes validation (and B == 0 launches nothing)
    assert indirect(anc=None, t=0, B=0) == N.FS_OK


def test_block_over_2gib_is_unsupported():
    # one (source, head) block of K/V is read through a 32-bit byte range
    f = N.lib().fs_beam_cross_attn_workspace_bytes
    assert f(1, 1, 1, 1 << 24, 128, N.FS_BF16) == 2**64 - 1
    assert "2 GiB" in N.last_error()
    assert attn(B=1, k=1, H=1, S=1 << 24, D=128, dtype=N.FS_BF16) == N.FS_ERR_UNSUPPORTED
    assert "2 GiB" in N.last_error()
    # just under the limit passes the size checks (then fails on a null pointer, before any launch)
    S = 0x7ff00000 // (128 * 2)
    assert f(1, 1, 1, S, 128, N.FS_BF16) != 2**64 - 1
    assert attn(B=1, k=1, H=1, S=S, D=128, dtype=N.FS_BF16, q=None) == N.FS_ERR_INVALID_ARG


def test_prefix_generated_block_over_2gib_is_unsupported():
    lib = N.lib()
    T = (0x7ff00000 // (64 * 4)) + 1
    far = 1 << 40   # the generated-token blocks span 2 GiB: keep every fake buffer apart
    st = lib.fs_beam_prefix_attn(FAKE, FAKE * 2, FAKE * 3, FAKE * 4, far, 2 * far, T, 1, 3 * far,
                                 1, 1, 1, 16, 64, N.FS_F32, 4 * far, 1 << 30, None)
    assert st == N.FS_ERR_UNSUPPORTED and "2 GiB" in N.last_error()


def step(**kw):
    a = dict(q=FAKE, K=FAKE * 2, V=FAKE * 3, src_len=FAKE * 4, out=FAKE * 5,
             B=2, k=4, H=2, S=64, D=16, dtype=N.FS_F32, tokens=FAKE * 7, ld=8, t=8, n=3,
             logits=FAKE * 8, vocab=100, ws=FAKE * 6, ws_bytes=1 << 16, stream=None)
    a.update(kw)
    return N.lib().fs_beam_decode_step(a["q"], a["K"], a["V"], a["src_len"], a["out"], a["B"], a["k"], a["H"],
                                       a["S"], a["D"], a["dtype"], a["tokens"], a["ld"], a["t"], a["n"],
                                       a["logits"], a["vocab"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,status,needle", [
    (dict(D=48), N.FS_ERR_UNSUPPORTED, "D=48"),
    (dict(n=0), N.FS_ERR_INVALID_ARG, "n=0"),
    (dict(ld=4), N.FS_ERR_INVALID_ARG, "ld_tokens"),
    (dict(q=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(tokens=None), N.FS_ERR_INVALID_ARG, "null"),
    (dict(out=FAKE * 2), N.FS_ERR_INVALID_ARG, "overlaps"),
    (dict(logits=FAKE * 7 + 16), N.FS_ERR_INVALID_ARG, "overlap tokens"),
    (dict(logits=FAKE * 5), N.FS_ERR_INVALID_ARG, "attention argument"),
    (dict(logits=FAKE * 2 + 128), N.FS_ERR_INVALID_ARG, "attention argument"),
    (dict(logits=FAKE * 6), N.FS_ERR_INVALID_ARG, "attention argument"),
    (dict(tokens=FAKE * 5), N.FS_ERR_INVALID_ARG, "tokens overlap"),
    (dict(ws_bytes=16), N.FS_ERR_INVALID_ARG, "workspace"),
])
def test_decode_step_rejects(kw, status, needle):
    assert step(**kw) == status
    assert needle in N.last_error()


def test_decode_step_empty_halves_return_ok_without_launch():
    # no attention and no n-gram window: nothing runs, nothing is read
    nulls = dict(q=None, K=None, V=None, src_len=None, out=None, ws=None, ws_bytes=0, tokens=None, logits=None)
    assert step(B=0, **nulls) == N.FS_OK
    assert step(H=0, t=2, n=3, **nulls) == N.FS_OK
    assert step(H=0, vocab=0, **nulls) == N.FS_OK


def test_tuning_controls():
    lib = N.lib()
    assert lib.fs_set_tuning(99, 0) == -1
    assert lib.fs_set_tuning(N.FS_TUNE_ATTN_PATH, 17) == -1
    assert lib.fs_set_tuning(N.FS_TUNE_SELECT_SLICES, -3) == -1
    prev = lib.fs_set_tuning(N.FS_TUNE_ATTN_PATH, N.ATTN_PATHS["whole1"])
    assert prev == N.ATTN_PATHS["auto"]
    assert lib.fs_set_tuning(N.FS_TUNE_ATTN_PATH, prev) == N.ATTN_PATHS["whole1"]
    assert lib.fs_set_tuning(N.FS_TUNE_SELECT_SLICES, 5) == 0
    assert lib.fs_set_tuning(N.FS_TUNE_SELECT_SLICES, 0) == 5
    assert lib.fs_set_tuning(N.FS_TUNE_VALIDATE, 2) == -1
    was = lib.fs_set_tuning(N.FS_TUNE_VALIDATE, 1)
    assert lib.fs_set_tuning(N.FS_TUNE_VALIDATE, was) == 1
    hdr = (ROOT / "include" / "fastseq_hip.h").read_text()
    for name, v in N.ATTN_PATHS.items():
        assert re.search(rf"FS_ATTN_PATH_{name.upper()} = {v}\b", hdr), name


def test_noalloc_step_refuses_records_beyond_its_scratch_array():
    # 127 (source, head) rows take the split-KV form; 64 chunks of records at
    # k = 8, D = 128 need about 67 MB, more than the library's array
    lib = N.lib()
    st = lib.fs_beam_decode_step_noalloc(FAKE, FAKE * 2, FAKE * 3, FAKE * 4, FAKE * 5, 1, 8, 127, 8192, 128,
                                         N.FS_BF16, FAKE * 6, 8, 8, 3, FAKE * 7, 100, None)
    assert st == N.FS_ERR_UNSUPPORTED and "scratch array" in N.last_error()
    # argument errors are those of fs_beam_decode_step
    st = lib.fs_beam_decode_step_noalloc(None, FAKE * 2, FAKE * 3, FAKE * 4, FAKE * 5, 2, 4, 2, 64, 16,
                                         N.FS_F32, FAKE * 6, 8, 8, 3, FAKE * 7, 100, None)
    assert st == N.FS_ERR_INVALID_ARG and "null" in N.last_error()
    hdr = (ROOT / "include" / "fastseq_hip.h").read_text()
    assert re.search(r"#define FS_NOALLOC_SCRATCH_BYTES \(8u << 20\)", hdr)


def test_postproc_rejects_bad_arguments_before_any_hip_call():
    import ctypes
    import numpy as np
    lib = N.lib()
    h = ctypes.c_void_p()
    off = np.array([0, 1, 3], np.int64)
    data = b"abc"
    assert lib.fs_postproc_create(None, data, off.ctypes.data, 2, 1, 4, 4, 2, None) == N.FS_ERR_INVALID_ARG
    assert lib.fs_postproc_create(ctypes.byref(h), data, off.ctypes.data, 0, 1, 4, 4, 2, None) == N.FS_ERR_INVALID_ARG
    assert "vocabulary" in N.last_error()
    assert lib.fs_postproc_create(ctypes.byref(h), data, off.ctypes.data, 2, 1, 0, 4, 2, None) == N.FS_ERR_INVALID_ARG
    assert lib.fs_postproc_create(ctypes.byref(h), data, off.ctypes.data, 2, 1, 4, 4, 0, None) == N.FS_ERR_INVALID_ARG
    bad = np.array([0, 2, 1], np.int64)
    assert lib.fs_postproc_create(ctypes.byref(h), data, bad.ctypes.data, 2, 1, 4, 4, 2, None) == N.FS_ERR_INVALID_ARG
    assert "decrease" in N.last_error()
    assert lib.fs_postproc_create(ctypes.byref(h), data, off.ctypes.data, 2, 1, 1 << 16, 1 << 16, 2, None) \
        == N.FS_ERR_UNSUPPORTED
    assert lib.fs_postproc_create(ctypes.byref(h), data, off.ctypes.data, 2, 1, 4, 4, 2,
                                  b"/nonexistent-dir/out.txt") == N.FS_ERR_INVALID_ARG
    assert h.value is None
    assert lib.fs_postproc_submit(None, FAKE, 4, 2, 4, None) == N.FS_ERR_INVALID_ARG
    assert lib.fs_postproc_flush(None) == N.FS_ERR_INVALID_ARG
    assert lib.fs_postproc_output(None, None, 0) == 0
    lib.fs_postproc_destroy(None)


def test_trace_set_needs_a_trace_build():
    lib = N.lib()
    assert lib.fs_trace_set(None, 64) == N.FS_ERR_INVALID_ARG and "null trace buffer" in N.last_error()
    assert lib.fs_trace_set(FAKE + 4, 64) == N.FS_ERR_INVALID_ARG and "aligned" in N.last_error()
    # a normal build holds no tracing code: refused before any HIP call
    assert lib.fs_trace_set(None, 0) == N.FS_ERR_UNSUPPORTED and "without workgroup tracing" in N.last_error()
