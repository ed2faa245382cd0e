"""Torch-tensor front end of the decode-step library.

Each function checks tensor placement, dtype and layout, then passes raw
device pointers and torch's current HIP stream to the C ABI.  PyTorch only
provides memory and streams here; all arithmetic runs in the HIP kernels.

A decode step is a few tens of microseconds of GPU time, so the per-call
host work is kept small: workspace sizes are cached per shape, the stream
handle is read without building a Stream object, the device is switched
only when the tensors are not on the current one, and the call itself goes
through the CPython marshalling module rather than ctypes.
"""
from __future__ import annotations

import contextlib

import torch

from . import _native as _N

_native_lib = _N.lib
_DTYPES = {torch.float32: _N.FS_F32, torch.bfloat16: _N.FS_BF16}
_WS_BYTES: dict = {}

_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_cur_device = getattr(torch._C, "_cuda_getDevice", None) or torch.cuda.current_device


def _stream_ptr(device: torch.device) -> int:
    if _raw_stream is not None:
        return _raw_stream(device.index)
    return torch.cuda.current_stream(device).cuda_stream


def _on(device: torch.device):
    """A device guard, or nothing if ``device`` is already current."""
    if device.index == _cur_device():
        return contextlib.nullcontext()
    return torch.cuda.device(device)


def _need_cuda(name: str, t: torch.Tensor) -> None:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def new_workspace(nbytes: int, device) -> torch.Tensor:
    """A zero-filled workspace of at least ``nbytes`` for the attention calls.

    The library tags every word it writes with its call, so a workspace
    needs zero-filling only once, before its first use; reuse it across
    calls (of any size that fits) without clearing.  A workspace of calls
    captured into a graph must keep serving calls of the same sizes while
    the graph is replayed.
    """
    return torch.zeros(max(int(nbytes), 16), dtype=torch.uint8, device=device)


def _size_or_raise(n: int) -> int:
    if n == 2**64 - 1:
        raise _N.NativeError(_N.FS_ERR_UNSUPPORTED, _N.last_error())
    return int(n)


def beam_cross_attn_workspace_bytes(B: int, k: int, H: int, S: int, D: int,
                                    dtype: torch.dtype = torch.bfloat16) -> int:
    """Bytes of workspace fs_beam_cross_attn needs for these sizes."""
    key = ("x", B, k, H, S, D, dtype)
    n = _WS_BYTES.get(key)
    if n is None:
        n = _size_or_raise(_N.lib().fs_beam_cross_attn_workspace_bytes(B, k, H, S, D, _DTYPES[dtype]))
        _WS_BYTES[key] = n
    return n


def beam_cross_attn(q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, src_len: torch.Tensor,
                    out: torch.Tensor | None = None,
                    workspace: torch.Tensor | None = None) -> torch.Tensor:
    """Encoder-decoder attention over de-duplicated K/V (Appendix B, Eq. 4).

    q [B,k,H,D], K/V [B,H,S,D] (same dtype: float32 or bfloat16), src_len [B]
    int32.  Returns out [B,k,H,D] in the input dtype.  ``workspace`` (from
    :func:`new_workspace`, zero-filled once, then reused) avoids an
    allocation and a fill per call.
    """
    for name, t in (("q", q), ("K", K), ("V", V), ("src_len", src_len)):
        _need_cuda(name, t)
    if q.dim() != 4 or K.dim() != 4 or K.shape != V.shape:
        raise ValueError("q must be [B,k,H,D] and K, V [B,H,S,D]")
    B, k, H, D = q.shape
    if K.shape[0] != B or K.shape[1] != H or K.shape[3] != D:
        raise ValueError(f"shape mismatch: q{tuple(q.shape)} K{tuple(K.shape)}")
    S = K.shape[2]
    dt = _DTYPES.get(q.dtype)
    if dt is None or K.dtype != q.dtype or V.dtype != q.dtype:
        raise ValueError("q, K and V must all be float32 or all bfloat16")
    if src_len.dtype != torch.int32 or src_len.shape != (B,):
        raise ValueError("src_len must be int32 [B]")
    dev = q.device
    if K.device != dev or V.device != dev or src_len.device != dev:
        raise ValueError("all tensors must be on one device")
    if out is None:
        out = torch.empty_like(q)
    else:
        _need_cuda("out", out)
        if out.shape != q.shape or out.dtype != q.dtype or out.device != dev:
            raise ValueError("out must match q in shape, dtype and device")
    if workspace is None:
        workspace = new_workspace(beam_cross_attn_workspace_bytes(B, k, H, S, D, q.dtype), dev)
    else:
        _need_cuda("workspace", workspace)
    with _on(dev):
        _N.check(_N.ext().fs_beam_cross_attn(
            q.data_ptr(), K.data_ptr(), V.data_ptr(), src_len.data_ptr(), out.data_ptr(),
            B, k, H, S, D, dt, workspace.data_ptr(), workspace.numel() * workspace.element_size(),
            _stream_ptr(dev)))
    return out


def beam_decode_step(q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, src_len: torch.Tensor,
                     tokens: torch.Tensor, n: int, logits: torch.Tensor, t: int | None = None,
                     out: torch.Tensor | None = None,
                     workspace: torch.Tensor | None = None) -> torch.Tensor:
    """The decode step in one launch: :func:`beam_cross_attn` and
    :func:`ngram_block` on the step's B*k hypotheses (tokens [B*k, ld],
    logits [B*k, vocab], modified in place).  Bit for bit the two calls.
    Returns ``out``."""
    for name, x in (("q", q), ("K", K), ("V", V), ("src_len", src_len)):
        _need_cuda(name, x)
    _need_cuda("logits", logits)
    if q.dim() != 4 or K.dim() != 4 or K.shape != V.shape:
        raise ValueError("q must be [B,k,H,D] and K, V [B,H,S,D]")
    B, k, H, D = q.shape
    if K.shape[0] != B or K.shape[1] != H or K.shape[3] != D:
        raise ValueError(f"shape mismatch: q{tuple(q.shape)} K{tuple(K.shape)}")
    S = K.shape[2]
    dt = _DTYPES.get(q.dtype)
    if dt is None or K.dtype != q.dtype or V.dtype != q.dtype:
        raise ValueError("q, K and V must all be float32 or all bfloat16")
    if src_len.dtype != torch.int32 or src_len.shape != (B,):
        raise ValueError("src_len must be int32 [B]")
    if not isinstance(tokens, torch.Tensor) or tokens.device.type != "cuda":
        raise ValueError("tokens must be a GPU tensor")
    if tokens.dim() != 2 or tokens.dtype != torch.int32 or tokens.shape[0] != B * k:
        raise ValueError("tokens must be int32 [B*k, ld]")
    rows, cols = tokens.shape
    if rows > 0 and cols > 1 and tokens.stride(1) != 1:
        raise ValueError("tokens must have unit column stride")
    if logits.dim() != 2 or logits.dtype != torch.float32 or logits.shape[0] != rows:
        raise ValueError("logits must be float32 [B*k, vocab]")
    dev = q.device
    if any(x.device != dev for x in (K, V, src_len, tokens, logits)):
        raise ValueError("all tensors must be on one device")
    ld = tokens.stride(0) if rows > 1 else cols
    if t is None:
        t = cols
    if t > cols:
        raise ValueError("t exceeds the columns of tokens")
    if out is None:
        out = torch.empty_like(q)
    else:
        _need_cuda("out", out)
        if out.shape != q.shape or out.dtype != q.dtype or out.device != dev:
            raise ValueError("out must match q in shape, dtype and device")
    if workspace is None:
        workspace = new_workspace(beam_cross_attn_workspace_bytes(B, k, H, S, D, q.dtype), dev)
    else:
        _need_cuda("workspace", workspace)
    with _on(dev):
        _N.check(_N.ext().fs_beam_decode_step(
            q.data_ptr(), K.data_ptr(), V.data_ptr(), src_len.data_ptr(), out.data_ptr(),
            B, k, H, S, D, dt, tokens.data_ptr(), ld, int(t), int(n), logits.data_ptr(), logits.shape[1],
            workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream_ptr(dev)))
    return out


def set_tuning(knob: int, value: int) -> int:
    """fs_set_tuning: replace a size rule for every later call in the
    process; returns the previous value."""
    prev = _N.lib().fs_set_tuning(int(knob), int(value))
    if prev < 0:
        raise ValueError(f"unknown tuning knob {knob} or value {value}")
    return prev


def trace_set(buffer: torch.Tensor | None) -> None:
    """fs_trace_set: in a library built with workgroup tracing
    (``build(trace=True)``), the device buffer the attention and selection
    kernels write their workgroup timelines to (8 int64 words per
    workgroup); None stops tracing.  Raises in other builds."""
    if buffer is None:
        st = _N.lib().fs_trace_set(None, 0)
    else:
        _need_cuda("buffer", buffer)
        st = _N.lib().fs_trace_set(buffer.data_ptr(), buffer.numel() * buffer.element_size())
    _N.check(st)


@contextlib.contextmanager
def attn_path(name: str):
    """Force one decomposition of the attention calls inside the block
    ('auto', 'split', 'whole1', 'whole2', 'whole4'); every decomposition
    gives the same bits."""
    prev = set_tuning(_N.FS_TUNE_ATTN_PATH, _N.ATTN_PATHS[name])
    try:
        yield
    finally:
        set_tuning(_N.FS_TUNE_ATTN_PATH, prev)


@contextlib.contextmanager
def validate_lengths(on: bool = True):
    """Debug mode inside the block: the attention calls copy the lengths to
    the host and reject out-of-range ones (FS_VALIDATE)."""
    prev = set_tuning(_N.FS_TUNE_VALIDATE, int(on))
    try:
        yield
    finally:
        set_tuning(_N.FS_TUNE_VALIDATE, prev)


@contextlib.contextmanager
def select_slices(n: int):
    """Force fs_beam_select's vocabulary slice count inside the block (0: the size rule)."""
    prev = set_tuning(_N.FS_TUNE_SELECT_SLICES, n)
    try:
        yield
    finally:
        set_tuning(_N.FS_TUNE_SELECT_SLICES, prev)


def beam_prefix_attn_workspace_bytes(B: int, k: int, H: int, N: int, T: int, D: int,
                                     dtype: torch.dtype = torch.bfloat16) -> int:
    """Bytes of workspace fs_beam_prefix_attn needs for these sizes."""
    key = ("p", B, k, H, N, T, D, dtype)
    n = _WS_BYTES.get(key)
    if n is None:
        n = _size_or_raise(_native_lib().fs_beam_prefix_attn_workspace_bytes(B, k, H, N, T, D, _DTYPES[dtype]))
        _WS_BYTES[key] = n
    return n


def beam_prefix_attn(q: torch.Tensor, Kp: torch.Tensor, Vp: torch.Tensor, prefix_len: torch.Tensor,
                     Kt: torch.Tensor, Vt: torch.Tensor, t: int, out: torch.Tensor | None = None,
                     workspace: torch.Tensor | None = None, anc: torch.Tensor | None = None) -> torch.Tensor:
    """Self-attention over a split cache (Appendix A, Eq. 2-3).

    q [B,k,H,D]; Kp, Vp [B,H,N,D] shared prefix with prefix_len [B] int32;
    Kt, Vt [B*k,H,T,D] per-beam generated tokens of which rows [0, t) are
    used.  One softmax covers both parts.  Returns out [B,k,H,D].  With
    ``anc`` ([B*k, ld] int32 ancestry table, see :func:`ancestry_step`) the
    generated row tau of hypothesis b*k + i is read from the block of
    hypothesis b*k + anc[b*k + i, tau] instead of its own.
    """
    for name, x in (("q", q), ("Kp", Kp), ("Vp", Vp), ("prefix_len", prefix_len), ("Kt", Kt), ("Vt", Vt)):
        _need_cuda(name, x)
    if q.dim() != 4 or Kp.dim() != 4 or Kp.shape != Vp.shape or Kt.dim() != 4 or Kt.shape != Vt.shape:
        raise ValueError("q [B,k,H,D], Kp/Vp [B,H,N,D], Kt/Vt [B*k,H,T,D]")
    B, k, H, D = q.shape
    Np, T = Kp.shape[2], Kt.shape[2]
    if Kp.shape != (B, H, Np, D) or Kt.shape != (B * k, H, T, D):
        raise ValueError(f"shape mismatch: q{tuple(q.shape)} Kp{tuple(Kp.shape)} Kt{tuple(Kt.shape)}")
    if q.dtype not in _DTYPES or any(x.dtype != q.dtype for x in (Kp, Vp, Kt, Vt)):
        raise ValueError("q, Kp, Vp, Kt and Vt must all be float32 or all bfloat16")
    if prefix_len.dtype != torch.int32 or prefix_len.shape != (B,):
        raise ValueError("prefix_len must be int32 [B]")
    dev = q.device
    if any(x.device != dev for x in (Kp, Vp, Kt, Vt, prefix_len)):
        raise ValueError("all tensors must be on one device")
    if out is None:
        out = torch.empty_like(q)
    else:
        _need_cuda("out", out)
        if out.shape != q.shape or out.dtype != q.dtype or out.device != dev:
            raise ValueError("out must match q in shape, dtype and device")
    if workspace is None:
        workspace = new_workspace(beam_prefix_attn_workspace_bytes(B, k, H, Np, T, D, q.dtype), dev)
    else:
        _need_cuda("workspace", workspace)
    if anc is not None:
        _need_cuda("anc", anc)
        if anc.dtype != torch.int32 or anc.dim() != 2 or anc.shape[0] != B * k or anc.device != dev:
            raise ValueError("anc must be int32 [B*k, ld] on q's device")
        if B * k > 1 and anc.shape[1] > 1 and anc.stride(1) != 1:
            raise ValueError("anc must have unit column stride")
        ld = anc.stride(0) if B * k > 1 else anc.shape[1]
        with _on(dev):
            _N.check(_N.ext().fs_beam_prefix_attn_indirect(
                q.data_ptr(), Kp.data_ptr(), Vp.data_ptr(), prefix_len.data_ptr(), Kt.data_ptr(), Vt.data_ptr(),
                anc.data_ptr(), ld, T, int(t), out.data_ptr(), B, k, H, Np, D, _DTYPES[q.dtype],
                workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream_ptr(dev)))
        return out
    with _on(dev):
        _N.check(_N.ext().fs_beam_prefix_attn(
            q.data_ptr(), Kp.data_ptr(), Vp.data_ptr(), prefix_len.data_ptr(), Kt.data_ptr(), Vt.data_ptr(),
            T, int(t), out.data_ptr(), B, k, H, Np, D, _DTYPES[q.dtype], workspace.data_ptr(),
            workspace.numel() * workspace.element_size(), _stream_ptr(dev)))
    return out


def ancestry_step(anc: torch.Tensor, parent: torch.Tensor, k: int, t: int) -> torch.Tensor:
    """One step of the ancestry table, in place (the reorder-free cache
    maintenance after a selection step).

    anc [B*k, ld] int32 (ld > t); parent [B*k] int32, the old beam each new
    hypothesis continues.  Columns tau < t of hypothesis b*k + j become those
    of b*k + parent[b*k + j]; column t becomes j (its new token, written to
    its own row).  Returns anc.
    """
    _need_cuda("anc", anc)
    _need_cuda("parent", parent)
    if anc.dtype != torch.int32 or anc.dim() != 2 or k < 1 or anc.shape[0] % k:
        raise ValueError("anc must be int32 [B*k, ld]")
    rows = anc.shape[0]
    if rows > 1 and anc.shape[1] > 1 and anc.stride(1) != 1:
        raise ValueError("anc must have unit column stride")
    if parent.dtype != torch.int32 or parent.shape != (rows,) or parent.device != anc.device:
        raise ValueError("parent must be int32 [B*k] on anc's device")
    ld = anc.stride(0) if rows > 1 else anc.shape[1]
    with _on(anc.device):
        _N.check(_N.ext().fs_beam_ancestry_step(anc.data_ptr(), ld, parent.data_ptr(), rows // k, int(k), int(t),
                                                _stream_ptr(anc.device)))
    return anc


def ngram_block(tokens: torch.Tensor, n: int, logits: torch.Tensor, t: int | None = None) -> torch.Tensor:
    """No-repeat-n-gram blocking in place (Section 4.2, Algorithm 1).

    tokens [rows, ld] int32 (row-contiguous; the first ``t`` columns are the
    history, default all); logits [rows, V] float32, contiguous.  Returns
    ``logits`` with banned entries set to -inf.
    """
    if not isinstance(tokens, torch.Tensor) or tokens.device.type != "cuda":
        raise ValueError("tokens must be a GPU tensor")
    _need_cuda("logits", logits)
    if tokens.dim() != 2 or tokens.dtype != torch.int32:
        raise ValueError("tokens must be int32 [rows, ld]")
    rows, cols = tokens.shape
    if rows > 0 and cols > 1 and tokens.stride(1) != 1:
        raise ValueError("tokens must have unit column stride")
    if logits.dim() != 2 or logits.dtype != torch.float32:
        raise ValueError("logits must be float32 [rows, V]")
    dev = tokens.device
    if logits.shape[0] != rows or logits.device != dev:
        raise ValueError("tokens and logits must have the same rows and device")
    ld = tokens.stride(0) if rows > 1 else cols
    if t is None:
        t = cols
    if t > cols:
        raise ValueError("t exceeds the columns of tokens")
    with _on(dev):
        _N.check(_N.ext().fs_ngram_block(tokens.data_ptr(), ld, rows, int(t), int(n),
                                         logits.data_ptr(), logits.shape[1], _stream_ptr(dev)))
    return logits


def beam_select_workspace_bytes(B: int, k: int, V: int, c: int) -> int:
    """Bytes of workspace fs_beam_select needs for these sizes."""
    key = ("s", B, k, V, c)
    n = _WS_BYTES.get(key)
    if n is None:
        n = _size_or_raise(_native_lib().fs_beam_select_workspace_bytes(B, k, V, c))
        _WS_BYTES[key] = n
    return n


def beam_select(logits: torch.Tensor, beam_scores: torch.Tensor, k: int, c: int,
                tokens: torch.Tensor | None = None, n: int = 0, t: int | None = None,
                out: tuple | None = None, workspace: torch.Tensor | None = None):
    """One beam-search selection step (Section 2.1) with no-repeat-n-gram bans
    (Section 4.2, Algorithm 1), in one pass over the logits.

    logits [B*k, V] float32 (not modified); beam_scores [B*k] float32;
    tokens [B*k, ld] int32 whose first ``t`` columns (default all) are the
    history, required when ``n > 0``.  Returns (scores float32 [B, c],
    beam int32 [B, c], token int32 [B, c]): each source's c best
    beam_score + log-softmax candidates, best first, ties to the smaller
    flat index beam*V + token.  ``out`` may pass the three output tensors.
    """
    _need_cuda("logits", logits)
    _need_cuda("beam_scores", beam_scores)
    if logits.dim() != 2 or logits.dtype != torch.float32:
        raise ValueError("logits must be float32 [B*k, V]")
    rows, V = logits.shape
    if k < 1 or rows % k:
        raise ValueError(f"rows={rows} is not a multiple of k={k}")
    B = rows // k
    dev = logits.device
    if beam_scores.dtype != torch.float32 or beam_scores.shape != (rows,) or beam_scores.device != dev:
        raise ValueError("beam_scores must be float32 [B*k] on the logits' device")
    ld, tp, tptr = 0, 0, 0
    if n > 0:
        if not isinstance(tokens, torch.Tensor) or tokens.device != dev:
            raise ValueError("tokens must be a GPU tensor on the logits' device when n > 0")
        if tokens.dim() != 2 or tokens.dtype != torch.int32 or tokens.shape[0] != rows:
            raise ValueError("tokens must be int32 [B*k, ld]")
        if rows > 0 and tokens.shape[1] > 1 and tokens.stride(1) != 1:
            raise ValueError("tokens must have unit column stride")
        ld = tokens.stride(0) if rows > 1 else tokens.shape[1]
        tp = tokens.shape[1] if t is None else int(t)
        if tp > tokens.shape[1]:
            raise ValueError("t exceeds the columns of tokens")
        tptr = tokens.data_ptr()
    if out is None:
        out = (torch.empty((B, c), dtype=torch.float32, device=dev),
               torch.empty((B, c), dtype=torch.int32, device=dev),
               torch.empty((B, c), dtype=torch.int32, device=dev))
    else:
        for o, dt in zip(out, (torch.float32, torch.int32, torch.int32)):
            _need_cuda("out", o)
            if o.shape != (B, c) or o.dtype != dt or o.device != dev:
                raise ValueError("out must be (float32, int32, int32) tensors of shape [B, c]")
    if workspace is None:
        workspace = new_workspace(beam_select_workspace_bytes(B, k, V, c), dev)
    else:
        _need_cuda("workspace", workspace)
    with _on(dev):
        _N.check(_N.ext().fs_beam_select(
            logits.data_ptr(), beam_scores.data_ptr(), tptr, ld, tp, int(n), out[0].data_ptr(),
            out[1].data_ptr(), out[2].data_ptr(), B, int(k), V, int(c), workspace.data_ptr(),
            workspace.numel() * workspace.element_size(), _stream_ptr(dev)))
    return out


def cache_reorder(K: torch.Tensor, V: torch.Tensor | None, parent: torch.Tensor, k: int,
                  t: int | None = None) -> None:
    """Per-beam cache reorder after a selection step (Section 2.2 cache
    maintenance; Section 4.1.1), in place.

    K, V [B*k, H, T, D] float32 or bfloat16 (V may be None); parent [B*k]
    int32, the old beam (within its source) each new hypothesis continues.
    Rows tau < ``t`` (default T) of hypothesis b*k + j become those of
    b*k + parent[b*k + j]; other rows, and beams whose parent is themselves or
    outside [0, k), keep their bytes.
    """
    _need_cuda("K", K)
    _need_cuda("parent", parent)
    if K.dim() != 4 or K.dtype not in _DTYPES or not K.is_contiguous():
        raise ValueError("K must be a contiguous float32/bfloat16 [B*k, H, T, D] tensor")
    rows, H, T, D = K.shape
    if k < 1 or rows % k:
        raise ValueError(f"rows={rows} is not a multiple of k={k}")
    dev = K.device
    if V is not None:
        _need_cuda("V", V)
        if V.shape != K.shape or V.dtype != K.dtype or V.device != dev or not V.is_contiguous():
            raise ValueError("V must match K (shape, dtype, device, contiguous)")
    if parent.dtype != torch.int32 or parent.shape != (rows,) or parent.device != dev:
        raise ValueError("parent must be int32 [B*k] on K's device")
    tp = T if t is None else int(t)
    with _on(dev):
        _N.check(_N.ext().fs_cache_reorder(K.data_ptr(), 0 if V is None else V.data_ptr(), parent.data_ptr(),
                                           rows // k, int(k), H, T, tp, D, _DTYPES[K.dtype], _stream_ptr(dev)))


class PostProcessor:
    """Asynchronous post-processing of finished hypotheses (Section 4.3).

    A host thread of the library turns the token ids of a finished batch
    into text -- byte-level detokenisation, one line per row up to its
    end-of-sequence id -- and writes it to ``path`` (or keeps it in memory),
    while the GPU goes on with the next batch.  ``vocab`` holds the token
    strings over the byte alphabet (see include/fastseq_hip.h).  The handle
    owns ``slots`` pinned staging buffers of ``max_rows`` x ``max_len`` ids.
    """

    def __init__(self, vocab: list, eos: int, max_rows: int, max_len: int, slots: int = 2,
                 path: str | None = None):
        import ctypes
        import numpy as np
        enc = [s.encode("utf-8") for s in vocab]
        off = np.zeros(len(enc) + 1, np.int64)
        off[1:] = np.cumsum([len(e) for e in enc])
        data = b"".join(enc) or b"\0"
        self._lib = _N.lib()
        self._h = ctypes.c_void_p()
        _N.check_lib(self._lib.fs_postproc_create(
            ctypes.byref(self._h), data, off.ctypes.data, len(vocab), int(eos), int(max_rows), int(max_len),
            int(slots), None if path is None else str(path).encode()))

    def submit(self, tokens: torch.Tensor, t: int | None = None) -> None:
        """Hand over a finished batch: tokens [rows, ld] int32 on the GPU
        (the first ``t`` columns, default all), after the work already on
        torch's current stream.  Returns at once unless every staging
        buffer is still being written."""
        if not isinstance(tokens, torch.Tensor) or tokens.device.type != "cuda" or tokens.dtype != torch.int32:
            raise ValueError("tokens must be an int32 GPU tensor")
        if tokens.dim() != 2 or (tokens.shape[1] > 1 and tokens.stride(1) != 1):
            raise ValueError("tokens must be [rows, ld] with unit column stride")
        rows, cols = tokens.shape
        t = cols if t is None else int(t)
        ld = tokens.stride(0) if rows > 1 else cols
        with _on(tokens.device):
            _N.check_lib(self._lib.fs_postproc_submit(self._h, tokens.data_ptr(), ld, rows, t,
                                                      _stream_ptr(tokens.device)))

    def flush(self) -> None:
        """Wait until every submitted batch is written."""
        _N.check_lib(self._lib.fs_postproc_flush(self._h))

    def output(self) -> bytes:
        """The text kept in memory (after a flush)."""
        import ctypes
        n = self._lib.fs_postproc_output(self._h, None, 0)
        buf = ctypes.create_string_buffer(max(1, n))
        self._lib.fs_postproc_output(self._h, buf, n)
        return buf.raw[:n]

    def busy_seconds(self) -> float:
        """Host time the worker has spent detokenising and writing."""
        return float(self._lib.fs_postproc_busy_seconds(self._h))

    def close(self) -> None:
        if self._h:
            self._lib.fs_postproc_destroy(self._h)
            self._h = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:  # noqa: BLE001 - interpreter shutdown
            pass
