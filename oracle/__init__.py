"""CPU oracle for the beam-search decode step (FastSeq, arXiv 2106.04718).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the GPU library in ``paper_2106_04718_amd`` and never imports it.

The arithmetic lives in ``oracle.c`` (plain C, fp64 for the attention); this
module only marshals numpy arrays into it:

* :func:`cross_attn` -- masked softmax(q K^T / sqrt(D)) V with one K/V copy
  per source shared by its k beams (Appendix B, Eq. 4).
* :func:`cross_attn_replicated` -- the same over K/V replicated per beam,
  [B*k,H,S,D] (the layout of Eq. 1 that Eq. 4 replaces).
* :func:`prefix_attn` -- self-attention over a shared prefix cache plus a
  per-beam generated-token cache, one softmax over both (Appendix A, Eq. 3).
* :func:`ngram_block` -- no-repeat-n-gram blocking as its definition
  (Section 4.2, Algorithm 1): ban v iff (last n-1 tokens, v) already occurred.
* :func:`ngram_banned` -- the same bans as a sorted (row, token) list.
* :func:`beam_select` -- one beam-search selection step (Section 2.1): the c
  best (running score + log-probability) candidates of each source, with the
  n-gram bans applied to the log-probabilities.
* :func:`cache_reorder` -- the per-beam cache reorder after a selection step
  (Section 2.2 cache maintenance, Section 4.1.1): each new hypothesis takes
  its parent's generated-token cache.
* :func:`detokenize` -- the post-processing of finished hypotheses
  (Section 4.3): byte-level detokenisation of each row up to its
  end-of-sequence id, one line per row.
* :func:`ancestry_step` and :func:`prefix_attn_indirect` -- the same
  maintenance without moving rows: a table of which beam's row holds each
  generated token, and the split-cache attention read through it.

bf16 inputs are passed as their uint16 bit patterns and widened exactly to
fp64 here (a bf16 value is the upper half of an fp32 value), so the oracle
sees exactly the numbers the GPU reads.
"""
import ctypes
import pathlib

import numpy as np

_HERE = pathlib.Path(__file__).resolve().parent
_LIB = None

_dp = ctypes.POINTER(ctypes.c_double)
_fp = ctypes.POINTER(ctypes.c_float)
_ip = ctypes.POINTER(ctypes.c_int32)


def _lib():
    global _LIB
    if _LIB is None:
        path = _HERE / "liboracle.so"
        if not path.exists():
            from . import build as _build
            _build.build()
        lib = ctypes.CDLL(str(path))
        lib.oracle_cross_attn.argtypes = [_dp, _dp, _dp, _ip, _dp] + [ctypes.c_int] * 5
        lib.oracle_cross_attn.restype = ctypes.c_int
        lib.oracle_cross_attn_replicated.argtypes = [_dp, _dp, _dp, _ip, _dp] + [ctypes.c_int] * 5
        lib.oracle_cross_attn_replicated.restype = ctypes.c_int
        lib.oracle_ngram_banned.argtypes = [_ip] + [ctypes.c_int] * 5 + [_ip, ctypes.c_long]
        lib.oracle_ngram_banned.restype = ctypes.c_long
        lib.oracle_prefix_attn.argtypes = [_dp, _dp, _dp, _ip, _dp, _dp, ctypes.c_int, _dp] + [ctypes.c_int] * 6
        lib.oracle_prefix_attn.restype = ctypes.c_int
        lib.oracle_ngram_block.argtypes = [_ip, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                           ctypes.c_int, _fp, ctypes.c_int]
        lib.oracle_ngram_block.restype = ctypes.c_int
        lib.oracle_beam_select.argtypes = [_fp, _fp, _ip] + [ctypes.c_int] * 7 + [_dp, _ip, _ip]
        lib.oracle_beam_select.restype = ctypes.c_int
        lib.oracle_cache_reorder.argtypes = [ctypes.c_void_p, _ip] + [ctypes.c_int] * 7
        lib.oracle_cache_reorder.restype = ctypes.c_int
        lib.oracle_ancestry_step.argtypes = [_ip, ctypes.c_int, _ip] + [ctypes.c_int] * 3
        lib.oracle_ancestry_step.restype = ctypes.c_int
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = ctypes.c_int
        lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
        lib.oracle_set_num_threads.restype = None
        _LIB = lib
    return _LIB


def widen(x: np.ndarray) -> np.ndarray:
    """Exact fp64 copy of an fp32/fp64 array or of bf16 bits stored as uint16."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if x.dtype in (np.float32, np.float64):
        return x.astype(np.float64)
    raise TypeError(f"unsupported input dtype {x.dtype}")


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_lib().oracle_num_threads())


def set_num_threads(n: int) -> None:
    _lib().oracle_set_num_threads(int(n))


def cross_attn(q, K, V, src_len) -> np.ndarray:
    """fp64 encoder-decoder attention over de-duplicated K/V (Eq. 4).

    q [B,k,H,D]; K, V [B,H,S,D] (fp32, fp64, or bf16 bits as uint16);
    src_len [B] int32 (clamped to [0, S]).  Returns out [B,k,H,D] fp64.
    """
    qd = np.ascontiguousarray(widen(q))
    Kd = np.ascontiguousarray(widen(K))
    Vd = np.ascontiguousarray(widen(V))
    return cross_attn_f64(qd, Kd, Vd, src_len)


def cross_attn_f64(q, K, V, src_len) -> np.ndarray:
    """As :func:`cross_attn` but takes contiguous fp64 arrays as they are."""
    if q.ndim != 4 or K.ndim != 4 or V.shape != K.shape:
        raise ValueError("q must be [B,k,H,D] and K, V [B,H,S,D]")
    B, k, H, D = q.shape
    if K.shape[0] != B or K.shape[1] != H or K.shape[3] != D:
        raise ValueError(f"shape mismatch q{q.shape} K{K.shape}")
    S = K.shape[2]
    for a in (q, K, V):
        if a.dtype != np.float64 or not a.flags.c_contiguous:
            raise ValueError("cross_attn_f64 takes contiguous fp64 arrays")
    lens = np.ascontiguousarray(np.asarray(src_len, dtype=np.int32))
    if lens.shape != (B,):
        raise ValueError("src_len must be [B]")
    out = np.empty((B, k, H, D), dtype=np.float64)
    rc = _lib().oracle_cross_attn(
        q.ctypes.data_as(_dp), K.ctypes.data_as(_dp), V.ctypes.data_as(_dp),
        lens.ctypes.data_as(_ip), out.ctypes.data_as(_dp), B, k, H, S, D)
    if rc != 0:
        raise ValueError("oracle_cross_attn rejected its arguments")
    return out


def cross_attn_replicated(q, K, V, src_len) -> np.ndarray:
    """fp64 attention with K/V replicated per beam (the layout of Eq. 1).

    q [B,k,H,D]; K, V [B*k,H,S,D]: hypothesis b*k + i reads K[b*k + i];
    src_len [B] (the length of each source, shared by its beams).
    """
    qd = np.ascontiguousarray(widen(q))
    Kd = np.ascontiguousarray(widen(K))
    Vd = np.ascontiguousarray(widen(V))
    if qd.ndim != 4 or Kd.ndim != 4 or Vd.shape != Kd.shape:
        raise ValueError("q must be [B,k,H,D] and K, V [B*k,H,S,D]")
    B, k, H, D = qd.shape
    if Kd.shape[0] != B * k or Kd.shape[1] != H or Kd.shape[3] != D:
        raise ValueError(f"shape mismatch q{qd.shape} K{Kd.shape}")
    lens = np.ascontiguousarray(np.asarray(src_len, dtype=np.int32))
    if lens.shape != (B,):
        raise ValueError("src_len must be [B]")
    out = np.empty((B, k, H, D), dtype=np.float64)
    rc = _lib().oracle_cross_attn_replicated(
        qd.ctypes.data_as(_dp), Kd.ctypes.data_as(_dp), Vd.ctypes.data_as(_dp),
        lens.ctypes.data_as(_ip), out.ctypes.data_as(_dp), B, k, H, Kd.shape[2], D)
    if rc != 0:
        raise ValueError("oracle_cross_attn_replicated rejected its arguments")
    return out


def prefix_attn(q, Kp, Vp, prefix_len, Kt, Vt, t: int) -> np.ndarray:
    """fp64 self-attention over a split cache (Eq. 2-3).

    q [B,k,H,D]; Kp, Vp [B,H,N,D] shared prefix; prefix_len [B] int32;
    Kt, Vt [B*k,H,T,D] per-beam generated tokens of which the first t rows
    are used.  Inputs may be fp32, fp64 or bf16 bits (uint16).  Returns
    out [B,k,H,D] fp64.
    """
    qd, Kpd, Vpd, Ktd, Vtd = (np.ascontiguousarray(widen(a)) for a in (q, Kp, Vp, Kt, Vt))
    if qd.ndim != 4 or Kpd.ndim != 4 or Vpd.shape != Kpd.shape or Ktd.ndim != 4 or Vtd.shape != Ktd.shape:
        raise ValueError("q [B,k,H,D], Kp/Vp [B,H,N,D], Kt/Vt [B*k,H,T,D]")
    B, k, H, D = qd.shape
    N, T = Kpd.shape[2], Ktd.shape[2]
    if Kpd.shape != (B, H, N, D) or Ktd.shape != (B * k, H, T, D):
        raise ValueError(f"shape mismatch q{qd.shape} Kp{Kpd.shape} Kt{Ktd.shape}")
    lens = np.ascontiguousarray(np.asarray(prefix_len, dtype=np.int32))
    if lens.shape != (B,):
        raise ValueError("prefix_len must be [B]")
    out = np.empty((B, k, H, D), dtype=np.float64)
    rc = _lib().oracle_prefix_attn(qd.ctypes.data_as(_dp), Kpd.ctypes.data_as(_dp), Vpd.ctypes.data_as(_dp),
                                   lens.ctypes.data_as(_ip), Ktd.ctypes.data_as(_dp), Vtd.ctypes.data_as(_dp),
                                   int(t), out.ctypes.data_as(_dp), B, k, H, N, T, D)
    if rc != 0:
        raise ValueError("oracle_prefix_attn rejected its arguments")
    return out


def ngram_block_inplace(tokens: np.ndarray, n: int, logits: np.ndarray, t: int) -> None:
    """As :func:`ngram_block` but writes into ``logits`` (contiguous float32)
    and takes contiguous int32 ``tokens`` as they are (no copies)."""
    if tokens.dtype != np.int32 or not tokens.flags.c_contiguous or tokens.ndim != 2:
        raise ValueError("tokens must be contiguous int32 [rows, ld]")
    if logits.dtype != np.float32 or not logits.flags.c_contiguous or logits.ndim != 2:
        raise ValueError("logits must be contiguous float32 [rows, V]")
    if tokens.shape[0] != logits.shape[0]:
        raise ValueError("tokens and logits must have the same rows")
    rc = _lib().oracle_ngram_block(tokens.ctypes.data_as(_ip), tokens.shape[1], tokens.shape[0],
                                   int(t), int(n), logits.ctypes.data_as(_fp), logits.shape[1])
    if rc != 0:
        raise ValueError("oracle_ngram_block rejected its arguments")


def ngram_block(tokens, n: int, logits, t: int | None = None) -> np.ndarray:
    """Return a copy of ``logits`` with no-repeat-n-gram bans applied.

    tokens [rows, ld] int32 (the first ``t`` columns are the history,
    default ``t = ld``); logits [rows, V] fp32.  Banned entries become -inf;
    all others are returned bit for bit.
    """
    tok = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
    lg = np.array(logits, dtype=np.float32, copy=True, order="C")
    if tok.ndim != 2 or lg.ndim != 2 or tok.shape[0] != lg.shape[0]:
        raise ValueError("tokens must be [rows, ld] and logits [rows, V]")
    rows, ld = tok.shape
    if t is None:
        t = ld
    rc = _lib().oracle_ngram_block(tok.ctypes.data_as(_ip), ld, rows, int(t), int(n),
                                   lg.ctypes.data_as(_fp), lg.shape[1])
    if rc != 0:
        raise ValueError("oracle_ngram_block rejected its arguments")
    return lg


def ngram_banned(tokens, n: int, V: int, t: int | None = None) -> np.ndarray:
    """The no-repeat-n-gram bans as an int32 array of (row, token) pairs,
    sorted by row then token, each once (the positions that
    :func:`ngram_block` sets to -inf)."""
    tok = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
    if tok.ndim != 2:
        raise ValueError("tokens must be [rows, ld]")
    rows, ld = tok.shape
    if t is None:
        t = ld
    lib = _lib()
    cap = max(1, rows * max(0, int(t) - int(n) + 1))
    for _ in range(2):
        pairs = np.empty((cap, 2), dtype=np.int32)
        got = lib.oracle_ngram_banned(tok.ctypes.data_as(_ip), ld, rows, int(t), int(n), int(V),
                                      pairs.ctypes.data_as(_ip), cap)
        if got < 0:
            raise ValueError("oracle_ngram_banned rejected its arguments")
        if got <= cap:
            return pairs[:got].copy()
        cap = int(got)
    raise RuntimeError("oracle_ngram_banned: pair count changed between calls")


def beam_select(logits, beam_scores, tokens, t: int, n: int, k: int, c: int):
    """One beam-search selection step (see ``oracle_beam_select`` in oracle.c).

    logits [B*k, V] fp32; beam_scores [B*k] fp32; tokens [B*k, ld] int32 whose
    first ``t`` columns are the history (ignored, and may be None, when
    ``n == 0``).  Returns (scores fp64 [B, c], beam int32 [B, c], token int32
    [B, c]) for every source, best first, equal values in increasing
    flat index beam*V + token.
    """
    lg = np.ascontiguousarray(np.asarray(logits, dtype=np.float32))
    bs = np.ascontiguousarray(np.asarray(beam_scores, dtype=np.float32))
    if lg.ndim != 2 or bs.shape != (lg.shape[0],) or k < 1 or lg.shape[0] % k:
        raise ValueError("logits must be [B*k, V] and beam_scores [B*k]")
    rows, V = lg.shape
    B = rows // k
    if n > 0:
        tok = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
        if tok.ndim != 2 or tok.shape[0] != rows:
            raise ValueError("tokens must be [B*k, ld]")
        ld = tok.shape[1]
    else:
        tok = np.zeros((rows, 1), dtype=np.int32)
        ld, t = 1, 0
    scores = np.empty((B, c), dtype=np.float64)
    beam = np.empty((B, c), dtype=np.int32)
    token = np.empty((B, c), dtype=np.int32)
    rc = _lib().oracle_beam_select(lg.ctypes.data_as(_fp), bs.ctypes.data_as(_fp), tok.ctypes.data_as(_ip),
                                   ld, int(t), int(n), B, int(k), V, int(c), scores.ctypes.data_as(_dp),
                                   beam.ctypes.data_as(_ip), token.ctypes.data_as(_ip))
    if rc != 0:
        raise ValueError("oracle_beam_select rejected its arguments")
    return scores, beam, token


def cache_reorder(cache, parent, k: int, t: int) -> np.ndarray:
    """Per-beam cache reorder (see ``oracle_cache_reorder`` in oracle.c).

    cache [B*k, H, T, D] of any fixed-size dtype (bf16 as uint16 bits);
    parent [B*k] int32, the old beam each new hypothesis continues.  Returns
    the reordered copy: rows tau < t of hypothesis b*k + j become those of
    b*k + parent[b*k + j]; other rows, and rows with a parent outside
    [0, k), keep their bytes.
    """
    x = np.array(cache, copy=True, order="C")
    par = np.ascontiguousarray(np.asarray(parent, dtype=np.int32))
    if x.ndim != 4 or k < 1 or x.shape[0] % k or par.shape != (x.shape[0],):
        raise ValueError("cache must be [B*k, H, T, D] and parent [B*k]")
    rows, H, T, D = x.shape
    rc = _lib().oracle_cache_reorder(x.ctypes.data_as(ctypes.c_void_p), par.ctypes.data_as(_ip), rows // k, int(k),
                                     H, T, int(t), D, x.dtype.itemsize)
    if rc != 0:
        raise ValueError("oracle_cache_reorder rejected its arguments")
    return x


def ancestry_step(anc, parent, k: int, t: int) -> np.ndarray:
    """One step of the ancestry table (see ``oracle_ancestry_step``).

    anc [B*k, ld] int32 with ld > t; parent [B*k] int32.  Returns the updated
    copy: columns tau < t of hypothesis b*k + j become those of
    b*k + parent[b*k + j], column t becomes j, later columns are kept.
    """
    a = np.array(anc, dtype=np.int32, copy=True, order="C")
    par = np.ascontiguousarray(np.asarray(parent, dtype=np.int32))
    if a.ndim != 2 or k < 1 or a.shape[0] % k or par.shape != (a.shape[0],):
        raise ValueError("anc must be [B*k, ld] and parent [B*k]")
    rc = _lib().oracle_ancestry_step(a.ctypes.data_as(_ip), a.shape[1], par.ctypes.data_as(_ip),
                                     a.shape[0] // k, int(k), int(t))
    if rc != 0:
        raise ValueError("oracle_ancestry_step rejected its arguments")
    return a


def gather_generated(Kt, anc, k: int, t: int) -> np.ndarray:
    """The generated-token cache as hypothesis r sees it through the table:
    out[r, h, tau] = Kt[b*k + anc[r, tau], h, tau] for tau < t (entries
    outside [0, k) read r's own row); positions tau >= t are copied as they
    are."""
    Kt = np.asarray(Kt)
    anc = np.asarray(anc)
    rows = Kt.shape[0]
    out = Kt.copy()
    own = np.arange(rows) % k
    for tau in range(t):
        a = anc[:, tau]
        a = np.where((a >= 0) & (a < k), a, own)
        out[:, :, tau] = Kt[(np.arange(rows) // k) * k + a, :, tau]
    return out


def prefix_attn_indirect(q, Kp, Vp, prefix_len, Kt, Vt, anc, t: int) -> np.ndarray:
    """Split-cache self-attention whose generated rows are read through the
    ancestry table (definition: gather the rows, then :func:`prefix_attn`)."""
    k = np.asarray(q).shape[1]
    return prefix_attn(q, Kp, Vp, prefix_len, gather_generated(Kt, anc, k, t), gather_generated(Vt, anc, k, t), t)


def _symbol_bytes() -> dict:
    """Code point -> byte of the byte-level alphabet: a printable byte
    (0x21-0x7E, 0xA1-0xAC, 0xAE-0xFF) is its own symbol, the remaining
    bytes in increasing order are the code points 0x100, 0x101, ..."""
    table, nxt = {}, 0x100
    for b in range(256):
        if 0x21 <= b <= 0x7E or 0xA1 <= b <= 0xAC or 0xAE <= b <= 0xFF:
            table[b] = b
        else:
            table[nxt] = b
            nxt += 1
    return table


def detokenize(tokens, vocab: list, eos: int) -> bytes:
    """Post-processing of finished hypotheses (Section 4.3), synchronously:
    each row of ``tokens`` [rows, t] becomes one line -- the bytes of its
    tokens up to its first ``eos`` id, then a newline.  A token is the
    symbol string ``vocab[id]``; each symbol of the byte alphabet gives back
    its byte, other characters give nothing, and ids outside the vocabulary
    are skipped."""
    table = _symbol_bytes()
    out = bytearray()
    for row in np.asarray(tokens):
        for v in row:
            v = int(v)
            if v == eos:
                break
            if 0 <= v < len(vocab):
                for ch in vocab[v]:
                    b = table.get(ord(ch))
                    if b is not None:
                        out.append(b)
        out.append(0x0A)
    return bytes(out)
