"""Seeded synthetic inputs for the beam-search decode step.

The paper measures on CNN/DailyMail summarisation and WMT16 translation with
trained BART, T5 and ProphetNet checkpoints (Section 5).  Neither the data nor
the weights are used here: these generators stand in for them with inputs of
the same shapes and value structure -- encoder K/V of BART-large, T5-base and
ProphetNet-large geometry, source lengths drawn over the model's input range
and padded to S, and decoder prefixes whose tokens follow a Zipf law over the
model vocabulary (so repeats occur as they do in text).

This module is shared by the tests and the benchmark.  It only draws numbers
and lays them out; it contains none of the attention or n-gram arithmetic.

Seeding: ``numpy.random.SeedSequence([210604718, cfg])`` spawned into six
streams (lengths, q, K, V, tokens, logits).  Additional K/V sets used to
rotate the benchmark's working set past the 256 MB last-level cache come from
``SeedSequence([210604718, cfg, rep])`` for ``rep >= 1``; they share the
lengths and queries of set 0.
"""
from __future__ import annotations

import dataclasses

import numpy as np

SEED_BASE = 210604718


@dataclasses.dataclass(frozen=True)
class Config:
    """One decode-step workload.  q [B,k,H,D], K/V [B,H,S,D], tokens [B*k,t]."""
    name: str
    index: int
    B: int
    k: int
    H: int
    D: int
    S: int
    len_lo: int
    len_hi: int
    dtype: str          # "f32" or "bf16": element type of q, K, V and out
    sigma: float        # q, K, V ~ N(0, sigma^2)
    t: int              # generated-prefix length (columns of tokens)
    token_dist: str     # "uniform" or "zipf"
    zipf_s: float
    V: int              # vocabulary size (columns of logits)
    n: int              # no-repeat n-gram size
    fixed_lens: tuple = ()

    @property
    def rows(self) -> int:
        return self.B * self.k

    @property
    def esize(self) -> int:
        return 4 if self.dtype == "f32" else 2


CONFIGS = {
    # Tiny: hand-checkable; small vocabulary so repeats are frequent.
    "tiny": Config("tiny", 0, B=2, k=4, H=2, D=16, S=64, len_lo=64, len_hi=64,
                   dtype="f32", sigma=1.0, t=32, token_dist="uniform", zipf_s=0.0,
                   V=50, n=3, fixed_lens=(64, 40)),
    # BART-large summarisation step: beam 4, no_repeat_ngram_size 3,
    # max_len_b 140, input up to 1024 tokens (Section 3 usage, Table 2).
    "bart": Config("bart", 1, B=32, k=4, H=16, D=64, S=1024, len_lo=400, len_hi=1024,
                   dtype="bf16", sigma=1.0, t=140, token_dist="zipf", zipf_s=1.1,
                   V=50264, n=3),
    # T5-base translation step.
    "t5": Config("t5", 2, B=64, k=4, H=12, D=64, S=512, len_lo=128, len_hi=512,
                 dtype="bf16", sigma=1.0, t=200, token_dist="zipf", zipf_s=1.1,
                 V=32128, n=3),
    # ProphetNet-large with a long generated prefix (stresses the n-gram scan).
    "prophetnet": Config("prophetnet", 3, B=128, k=5, H=16, D=64, S=512, len_lo=512,
                         len_hi=512, dtype="bf16", sigma=0.5, t=512, token_dist="zipf",
                         zipf_s=1.05, V=30522, n=4),
    # Large batch made possible by de-duplication (Table 2: batch 32 -> 128);
    # the prefix length is swept over t = 1..140 using the first t columns.
    "large": Config("large", 4, B=320, k=4, H=16, D=64, S=1024, len_lo=256, len_hi=1024,
                    dtype="bf16", sigma=1.0, t=140, token_dist="zipf", zipf_s=1.1,
                    V=50264, n=3),
}


@dataclasses.dataclass(frozen=True)
class PrefixConfig:
    """Self-attention step over a split cache: a shared prefix of up to N
    tokens per sample ([B,H,N,D]) and t generated tokens per beam
    ([B*k,H,T,D], T the capacity)."""
    name: str
    index: int
    B: int
    k: int
    H: int
    D: int
    N: int
    len_lo: int
    len_hi: int
    T: int
    t: int
    dtype: str
    sigma: float

    @property
    def esize(self) -> int:
        return 4 if self.dtype == "f32" else 2


PREFIX_CONFIGS = {
    # GPT2-shaped decoder-only summarisation step (12 heads x 64): the
    # article is the shared prefix, beam 4, generated length up to 140.
    "gpt2": PrefixConfig("gpt2", 10, B=16, k=4, H=12, D=64, N=1024, len_lo=400, len_hi=1024,
                         T=140, t=64, dtype="bf16", sigma=1.0),
    "tiny_prefix": PrefixConfig("tiny_prefix", 11, B=2, k=3, H=2, D=16, N=40, len_lo=1, len_hi=40,
                                T=24, t=9, dtype="f32", sigma=1.0),
}


def prefix_inputs(cfg, rep: int = 0, pad: str = "zero") -> dict:
    """q [B,k,H,D], Kp/Vp [B,H,N,D] + prefix_len [B], Kt/Vt [B*k,H,T,D], t.

    Rows j >= prefix_len[b] of Kp/Vp and rows j >= t of Kt/Vt hold ``pad``
    ("zero" or "nan").  K/V of ``rep`` >= 1 come from their own streams.
    """
    if isinstance(cfg, str):
        cfg = PREFIX_CONFIGS[cfg]
    st = streams(cfg.index)
    lens = st[0].integers(cfg.len_lo, cfg.len_hi + 1, size=cfg.B).astype(np.int32)
    q = _normal(st[1], (cfg.B, cfg.k, cfg.H, cfg.D), cfg.sigma, cfg.dtype)
    kst, vst = (st[2], st[3]) if rep == 0 else streams(cfg.index, rep)[2:4]
    Kp = _normal(kst, (cfg.B, cfg.H, cfg.N, cfg.D), cfg.sigma, cfg.dtype)
    Vp = _normal(vst, (cfg.B, cfg.H, cfg.N, cfg.D), cfg.sigma, cfg.dtype)
    Kt = _normal(kst, (cfg.B * cfg.k, cfg.H, cfg.T, cfg.D), cfg.sigma, cfg.dtype)
    Vt = _normal(vst, (cfg.B * cfg.k, cfg.H, cfg.T, cfg.D), cfg.sigma, cfg.dtype)
    fill_padding(Kp, lens, pad)
    fill_padding(Vp, lens, pad)
    tl = np.full(cfg.B * cfg.k, cfg.t, dtype=np.int32)
    fill_padding(Kt, tl, pad)
    fill_padding(Vt, tl, pad)
    return {"q": q, "Kp": Kp, "Vp": Vp, "prefix_len": lens, "Kt": Kt, "Vt": Vt, "t": cfg.t}


def get(name_or_index) -> Config:
    if isinstance(name_or_index, Config):
        return name_or_index
    if isinstance(name_or_index, int):
        for c in CONFIGS.values():
            if c.index == name_or_index:
                return c
        raise KeyError(name_or_index)
    return CONFIGS[name_or_index]


def streams(cfg, rep: int = 0) -> list:
    """Six independent generators: lengths, q, K, V, tokens, logits.

    ``cfg`` is a config or its index."""
    index = cfg if isinstance(cfg, int) else cfg.index
    key = [SEED_BASE, index] if rep == 0 else [SEED_BASE, index, rep]
    return [np.random.default_rng(s) for s in np.random.SeedSequence(key).spawn(6)]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


BF16_NAN = np.uint16(0x7FC0)


def _normal(rng, shape, sigma, dtype):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if sigma != 1.0:
        x *= np.float32(sigma)
    return x if dtype == "f32" else f32_to_bf16_bits(x)


def source_lengths(cfg: Config) -> np.ndarray:
    if cfg.fixed_lens:
        return np.asarray(cfg.fixed_lens, dtype=np.int32)
    rng = streams(cfg)[0]
    return rng.integers(cfg.len_lo, cfg.len_hi + 1, size=cfg.B).astype(np.int32)


def fill_padding(K: np.ndarray, lens: np.ndarray, pad: str) -> None:
    """Overwrite rows j >= lens[b] of a [B,H,S,D] array with zeros or NaN."""
    fill = 0 if pad == "zero" else (BF16_NAN if K.dtype == np.uint16 else np.float32(np.nan))
    for b, L in enumerate(lens):
        K[b, :, int(L):, :] = fill


def attn_inputs(cfg, rep: int = 0, pad: str = "zero") -> dict:
    """q [B,k,H,D], K, V [B,H,S,D], src_len [B].

    fp32 configs give float32 arrays; bf16 configs give uint16 bf16 bits.
    ``pad`` is "zero" or "nan" (the value written to rows j >= src_len[b]).
    """
    cfg = get(cfg)
    st = streams(cfg)
    lens = source_lengths(cfg)
    q = _normal(st[1], (cfg.B, cfg.k, cfg.H, cfg.D), cfg.sigma, cfg.dtype)
    if rep == 0:
        kst, vst = st[2], st[3]
    else:
        rs = streams(cfg, rep)
        kst, vst = rs[2], rs[3]
    K = _normal(kst, (cfg.B, cfg.H, cfg.S, cfg.D), cfg.sigma, cfg.dtype)
    V = _normal(vst, (cfg.B, cfg.H, cfg.S, cfg.D), cfg.sigma, cfg.dtype)
    fill_padding(K, lens, pad)
    fill_padding(V, lens, pad)
    return {"q": q, "K": K, "V": V, "src_len": lens}


def zipf_tokens(rng, shape, V: int, s: float) -> np.ndarray:
    """Token ids with P(id = r-1) proportional to r^-s, r = 1..V (inverse CDF)."""
    p = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(p)
    cdf /= cdf[-1]
    u = rng.random(size=shape)
    ids = np.searchsorted(cdf, u, side="right")
    return np.minimum(ids, V - 1).astype(np.int32)


def ngram_inputs(cfg) -> dict:
    """tokens [B*k, t] int32 and logits [B*k, V] float32 ~ N(0,1)."""
    cfg = get(cfg)
    st = streams(cfg)
    shape = (cfg.rows, cfg.t)
    if cfg.token_dist == "uniform":
        tokens = st[4].integers(0, cfg.V, size=shape).astype(np.int32)
    else:
        tokens = zipf_tokens(st[4], shape, cfg.V, cfg.zipf_s)
    logits = st[5].standard_normal(size=(cfg.rows, cfg.V), dtype=np.float32)
    return {"tokens": tokens, "logits": logits, "n": cfg.n, "V": cfg.V}


def plant_repeats(tokens: np.ndarray, n: int, t: int, rng, per_row: int = 3) -> np.ndarray:
    """Copy each row's trailing n-1 tokens to ``per_row`` random earlier starts.

    Copies are placed at starts p <= t - 2n + 2 so they never touch the
    trailing n-1 tokens; each copy therefore creates a matching window.  Rows
    too short for that are left unchanged.  Returns a new array.
    """
    out = np.array(tokens, dtype=np.int32, copy=True)
    if n < 2:
        return out
    hi = t - 2 * n + 2
    if hi < 0:
        return out
    for r in range(out.shape[0]):
        suffix = out[r, t - n + 1:t].copy()
        for p in rng.integers(0, hi + 1, size=per_row):
            out[r, p:p + n - 1] = suffix
    return out


def low_entropy_rows(rows: int, t: int, rng) -> np.ndarray:
    """Rows that repeat heavily: constant, periodic, and uniform over 2-3 ids."""
    out = np.empty((rows, t), dtype=np.int32)
    for r in range(rows):
        kind = r % 4
        if kind == 0:
            out[r] = r % 7
        elif kind == 1:
            period = 2 + (r // 4) % 4
            out[r] = (np.arange(t) % period).astype(np.int32)
        else:
            out[r] = rng.integers(0, 2 + (kind - 2), size=t)
    return out


def select_inputs(cfg, planted: int = 1) -> dict:
    """Inputs of one beam-selection step on a decode-step config.

    logits and tokens are those of :func:`ngram_inputs`; every row also gets
    ``planted`` copies of its trailing n-1 tokens (so that bans occur on the
    Zipf data, which rarely repeats an n-gram by itself).  beam_scores are the
    running log-probabilities of the k hypotheses of each source: per source,
    k draws of -|N(0, 1)| * 2 - 10 sorted best first, from the seed stream
    SeedSequence([210604718, cfg, 1000]) (apart from the K/V rotation sets,
    which use small third keys).  c = 2k candidates are kept.
    """
    cfg = get(cfg)
    d = ngram_inputs(cfg)
    rng = np.random.default_rng(np.random.SeedSequence([SEED_BASE, cfg.index, 1000]))
    tokens = plant_repeats(d["tokens"], cfg.n, cfg.t, rng, per_row=planted) if planted else d["tokens"]
    bs = -np.abs(rng.standard_normal(size=(cfg.B, cfg.k))) * 2.0 - 10.0
    bs = -np.sort(-bs, axis=1)
    return {"logits": d["logits"], "tokens": tokens, "beam_scores": bs.astype(np.float32).reshape(-1),
            "n": cfg.n, "t": cfg.t, "k": cfg.k, "c": 2 * cfg.k, "B": cfg.B, "V": cfg.V}


def reorder_inputs(cfg) -> dict:
    """Parents of one per-beam cache reorder on a decode-step config.

    The new hypothesis j of source b continues old beam parent[b*k + j]:
    floor(k * u^2) with u ~ U[0, 1), which favours the best beams as beam
    search does, from SeedSequence([210604718, cfg, 2000]).  The cache is one
    decoder layer's self-attention K and V, [B*k, H, T, D] with T = t = the
    config's history length (the last step of generation); its contents do
    not matter to a byte copy.
    """
    cfg = get(cfg)
    rng = np.random.default_rng(np.random.SeedSequence([SEED_BASE, cfg.index, 2000]))
    parent = np.floor(cfg.k * rng.random(cfg.B * cfg.k) ** 2).astype(np.int32)
    return {"parent": parent, "B": cfg.B, "k": cfg.k, "H": cfg.H, "T": cfg.t, "t": cfg.t, "D": cfg.D,
            "dtype": cfg.dtype}


def ancestry_inputs(cfg) -> dict:
    """An ancestry table and parents for the split-cache workload.

    anc [B*k, T] int32: for each hypothesis and generated position tau < t,
    the beam (within its source) whose row holds that token, floor(k * u^2)
    with u ~ U[0, 1) (favouring the best beams, every position drawn on its
    own: few rows come from the hypothesis' own block); positions tau >= t
    hold the hypothesis' own index.  parent [B*k]: the same law, for a
    reorder of the same cache.  Streams SeedSequence([210604718, cfg, 3000])
    and [.., 3001].
    """
    if isinstance(cfg, str):
        cfg = PREFIX_CONFIGS[cfg]
    rows = cfg.B * cfg.k
    rng = np.random.default_rng(np.random.SeedSequence([SEED_BASE, cfg.index, 3000]))
    anc = np.tile((np.arange(rows) % cfg.k).astype(np.int32)[:, None], (1, cfg.T))
    anc[:, :cfg.t] = np.floor(cfg.k * rng.random((rows, cfg.t)) ** 2).astype(np.int32)
    prng = np.random.default_rng(np.random.SeedSequence([SEED_BASE, cfg.index, 3001]))
    parent = np.floor(cfg.k * prng.random(rows) ** 2).astype(np.int32)
    return {"anc": anc, "parent": parent}


# ---- post-processing workload (Section 4.3) ---------------------------------
#
# A synthetic byte-level vocabulary in the form byte-level BPE vocabularies
# take: every byte is written as one symbol (a printable byte as itself, the
# others -- in increasing order -- as the code points 0x100, 0x101, ...), and
# a token is the symbol string of a few bytes of text-like content.  The last
# id is the end-of-sequence token.

def _byte_symbol(b: int) -> str:
    printable = 0x21 <= b <= 0x7E or 0xA1 <= b <= 0xAC or 0xAE <= b <= 0xFF
    if printable:
        return chr(b)
    others = [x for x in range(256) if not (0x21 <= x <= 0x7E or 0xA1 <= x <= 0xAC or 0xAE <= x <= 0xFF)]
    return chr(0x100 + others.index(b))


_SYMBOLS = [_byte_symbol(b) for b in range(256)]


def byte_vocab(V: int, seed: int = 0) -> list:
    """V token strings over the byte alphabet; id V-1 is '</s>'."""
    rng = np.random.default_rng(np.random.SeedSequence([SEED_BASE, 4300, seed]))
    letters = np.frombuffer(b"etaoinshrdlucmfwypvbgkjqxz", np.uint8)
    punct = np.frombuffer(b".,;:'\"!?-()0123456789", np.uint8)
    vocab = []
    for _ in range(V - 1):
        n = int(min(12, 1 + rng.poisson(3)))
        kind = rng.random(n)
        raw = np.where(kind < 0.72, letters[rng.integers(0, len(letters), n)],
                       np.where(kind < 0.87, 0x20,
                                np.where(kind < 0.96, punct[rng.integers(0, len(punct), n)],
                                         rng.integers(0x80, 0x100, n))))
        vocab.append("".join(_SYMBOLS[int(b)] for b in raw))
    vocab.append("</s>")
    return vocab


def vocab_utf8(vocab: list):
    """The vocabulary as one UTF-8 byte string and int64 offsets [V+1]."""
    enc = [s.encode("utf-8") for s in vocab]
    off = np.zeros(len(enc) + 1, np.int64)
    off[1:] = np.cumsum([len(e) for e in enc])
    return b"".join(enc), off


def finished_batches(cfg, batches: int, seed: int = 0) -> np.ndarray:
    """Token ids of `batches` batches of finished hypotheses [batches, rows, t]
    (Zipf ids over the vocabulary, each row ended by the end-of-sequence id
    V-1 at a uniform position in its second half)."""
    rng = np.random.default_rng(np.random.SeedSequence([SEED_BASE, 4301, cfg.index, seed]))
    tok = zipf_tokens(rng, (batches, cfg.rows, cfg.t), cfg.V - 1, cfg.zipf_s if cfg.token_dist == "zipf" else 1.1)
    ends = rng.integers(cfg.t // 2, cfg.t + 1, size=(batches, cfg.rows))
    for bi in range(batches):
        for r in range(cfg.rows):
            if ends[bi, r] < cfg.t:
                tok[bi, r, ends[bi, r]] = cfg.V - 1
    return np.ascontiguousarray(tok.astype(np.int32))
