"""Pins for the oracle's no-repeat-n-gram blocking (Section 4.2, Algorithm 1).

The oracle is checked against things other than itself: a hand-derived table
of banned sets, brute force over every candidate token, an n-gram-set
formulation, and invariants of the definition.
"""
import pathlib

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from paper_2106_04718_amd import workloads

GOLDEN = pathlib.Path(__file__).parent / "golden" / "ngram_hand.txt"


def load_hand_cases():
    cases = []
    for line in GOLDEN.read_text().splitlines():
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        V, n, toks, banned, note = [f.strip() for f in line.split("|")]
        tokens = [int(x) for x in toks.split()]
        ban = set() if banned == "-" else {int(x) for x in banned.split()}
        cases.append((int(V), int(n), tokens, ban, note))
    return cases


HAND = load_hand_cases()


def banned_of(logits_before, logits_after):
    """Set of columns turned into -inf; also asserts nothing else changed."""
    a = logits_before.view(np.uint32)
    b = logits_after.view(np.uint32)
    changed = np.nonzero(a != b)[0]
    assert np.all(np.isneginf(logits_after[changed]))
    return {int(c) for c in changed}


@pytest.mark.parametrize("V,n,tokens,banned,note", HAND, ids=[c[4][:40] for c in HAND])
def test_hand_table(V, n, tokens, banned, note):
    tok = np.array([tokens], dtype=np.int32).reshape(1, len(tokens))
    lg = np.arange(V, dtype=np.float32).reshape(1, V) + 0.5
    out = oracle.ngram_block(tok, n, lg)
    assert banned_of(lg[0], out[0]) == banned, note


def test_hand_table_is_not_trivial():
    # the table exercises bans, non-bans, n=1, t<n, n=t and out-of-range ids
    assert len(HAND) >= 15
    assert any(not b for *_, b, _ in HAND) and any(len(b) > 1 for *_, b, _ in HAND)


def brute_force_banned(row, n, V):
    """Candidate by candidate: v is banned iff (suffix, v) is an n-gram of the row."""
    t = len(row)
    if t < n:
        return set()
    suffix = list(row[t - n + 1:]) if n > 1 else []
    grams = {tuple(row[j:j + n]) for j in range(0, t - n + 1)}
    return {v for v in range(V) if tuple(suffix + [v]) in grams}


def set_formulation_banned(row, n, V):
    """Map every (n-1)-prefix to the tokens that followed it, then look up the suffix."""
    t = len(row)
    if t < n:
        return set()
    follow = {}
    for j in range(0, t - n + 1):
        follow.setdefault(tuple(row[j:j + n - 1]), set()).add(row[j + n - 1])
    nxt = follow.get(tuple(row[t - n + 1:]), set())
    return {v for v in nxt if 0 <= v < V}


@settings(max_examples=300, deadline=None)
@given(
    V=st.sampled_from([2, 3, 5]),
    n=st.integers(1, 5),
    rows=st.lists(st.lists(st.integers(0, 4), min_size=0, max_size=24), min_size=1, max_size=6),
)
def test_against_brute_force_and_sets(V, n, rows):
    t = min(len(r) for r in rows)
    tok = np.array([r[:t] for r in rows], dtype=np.int32).reshape(len(rows), t)
    lg = np.random.default_rng(0).standard_normal((len(rows), V)).astype(np.float32)
    out = oracle.ngram_block(tok, n, lg)
    for r in range(len(rows)):
        got = banned_of(lg[r], out[r])
        row = [int(x) for x in tok[r]]
        assert got == brute_force_banned(row, n, V)
        assert got == set_formulation_banned(row, n, V)


def test_leading_dimension_uses_first_t_columns():
    rng = np.random.default_rng(1)
    tok = rng.integers(0, 3, size=(16, 40)).astype(np.int32)
    lg = rng.standard_normal((16, 3)).astype(np.float32)
    for t in (0, 1, 2, 3, 17, 39, 40):
        a = oracle.ngram_block(tok, 3, lg, t=t)
        b = oracle.ngram_block(np.ascontiguousarray(tok[:, :t]), 3, lg)
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_invariants_on_zipf_rows_with_planted_repeats():
    cfg = workloads.get("bart")
    rng = np.random.default_rng(7)
    tok = workloads.zipf_tokens(rng, (64, 140), cfg.V, cfg.zipf_s)
    tok = workloads.plant_repeats(tok, 3, 140, rng, per_row=2)
    lg = rng.standard_normal((64, cfg.V)).astype(np.float32)
    out = oracle.ngram_block(tok, 3, lg)
    nbanned = 0
    for r in range(64):
        ban = banned_of(lg[r], out[r])
        assert ban <= set(int(x) for x in tok[r])          # banned tokens occurred
        assert len(ban) <= 140 - 3 + 1                      # at most one per window
        assert ban == set_formulation_banned([int(x) for x in tok[r]], 3, cfg.V)
        nbanned += len(ban)
    assert nbanned >= 64                                   # planted copies ban something
    # applying twice changes nothing more (idempotent)
    again = oracle.ngram_block(tok, 3, out)
    assert np.array_equal(again.view(np.uint32), out.view(np.uint32))
    # rows are independent: permuting rows permutes the result
    perm = rng.permutation(64)
    outp = oracle.ngram_block(tok[perm], 3, lg[perm])
    assert np.array_equal(outp.view(np.uint32), out[perm].view(np.uint32))


def test_n1_bans_every_token_of_the_row():
    rng = np.random.default_rng(3)
    tok = rng.integers(0, 30, size=(8, 12)).astype(np.int32)
    lg = np.zeros((8, 30), np.float32)
    out = oracle.ngram_block(tok, 1, lg)
    for r in range(8):
        assert banned_of(lg[r], out[r]) == set(int(x) for x in tok[r])


def test_untouched_logits_keep_their_bits_including_nan():
    tok = np.array([[1, 2, 1, 2]], np.int32)
    lg = np.array([[np.nan, 3.0, -0.0, np.inf]], np.float32)
    out = oracle.ngram_block(tok, 2, lg)   # suffix (2) at j=1 -> ban 1
    assert np.isneginf(out[0, 1])
    keep = [0, 2, 3]
    assert np.array_equal(out[0, keep].view(np.uint32), lg[0, keep].view(np.uint32))


def test_rejects_invalid_arguments():
    tok = np.zeros((2, 4), np.int32)
    lg = np.zeros((2, 5), np.float32)
    with pytest.raises(ValueError):
        oracle.ngram_block(tok, 0, lg)
    with pytest.raises(ValueError):
        oracle.ngram_block(tok, 2, lg, t=5)      # t > ld


def test_configs_rarely_ban_without_planting():
    # Zipf prefixes alone give ~0.1 matches per row for BART-like rows; this is why
    # parity tests also plant repeats.
    cfg = workloads.get("bart")
    d = workloads.ngram_inputs(cfg)
    out = oracle.ngram_block(d["tokens"], cfg.n, d["logits"])
    per_row = np.isneginf(out).sum() / cfg.rows
    assert per_row < 1.0


# ---- the bans as a list of (row, token) pairs ------------------------------

@pytest.mark.parametrize("V,n,tokens,banned,note", HAND, ids=[c[4][:40] for c in HAND])
def test_banned_pairs_hand_table(V, n, tokens, banned, note):
    tok = np.array([tokens], dtype=np.int32).reshape(1, len(tokens))
    pairs = oracle.ngram_banned(tok, n, V)
    assert [int(r) for r in pairs[:, 0]] == [0] * len(pairs), note
    assert [int(v) for v in pairs[:, 1]] == sorted(banned), note


@settings(max_examples=200, deadline=None)
@given(
    V=st.sampled_from([2, 3, 5]),
    n=st.integers(1, 5),
    rows=st.lists(st.lists(st.integers(-1, 5), min_size=0, max_size=24), min_size=1, max_size=6),
)
def test_banned_pairs_against_brute_force(V, n, rows):
    t = min(len(r) for r in rows)
    tok = np.array([r[:t] for r in rows], dtype=np.int32).reshape(len(rows), t)
    pairs = oracle.ngram_banned(tok, n, V)
    want = [(r, v) for r in range(len(rows))
            for v in sorted(brute_force_banned([int(x) for x in tok[r]], n, V))]
    assert [tuple(int(x) for x in p) for p in pairs] == want


def test_banned_pairs_are_the_blocked_positions_with_a_leading_dimension():
    rng = np.random.default_rng(11)
    tok = workloads.plant_repeats(rng.integers(0, 9, size=(40, 60)).astype(np.int32), 3, 60, rng, per_row=2)
    lg = rng.standard_normal((40, 7)).astype(np.float32)
    for t in (0, 2, 3, 10, 59, 60):
        out = oracle.ngram_block(tok, 3, lg, t=t)
        r, v = np.nonzero(np.isneginf(out))
        pairs = oracle.ngram_banned(tok, 3, 7, t=t)
        assert np.array_equal(pairs, np.stack([r, v], axis=1).astype(np.int32).reshape(-1, 2))


def test_banned_pairs_rejects_invalid_arguments():
    tok = np.zeros((2, 4), np.int32)
    with pytest.raises(ValueError):
        oracle.ngram_banned(tok, 0, 5)
    with pytest.raises(ValueError):
        oracle.ngram_banned(tok, 2, 5, t=5)
