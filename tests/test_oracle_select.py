"""Pins of the oracle's beam-search selection step (Section 2.1; bans from
Section 4.2, Algorithm 1).

The oracle computes, per source, the c best candidates beam_score + lp where
lp = logits - logsumexp(logits) over every token, with banned tokens at -inf,
best first and equal values in increasing flat index beam*V + token.  It is
pinned here against values worked out by hand, an independent numpy
formulation (logsumexp, a set of n-grams, a lexicographic sort) on random
tiny inputs, the n-gram oracle's own ban set, and invariants of the
definition.
"""
import math

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle


def numpy_select(logits, beam_scores, tokens, t, n, k, c):
    """Independent formulation: every candidate scored in fp64, banned ones
    from the set of the row's n-grams, then one lexicographic sort."""
    lg = np.asarray(logits, np.float64)
    rows, V = lg.shape
    B = rows // k
    lse = np.full(rows, -np.inf)
    for r in range(rows):
        if np.isfinite(lg[r]).any():
            m = lg[r].max()
            lse[r] = m + math.log(np.exp(lg[r] - m).sum())
    with np.errstate(invalid="ignore"):
        lp = np.where(np.isfinite(lse)[:, None], lg - lse[:, None], -np.inf)
    if n > 0:
        for r in range(rows):
            x = [int(v) for v in tokens[r][:t]]
            grams = {tuple(x[j:j + n]) for j in range(len(x) - n + 1)}
            suffix = tuple(x[len(x) - n + 1:]) if n > 1 else ()
            for g in grams:
                if g[:-1] == suffix and 0 <= g[-1] < V:
                    lp[r, g[-1]] = -np.inf
    cand = (np.asarray(beam_scores, np.float64)[:, None] + lp).reshape(B, k * V)
    scores = np.empty((B, c))
    flat = np.empty((B, c), np.int64)
    for b in range(B):
        f = np.arange(k * V)
        order = np.lexsort((f, -cand[b]))[:c]   # value descending, then flat index
        scores[b], flat[b] = cand[b][order], order
    return scores, (flat // V).astype(np.int32), (flat % V).astype(np.int32)


def test_closed_form_without_bans():
    # row 0: logits (0, 0, 0) -> lse = ln 3; row 1: (1, 0, 0) -> lse = ln(e + 2)
    lg = np.array([[0, 0, 0], [1, 0, 0]], np.float32)
    bs = np.array([-1.0, -0.5], np.float32)
    s, i, v = oracle.beam_select(lg, bs, None, 0, 0, k=2, c=4)
    l1 = math.log(math.e + 2)
    want = [(-0.5 + 1 - l1, 1, 0), (-0.5 - l1, 1, 1), (-0.5 - l1, 1, 2), (-1 - math.log(3), 0, 0)]
    assert [(int(a), int(b)) for a, b in zip(i[0], v[0])] == [(w[1], w[2]) for w in want]
    np.testing.assert_allclose(s[0], [w[0] for w in want], rtol=0, atol=1e-14)


def test_closed_form_with_bans_keeps_the_normaliser():
    # n = 2 bans the token after every earlier copy of the last token:
    # row 0 (2, 2, 2) bans 2; row 1 (1, 0, 1) bans 0.  The normalisers stay
    # ln 3 and ln(e + 2): the ban does not renormalise.
    lg = np.array([[0, 0, 0], [1, 0, 0]], np.float32)
    bs = np.array([-1.0, -0.5], np.float32)
    tok = np.array([[2, 2, 2], [1, 0, 1]], np.int32)
    s, i, v = oracle.beam_select(lg, bs, tok, 3, 2, k=2, c=6)
    l1 = math.log(math.e + 2)
    assert list(zip(i[0].tolist(), v[0].tolist())) == [(1, 1), (1, 2), (0, 0), (0, 1), (0, 2), (1, 0)]
    np.testing.assert_allclose(s[0][:4], [-0.5 - l1, -0.5 - l1, -1 - math.log(3), -1 - math.log(3)],
                               rtol=0, atol=1e-14)
    assert np.all(np.isneginf(s[0][4:]))   # the banned candidates come last, by flat index


def test_ties_go_to_the_smaller_flat_index():
    lg = np.zeros((6, 5), np.float32)
    s, i, v = oracle.beam_select(lg, np.zeros(6, np.float32), None, 0, 0, k=3, c=15)
    assert (i * 5 + v).tolist() == [list(range(15)), list(range(15))]
    assert np.all(s == -math.log(5))


@settings(max_examples=150, deadline=None)
@given(st.data())
def test_agrees_with_an_independent_formulation(data):
    k = data.draw(st.integers(1, 3))
    B = data.draw(st.integers(1, 3))
    V = data.draw(st.integers(1, 7))
    c = data.draw(st.integers(1, k * V))
    n = data.draw(st.integers(0, 4))
    t = data.draw(st.integers(0, 9))
    seed = data.draw(st.integers(0, 2**31 - 1))
    rng = np.random.default_rng(seed)
    lg = rng.standard_normal((B * k, V)).astype(np.float32)
    # exact ties inside rows, and a few -inf logits
    lg[rng.random(lg.shape) < 0.2] = lg.flat[0]
    lg[rng.random(lg.shape) < 0.1] = -np.inf
    bs = (rng.standard_normal(B * k) * 3).astype(np.float32)
    tok = rng.integers(-1, V + 1, size=(B * k, max(t, 1))).astype(np.int32)
    got = oracle.beam_select(lg, bs, tok, t, n, k, c)
    want = numpy_select(lg, bs, tok, t, n, k, c)
    np.testing.assert_array_equal(got[1], want[1])
    np.testing.assert_array_equal(got[2], want[2])
    fin = np.isfinite(want[0])
    np.testing.assert_array_equal(np.isfinite(got[0]), fin)
    np.testing.assert_allclose(got[0][fin], want[0][fin], rtol=0, atol=1e-12)


def test_banned_set_is_the_ngram_oracles():
    rng = np.random.default_rng(3)
    k, V, t, n = 4, 6, 24, 3
    lg = rng.standard_normal((2 * k, V)).astype(np.float32)
    tok = rng.integers(0, 3, size=(2 * k, t)).astype(np.int32)
    s, i, v = oracle.beam_select(lg, np.zeros(2 * k, np.float32), tok, t, n, k, k * V)
    banned = np.isneginf(oracle.ngram_block(tok, n, lg))
    assert banned.any()
    for b in range(2):
        for j in range(k * V):
            assert np.isneginf(s[b, j]) == banned[b * k + i[b, j], v[b, j]]


def test_every_candidate_in_order_when_c_is_k_times_V():
    rng = np.random.default_rng(4)
    k, V = 3, 11
    lg = rng.standard_normal((2 * k, V)).astype(np.float32)
    bs = rng.standard_normal(2 * k).astype(np.float32)
    s, i, v = oracle.beam_select(lg, bs, None, 0, 0, k, k * V)
    for b in range(2):
        assert sorted((i[b] * V + v[b]).tolist()) == list(range(k * V))
        assert np.all(np.diff(s[b]) <= 0)


def test_shift_of_a_row_leaves_the_selection():
    # log-softmax is invariant to adding a constant to a row's logits
    rng = np.random.default_rng(5)
    k, V, c = 4, 40, 8
    lg = (rng.integers(-64, 64, size=(3 * k, V)) / 8).astype(np.float32)
    bs = rng.standard_normal(3 * k).astype(np.float32)
    a = oracle.beam_select(lg, bs, None, 0, 0, k, c)
    lg2 = lg.copy()
    lg2[1] += 2.0
    lg2[6] -= 4.0
    b = oracle.beam_select(lg2, bs, None, 0, 0, k, c)
    np.testing.assert_array_equal(a[1], b[1])
    np.testing.assert_array_equal(a[2], b[2])
    np.testing.assert_allclose(a[0], b[0], rtol=0, atol=1e-12)


def test_permuting_beams_permutes_beam_indices():
    rng = np.random.default_rng(6)
    k, V, c, t, n = 5, 30, 10, 12, 2
    lg = rng.standard_normal((2 * k, V)).astype(np.float32)
    bs = rng.standard_normal(2 * k).astype(np.float32)
    tok = rng.integers(0, V, size=(2 * k, t)).astype(np.int32)
    perm = np.array([3, 0, 4, 1, 2])
    rows = np.concatenate([perm, k + perm])   # new beam j holds old beam perm[j]
    a = oracle.beam_select(lg, bs, tok, t, n, k, c)
    b = oracle.beam_select(lg[rows], bs[rows], tok[rows], t, n, k, c)
    np.testing.assert_array_equal(a[1], perm[b[1]])
    np.testing.assert_array_equal(a[2], b[2])
    np.testing.assert_array_equal(a[0], b[0])


def test_n_one_bans_every_history_token_and_all_neg_inf_rows_go_last():
    k, V = 2, 8
    lg = np.zeros((k, V), np.float32)
    lg[1] = -np.inf
    tok = np.array([[1, 3, 3, 6], [0, 0, 0, 0]], np.int32)
    s, i, v = oracle.beam_select(lg, np.zeros(k, np.float32), tok, 4, 1, k, k * V)
    picked = list(zip(i[0].tolist(), v[0].tolist()))
    assert picked[:5] == [(0, 0), (0, 2), (0, 4), (0, 5), (0, 7)]   # 1, 3, 6 banned
    np.testing.assert_allclose(s[0][:5], -math.log(8), rtol=0, atol=1e-15)
    assert picked[5:8] == [(0, 1), (0, 3), (0, 6)]                   # then -inf, by flat index
    assert picked[8:] == [(1, j) for j in range(V)]
    assert np.all(np.isneginf(s[0][5:]))


def test_invalid_arguments():
    lg = np.zeros((2, 3), np.float32)
    with pytest.raises(ValueError):
        oracle.beam_select(lg, np.zeros(2, np.float32), None, 0, 0, 2, 7)   # c > k*V
    with pytest.raises(ValueError):
        oracle.beam_select(lg, np.zeros(2, np.float32), None, 0, -1, 2, 2)
    with pytest.raises(ValueError):
        oracle.beam_select(lg, np.zeros(3, np.float32), None, 0, 0, 2, 2)
