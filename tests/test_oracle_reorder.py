"""Pins of the oracle's per-beam cache reorder (Section 2.2, cache
maintenance; Section 4.1.1: only the per-beam generated-token cache is
reordered).

After a selection step, hypothesis j of source b continues old hypothesis
parent[b*k + j] of the same source, so rows tau < t of its cache become that
parent's; rows tau >= t and rows with a parent outside [0, k) keep their
bytes.  The oracle is pinned here against a worked example, a gather written
with numpy indexing on random shapes, and laws the definition implies:
identity, composition of two steps, a shared parent, the untouched capacity
rows (NaN payloads included), and per-source independence.
"""
import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle


def test_worked_example():
    # B=1, k=3, H=1, T=2, D=1: beams hold (0, 1), (2, 3), (4, 5) over tau
    x = np.arange(6, dtype=np.float32).reshape(3, 1, 2, 1)
    got = oracle.cache_reorder(x, np.array([2, 0, 0], np.int32), k=3, t=1)
    # tau = 0 comes from beams 2, 0, 0; tau = 1 (>= t) stays
    assert got.ravel().tolist() == [4, 1, 0, 3, 0, 5]
    got = oracle.cache_reorder(x, np.array([2, 0, 0], np.int32), k=3, t=2)
    assert got.ravel().tolist() == [4, 5, 0, 1, 0, 1]


def numpy_gather(x, parent, k, t):
    rows = x.shape[0]
    own = np.arange(rows)
    src = (own // k) * k + parent
    valid = (parent >= 0) & (parent < k)
    src = np.where(valid, src, own)
    out = x.copy()
    out[:, :, :t] = x[src][:, :, :t]
    return out


@settings(max_examples=150, deadline=None)
@given(st.data())
def test_agrees_with_an_indexed_gather(data):
    k = data.draw(st.integers(1, 6))
    B = data.draw(st.integers(1, 4))
    H = data.draw(st.integers(1, 3))
    T = data.draw(st.integers(1, 6))
    t = data.draw(st.integers(0, T))
    D = data.draw(st.integers(1, 5))
    dt = data.draw(st.sampled_from([np.uint16, np.float32, np.uint8, np.float64]))
    seed = data.draw(st.integers(0, 2**31 - 1))
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 200, size=(B * k, H, T, D)).astype(dt)
    parent = rng.integers(-1, k + 1, size=B * k).astype(np.int32)
    got = oracle.cache_reorder(x, parent, k, t)
    np.testing.assert_array_equal(got.view(np.uint8), numpy_gather(x, parent, k, t).view(np.uint8))


def test_identity_and_empty_history_leave_every_bit():
    rng = np.random.default_rng(1)
    x = rng.integers(0, 2**16, size=(8, 3, 5, 4)).astype(np.uint16)
    assert np.array_equal(oracle.cache_reorder(x, np.tile(np.arange(4, dtype=np.int32), 2), 4, 5), x)
    assert np.array_equal(oracle.cache_reorder(x, np.array([3, 2, 1, 0] * 2, np.int32), 4, 0), x)


def test_two_steps_compose():
    # after p, row j holds old[p[j]]; after q, row j holds old[p[q[j]]]
    rng = np.random.default_rng(2)
    k, B = 5, 3
    x = rng.standard_normal((B * k, 2, 4, 3)).astype(np.float32)
    p = rng.integers(0, k, size=B * k).astype(np.int32)
    q = rng.integers(0, k, size=B * k).astype(np.int32)
    two = oracle.cache_reorder(oracle.cache_reorder(x, p, k, 4), q, k, 4)
    pq = np.array([p[(r // k) * k + q[r]] for r in range(B * k)], np.int32)
    np.testing.assert_array_equal(two, oracle.cache_reorder(x, pq, k, 4))


def test_one_parent_for_all_beams_copies_it_everywhere():
    rng = np.random.default_rng(3)
    k = 4
    x = rng.standard_normal((2 * k, 2, 6, 8)).astype(np.float32)
    got = oracle.cache_reorder(x, np.array([2] * k + [0] * k, np.int32), k, 6)
    for j in range(k):
        np.testing.assert_array_equal(got[j], x[2])
        np.testing.assert_array_equal(got[k + j], x[k])


def test_capacity_rows_and_nan_payloads_keep_their_bits():
    rng = np.random.default_rng(4)
    k, T, t = 3, 7, 4
    x = rng.standard_normal((2 * k, 2, T, 5)).astype(np.float32)
    bits = x.view(np.uint32)
    bits[:, :, t:] = 0x7FC00001 + np.arange(bits[:, :, t:].size, dtype=np.uint32).reshape(bits[:, :, t:].shape) % 7
    bits[0, 1, 2, 3] = 0x7F800001   # a signalling-NaN payload inside the history
    got = oracle.cache_reorder(x, np.array([1, 0, 2, 2, 2, 0], np.int32), k, t)
    np.testing.assert_array_equal(got.view(np.uint32)[:, :, t:], bits[:, :, t:])
    assert got.view(np.uint32)[1, 1, 2, 3] == 0x7F800001


def test_sources_are_independent():
    rng = np.random.default_rng(5)
    k, B = 4, 3
    x = rng.standard_normal((B * k, 2, 3, 4)).astype(np.float32)
    parent = rng.integers(0, k, size=B * k).astype(np.int32)
    whole = oracle.cache_reorder(x, parent, k, 3)
    for b in range(B):
        sl = slice(b * k, (b + 1) * k)
        np.testing.assert_array_equal(whole[sl], oracle.cache_reorder(x[sl], parent[sl], k, 3))


def test_invalid_arguments():
    x = np.zeros((4, 1, 3, 2), np.float32)
    with pytest.raises(ValueError):
        oracle.cache_reorder(x, np.zeros(4, np.int32), 4, 4)    # t > T
    with pytest.raises(ValueError):
        oracle.cache_reorder(x, np.zeros(4, np.int32), 4, -1)
    with pytest.raises(ValueError):
        oracle.cache_reorder(x, np.zeros(4, np.int32), 3, 1)    # rows not a multiple of k
    with pytest.raises(ValueError):
        oracle.cache_reorder(x, np.zeros(3, np.int32), 4, 1)
