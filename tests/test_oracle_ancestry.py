"""Pins of the oracle's ancestry table: the per-beam cache maintenance of
Section 2.2 (and Section 4.1.1's per-beam part) done without moving rows.

The table is pinned against the physical reorder itself: a simulated decode
keeps one cache that is reordered after every selection step
(oracle.cache_reorder, pinned separately) and one that is never moved but
read through the table; every step, both give every hypothesis the same rows,
bit for bit.  Further pins: a worked example, an identity table, and the
split-cache attention read through the table equal to the attention on the
reordered cache.
"""
import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle


def test_worked_example():
    # k = 3, one source; every hypothesis starts from its own first token
    anc = np.zeros((3, 4), np.int32)
    anc = oracle.ancestry_step(anc, np.array([0, 1, 2], np.int32), 3, 0)
    assert anc[:, 0].tolist() == [0, 1, 2]
    # step 1: new beams continue 2, 2, 0
    anc = oracle.ancestry_step(anc, np.array([2, 2, 0], np.int32), 3, 1)
    assert anc[:, :2].tolist() == [[2, 0], [2, 1], [0, 2]]
    # step 2: new beams continue 1, 0, 0 (out-of-range parent keeps its own)
    anc = oracle.ancestry_step(anc, np.array([1, 0, 7], np.int32), 3, 2)
    assert anc[:, :3].tolist() == [[2, 1, 0], [2, 0, 1], [0, 2, 2]]
    assert anc[:, 3].tolist() == [0, 0, 0]   # not yet written


def simulate(B, k, H, T, D, steps, seed, value_seed=None):
    """Physical reorder against the table, step by step (parents from `seed`,
    the new tokens' values from `value_seed`, default the same stream)."""
    rng = np.random.default_rng(seed)
    vrng = rng if value_seed is None else np.random.default_rng(value_seed)
    phys = np.zeros((B * k, H, T, D), np.float32)
    ind = np.zeros_like(phys)
    anc = np.full((B * k, T), -1, np.int32)
    for t in range(steps):
        parent = rng.integers(0, k, size=B * k).astype(np.int32)
        if t > 0 and rng.random() < 0.2:
            parent[rng.integers(0, B * k)] = -3            # an out-of-range parent now and then
        phys = oracle.cache_reorder(phys, parent, k, t)
        anc = oracle.ancestry_step(anc, parent, k, t)
        new = vrng.standard_normal((B * k, H, D)).astype(np.float32)
        phys[:, :, t] = new                                 # the step's token, in each row's own slot
        ind[:, :, t] = new
        yield t + 1, phys, ind, anc


@settings(max_examples=40, deadline=None)
@given(st.integers(1, 3), st.integers(1, 5), st.integers(1, 3), st.integers(1, 9), st.integers(0, 2**31 - 1))
def test_table_reads_what_the_reordered_cache_holds(B, k, H, T, seed):
    for t, phys, ind, anc in simulate(B, k, H, T, 2, T, seed):
        got = oracle.gather_generated(ind, anc, k, t)
        np.testing.assert_array_equal(got[:, :, :t], phys[:, :, :t])


def test_identity_table_reads_each_row_itself():
    rng = np.random.default_rng(1)
    k, T = 4, 6
    Kt = rng.standard_normal((2 * k, 3, T, 5)).astype(np.float32)
    anc = np.tile(np.arange(k, dtype=np.int32)[:, None], (2, T))
    np.testing.assert_array_equal(oracle.gather_generated(Kt, anc, k, T), Kt)


def test_attention_through_the_table_equals_attention_on_the_reordered_cache():
    B, k, H, N, T, D = 2, 4, 2, 7, 6, 16
    rng = np.random.default_rng(2)
    q = rng.standard_normal((B, k, H, D)).astype(np.float32)
    Kp = rng.standard_normal((B, H, N, D)).astype(np.float32)
    Vp = rng.standard_normal((B, H, N, D)).astype(np.float32)
    plen = np.array([5, 7], np.int32)
    sim_k = simulate(B, k, H, T, D, T, seed=3, value_seed=30)
    sim_v = simulate(B, k, H, T, D, T, seed=3, value_seed=31)   # same parents, so the same table
    for (t, pk, ik, anc), (_, pv, iv, _) in zip(sim_k, sim_v):
        want = oracle.prefix_attn(q, Kp, Vp, plen, pk, pv, t)
        got = oracle.prefix_attn_indirect(q, Kp, Vp, plen, ik, iv, anc, t)
        np.testing.assert_array_equal(got, want)


def test_invalid_arguments():
    anc = np.zeros((4, 3), np.int32)
    with pytest.raises(ValueError):
        oracle.ancestry_step(anc, np.zeros(4, np.int32), 4, 3)     # column t = 3 does not exist
    with pytest.raises(ValueError):
        oracle.ancestry_step(anc, np.zeros(4, np.int32), 3, 0)     # rows not a multiple of k
    with pytest.raises(ValueError):
        oracle.ancestry_step(anc, np.zeros(4, np.int32), 4, -1)
