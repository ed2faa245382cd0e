"""Pins for the oracle's encoder-decoder attention (Appendix B, Eq. 4).

The oracle is checked against closed forms worked out by hand for specific
inputs, a library routine (PyTorch's CPU scaled_dot_product_attention in
fp64 with a key mask), and invariants the definition implies: beam-replicated
K/V gives the same result (Eq. 1 vs Eq. 4), padding is never read, beams
and keys can be permuted, and a common shift of all keys cancels.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from hypothesis import given, settings, strategies as st

import oracle
from paper_2106_04718_amd import workloads


def one(qv, Krows, Vrows, L=None):
    """Single source, beam and head: q [D], K/V [S, D]."""
    q = np.asarray(qv, np.float64).reshape(1, 1, 1, -1)
    K = np.asarray(Krows, np.float64)[None, None]
    V = np.asarray(Vrows, np.float64)[None, None]
    S = K.shape[2]
    lens = np.array([S if L is None else L], np.int32)
    return oracle.cross_attn(q, K, V, lens)[0, 0, 0]


def test_closed_form_two_keys_d4():
    # D=4: scale 1/2.  scores (q.K0, q.K1)/2 = (1, 0)  ->  p0 = e/(e+1)
    out = one([2, 0, 0, 0], [[1, 0, 0, 0], [0, 0, 0, 0]], [[1, 2, 3, 4], [5, 6, 7, 8]])
    p0 = math.e / (math.e + 1.0)
    want = p0 * np.array([1, 2, 3, 4.0]) + (1 - p0) * np.array([5, 6, 7, 8.0])
    np.testing.assert_allclose(out, want, rtol=0, atol=1e-15)


def test_closed_form_scale_is_inverse_sqrt_d():
    # D=16: scale 1/4 (1/D or 2/D would give different weights).  q = 4 e0,
    # keys 2 e0, 0, -e0 -> scores 2, 0, -1.
    D = 16
    q = np.zeros(D); q[0] = 4
    K = np.zeros((3, D)); K[0, 0] = 2; K[2, 0] = -1
    V = np.zeros((3, D)); V[0, :] = 1; V[2, 3] = 1
    out = one(q, K, V)
    w = np.array([math.exp(2), 1.0, math.exp(-1)])
    w /= w.sum()
    want = w[0] * V[0] + w[1] * V[1] + w[2] * V[2]
    np.testing.assert_allclose(out, want, rtol=0, atol=1e-15)


def test_closed_form_pins_operand_order():
    # Asymmetric q and K: q.K0 = 2, q.K1 = 1 with D=4 -> scores 1, 0.5.
    out = one([1, 2, 0, 0], [[0, 1, 0, 0], [1, 0, 0, 0]], [[1, 0, 0, 0], [0, 1, 0, 0]])
    p0 = 1.0 / (1.0 + math.exp(-0.5))
    np.testing.assert_allclose(out, [p0, 1 - p0, 0, 0], rtol=0, atol=1e-15)


def test_large_scores_are_stable():
    # scores 1000 and 999.5: exp() of the raw scores would overflow fp64.
    out = one([2000, 0, 0, 0], [[1, 0, 0, 0], [0.9995, 0, 0, 0]], [[1, 0, 0, 0], [0, 1, 0, 0]])
    p0 = 1.0 / (1.0 + math.exp(-0.5))
    np.testing.assert_allclose(out, [p0, 1 - p0, 0, 0], rtol=0, atol=1e-12)


def test_single_key_returns_its_value_exactly():
    rng = np.random.default_rng(0)
    B, k, H, S, D = 3, 4, 2, 9, 16
    q = rng.standard_normal((B, k, H, D))
    K = rng.standard_normal((B, H, S, D))
    V = rng.standard_normal((B, H, S, D))
    out = oracle.cross_attn(q, K, V, np.ones(B, np.int32))
    for b in range(B):
        for i in range(k):
            for h in range(H):
                assert np.array_equal(out[b, i, h], V[b, h, 0])


def test_constant_values_and_zero_query():
    rng = np.random.default_rng(1)
    B, k, H, S, D = 2, 3, 2, 11, 8
    lens = np.array([11, 5], np.int32)
    K = rng.standard_normal((B, H, S, D))
    c = rng.standard_normal(D)
    Vc = np.broadcast_to(c, (B, H, S, D)).copy()
    out = oracle.cross_attn(rng.standard_normal((B, k, H, D)), K, Vc, lens)
    np.testing.assert_allclose(out, np.broadcast_to(c, out.shape), rtol=0, atol=1e-14)
    # q = 0: uniform weights -> mean of the valid value rows
    V = rng.standard_normal((B, H, S, D))
    out0 = oracle.cross_attn(np.zeros((B, k, H, D)), K, V, lens)
    for b in range(B):
        mean = V[b, :, :lens[b], :].mean(axis=1)            # [H, D]
        for i in range(k):
            np.testing.assert_allclose(out0[b, i], mean, rtol=0, atol=1e-14)


def sdpa_reference(q, K, V, lens):
    """PyTorch CPU SDPA in fp64, per source, with a boolean key mask."""
    B, k, H, D = q.shape
    S = K.shape[2]
    out = np.zeros((B, k, H, D))
    for b in range(B):
        L = int(min(max(lens[b], 0), S))
        if L == 0:
            continue
        qt = torch.from_numpy(np.ascontiguousarray(q[b].transpose(1, 0, 2)))  # [H, k, D]
        mask = torch.zeros(k, S, dtype=torch.bool)
        mask[:, :L] = True
        o = F.scaled_dot_product_attention(qt, torch.from_numpy(K[b]), torch.from_numpy(V[b]),
                                           attn_mask=mask)
        out[b] = o.numpy().transpose(1, 0, 2)
    return out


@settings(max_examples=60, deadline=None)
@given(B=st.integers(1, 3), k=st.integers(1, 5), H=st.integers(1, 3), S=st.integers(1, 40),
       D=st.sampled_from([1, 2, 3, 8, 16, 64]), seed=st.integers(0, 2**31 - 1))
def test_matches_library_sdpa(B, k, H, S, D, seed):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, k, H, D)) * 2
    K = rng.standard_normal((B, H, S, D))
    V = rng.standard_normal((B, H, S, D))
    lens = rng.integers(-2, S + 3, size=B).astype(np.int32)   # includes clamped values
    got = oracle.cross_attn(q, K, V, lens)
    want = sdpa_reference(q, K, V, lens)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_tiny_config_matches_library_sdpa():
    d = workloads.attn_inputs("tiny")
    got = oracle.cross_attn(d["q"], d["K"], d["V"], d["src_len"])
    want = sdpa_reference(*(oracle.widen(d[x]) for x in ("q", "K", "V")), d["src_len"])
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_bf16_inputs_are_widened_exactly():
    x = np.array([1.0, -2.5, 3.140625, 1e-3, 65504.0], np.float32)
    bits = workloads.f32_to_bf16_bits(x)
    w = oracle.widen(bits)
    # every bf16 value is an fp32 value with the low 16 bits zero
    assert np.array_equal(w.astype(np.float32).view(np.uint32) & 0xFFFF, np.zeros(5, np.uint32))
    assert w[0] == 1.0 and w[1] == -2.5 and w[2] == 3.140625


def test_dedup_equals_replicated_bitwise():
    # Eq. 4 (one K/V copy per source) vs Eq. 1 (K/V replicated per beam).
    rng = np.random.default_rng(2)
    B, k, H, S, D = 3, 4, 2, 33, 16
    q = rng.standard_normal((B, k, H, D))
    K = rng.standard_normal((B, H, S, D))
    V = rng.standard_normal((B, H, S, D))
    lens = np.array([33, 20, 1], np.int32)
    dedup = oracle.cross_attn(q, K, V, lens)
    rep = oracle.cross_attn(q.reshape(B * k, 1, H, D), np.repeat(K, k, axis=0),
                            np.repeat(V, k, axis=0), np.repeat(lens, k))
    assert np.array_equal(dedup.reshape(B * k, 1, H, D), rep)


def test_padding_is_never_read():
    d = workloads.attn_inputs("tiny")
    dn = workloads.attn_inputs("tiny", pad="nan")
    a = oracle.cross_attn(d["q"], d["K"], d["V"], d["src_len"])
    b = oracle.cross_attn(dn["q"], dn["K"], dn["V"], dn["src_len"])
    assert np.isnan(oracle.widen(dn["K"])).any()
    assert np.array_equal(a, b)


def test_beam_permutation_and_key_permutation_and_shift():
    rng = np.random.default_rng(4)
    B, k, H, S, D = 2, 5, 3, 17, 8
    q = rng.standard_normal((B, k, H, D))
    K = rng.standard_normal((B, H, S, D))
    V = rng.standard_normal((B, H, S, D))
    lens = np.array([17, 9], np.int32)
    base = oracle.cross_attn(q, K, V, lens)
    perm = rng.permutation(k)
    assert np.array_equal(oracle.cross_attn(q[:, perm], K, V, lens), base[:, perm])
    # permute the valid keys of every source (K and V together)
    K2, V2 = K.copy(), V.copy()
    for b in range(B):
        p = rng.permutation(lens[b])
        K2[b, :, :lens[b]] = K[b, :, p].transpose(1, 0, 2)
        V2[b, :, :lens[b]] = V[b, :, p].transpose(1, 0, 2)
    np.testing.assert_allclose(oracle.cross_attn(q, K2, V2, lens), base, rtol=0, atol=1e-13)
    # adding one vector to every key of a (source, head) shifts all its scores equally
    K3 = K + rng.standard_normal((B, H, 1, D))
    np.testing.assert_allclose(oracle.cross_attn(q, K3, V, lens), base, rtol=0, atol=1e-12)


def test_length_clamping_and_empty_sources():
    rng = np.random.default_rng(5)
    B, k, H, S, D = 4, 2, 2, 6, 4
    q = rng.standard_normal((B, k, H, D))
    K = rng.standard_normal((B, H, S, D))
    V = rng.standard_normal((B, H, S, D))
    out = oracle.cross_attn(q, K, V, np.array([0, -3, 99, 6], np.int32))
    assert np.array_equal(out[0], np.zeros((k, H, D)))
    assert np.array_equal(out[1], np.zeros((k, H, D)))
    assert np.array_equal(out[2], out[3] * 0 + oracle.cross_attn(
        q[2:3], K[2:3], V[2:3], np.array([6], np.int32))[0])


def test_rejects_bad_shapes():
    with pytest.raises(ValueError):
        oracle.cross_attn(np.zeros((1, 1, 1, 4)), np.zeros((1, 1, 3, 5)), np.zeros((1, 1, 3, 5)),
                          np.ones(1, np.int32))


# ---- the layout of Eq. 1: K/V replicated per beam ---------------------------

@settings(max_examples=40, deadline=None)
@given(B=st.integers(1, 3), k=st.integers(1, 4), H=st.integers(1, 3), S=st.integers(1, 30),
       D=st.sampled_from([1, 4, 16]), seed=st.integers(0, 2**31 - 1))
def test_replicated_layout_matches_library_sdpa_per_hypothesis(B, k, H, S, D, seed):
    # every hypothesis has its own K/V copy here (they need not be equal)
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, k, H, D))
    K = rng.standard_normal((B * k, H, S, D))
    V = rng.standard_normal((B * k, H, S, D))
    lens = rng.integers(-1, S + 2, size=B).astype(np.int32)
    got = oracle.cross_attn_replicated(q, K, V, lens)
    want = sdpa_reference(q.reshape(B * k, 1, H, D), K, V, np.repeat(lens, k)).reshape(B, k, H, D)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_replicated_copies_equal_dedup_bitwise():
    # Eq. 4's claim: with every beam's copy equal to the source's, the
    # de-duplicated cache gives exactly the replicated result.
    rng = np.random.default_rng(21)
    B, k, H, S, D = 3, 5, 2, 41, 16
    q = rng.standard_normal((B, k, H, D))
    K = rng.standard_normal((B, H, S, D))
    V = rng.standard_normal((B, H, S, D))
    lens = np.array([41, 7, 0], np.int32)
    rep = oracle.cross_attn_replicated(q, np.repeat(K, k, axis=0), np.repeat(V, k, axis=0), lens)
    assert np.array_equal(rep, oracle.cross_attn(q, K, V, lens))


def test_replicated_rejects_bad_shapes():
    q = np.zeros((2, 3, 1, 4))
    with pytest.raises(ValueError):
        oracle.cross_attn_replicated(q, np.zeros((2, 1, 5, 4)), np.zeros((2, 1, 5, 4)), [5, 5])
