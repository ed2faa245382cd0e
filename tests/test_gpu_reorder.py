"""GPU parity of fs_cache_reorder against the oracle (per-beam cache reorder,
Section 2.2 cache maintenance; Section 4.1.1).

The reorder moves bytes, so the bar is bit equality with the oracle on the
whole cache: the reordered rows, the capacity rows tau >= t (filled with NaN
payloads that must survive) and the rows of beams that keep their history.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2106_04718_amd import api

from _gpu import device, say

pytestmark = pytest.mark.gpu


def make_cache(rows, H, T, D, dtype, seed, t=None):
    """Random bit patterns; capacity rows tau >= t hold NaN payloads."""
    rng = np.random.default_rng(seed)
    if dtype == torch.bfloat16:
        bits = rng.integers(-2**15, 2**15, size=(rows, H, T, D)).astype(np.int16)
        if t is not None and t < T:
            bits[:, :, t:] = np.int16(0x7FC1)   # a bf16 NaN payload
        return bits
    bits = rng.integers(0, 2**32, size=(rows, H, T, D), dtype=np.uint64).astype(np.uint32)
    if t is not None and t < T:
        bits[:, :, t:] = 0x7FC00001 + (np.arange(bits[:, :, t:].size, dtype=np.uint32) % 5).reshape(bits[:, :, t:].shape)
    return bits


def to_dev(bits, dtype, dev, shift=0):
    """Device tensor with these bit patterns; `shift` elements of padding
    before it move the base pointer off a 16-byte boundary."""
    flat_t = torch.from_numpy(bits.view(np.int16) if dtype == torch.bfloat16 else bits.view(np.int32))
    flat = torch.empty(bits.size + shift, dtype=flat_t.dtype, device=dev)
    x = flat[shift:].view(bits.shape)
    x.copy_(flat_t.to(dev))
    return x.view(dtype)


def bits_of(x):
    return x.view(torch.int16 if x.dtype == torch.bfloat16 else torch.int32).cpu().numpy()


def check(B, k, H, T, t, D, dtype, parent, seed, what, shift=0, with_v=True):
    say(f"[reorder parity] {what}: B={B} k={k} H={H} T={T} t={t} D={D} {dtype} shift={shift}")
    dev = device()
    kb = make_cache(B * k, H, T, D, dtype, seed, t)
    vb = make_cache(B * k, H, T, D, dtype, seed + 1, t)
    K = to_dev(kb, dtype, dev, shift)
    V = to_dev(vb, dtype, dev, shift) if with_v else None
    par = torch.from_numpy(np.asarray(parent, np.int32)).to(dev)
    api.cache_reorder(K, V, par, k, t)
    torch.cuda.synchronize()
    want_k = oracle.cache_reorder(kb, parent, k, t)
    assert np.array_equal(bits_of(K), want_k.view(bits_of(K).dtype)), f"{what}: K differs"
    if with_v:
        want_v = oracle.cache_reorder(vb, parent, k, t)
        assert np.array_equal(bits_of(V), want_v.view(bits_of(V).dtype)), f"{what}: V differs"


def random_parent(B, k, seed, bad=0.0):
    rng = np.random.default_rng(seed)
    p = rng.integers(0, k, size=B * k).astype(np.int32)
    if bad:
        m = rng.random(B * k) < bad
        p[m] = rng.choice(np.array([-1, k, k + 7, -2**31], np.int32), size=int(m.sum()))
    return p


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_decode_shaped_caches(dtype):
    # BART-large-shaped decoder self-attention cache (16 heads, D = 64, 140
    # positions) at the middle and the end of generation, and a GPT2-shaped one
    for (B, k, H, T, D), t in (((32, 4, 16, 140, 64), 70), ((32, 4, 16, 140, 64), 140), ((16, 4, 12, 64, 64), 64)):
        check(B, k, H, T, t, D, dtype, random_parent(B, k, seed=B + t), seed=t, what="decode shape")


@pytest.mark.parametrize("k", [1, 2, 3, 5, 8, 9, 16])
def test_beam_counts(k):
    B, H, T, D = 5, 3, 33, 32
    check(B, k, H, T, 29, D, torch.bfloat16, random_parent(B, k, seed=k), seed=100 + k, what=f"k={k}")


@pytest.mark.parametrize("D,dtype", [(16, torch.bfloat16), (128, torch.bfloat16), (6, torch.bfloat16),
                                     (3, torch.float32), (5, torch.float32), (2, torch.bfloat16)])
def test_row_widths_and_4_byte_moves(D, dtype):
    # rows that are not a whole number of 16 bytes take the 4-byte path
    B, k, H, T = 3, 4, 2, 17
    check(B, k, H, T, 11, D, dtype, random_parent(B, k, seed=D), seed=200 + D, what=f"D={D}")


@pytest.mark.parametrize("shift", [1, 2, 3])
def test_cache_not_on_a_16_byte_boundary(shift):
    B, k, H, T, D = 4, 4, 2, 24, 16
    check(B, k, H, T, 24, D, torch.float32, random_parent(B, k, seed=shift), seed=300 + shift,
          what="unaligned base", shift=shift)


def test_parent_patterns():
    B, k, H, T, D = 6, 4, 4, 40, 64
    patterns = {
        "identity": np.tile(np.arange(k, dtype=np.int32), B),
        "all from beam 0": np.zeros(B * k, np.int32),
        "reversed": np.tile(np.arange(k - 1, -1, -1, dtype=np.int32), B),
        "swap pairs": np.tile(np.array([1, 0, 3, 2], np.int32), B),
        "rotation": np.tile(np.array([1, 2, 3, 0], np.int32), B),
        "out of range mixed in": random_parent(B, k, seed=9, bad=0.4),
    }
    for name, p in patterns.items():
        check(B, k, H, T, 33, D, torch.bfloat16, p, seed=400, what=name)


def test_empty_history_and_one_tensor():
    B, k, H, T, D = 3, 4, 2, 10, 16
    p = random_parent(B, k, seed=1)
    check(B, k, H, T, 0, D, torch.bfloat16, p, seed=500, what="t = 0")
    check(B, k, H, T, 7, D, torch.bfloat16, p, seed=501, what="K only", with_v=False)


def test_two_steps_in_a_row_match_the_oracle():
    dev = device()
    B, k, H, T, D = 8, 4, 4, 30, 64
    kb = make_cache(B * k, H, T, D, torch.bfloat16, 600)
    K = to_dev(kb, torch.bfloat16, dev)
    want = kb
    for step, t in enumerate((10, 11, 12)):
        p = random_parent(B, k, seed=700 + step)
        api.cache_reorder(K, None, torch.from_numpy(p).to(dev), k, t)
        want = oracle.cache_reorder(want, p, k, t)
    torch.cuda.synchronize()
    assert np.array_equal(bits_of(K), want)


def test_rejects_bad_arguments_on_device_tensors():
    dev = device()
    K = torch.zeros((8, 2, 5, 16), dtype=torch.bfloat16, device=dev)
    p = torch.zeros(8, dtype=torch.int32, device=dev)
    with pytest.raises(Exception, match="t=6"):
        api.cache_reorder(K, None, p, 4, 6)
    with pytest.raises(Exception, match="k=17"):
        api.cache_reorder(torch.zeros((17, 1, 2, 16), dtype=torch.bfloat16, device=dev), None,
                          torch.zeros(17, dtype=torch.int32, device=dev), 17, 2)
    with pytest.raises(Exception, match="overlaps"):
        api.cache_reorder(K, K, p, 4, 5)
    with pytest.raises(Exception, match="4-byte"):
        api.cache_reorder(torch.zeros((4, 1, 3, 3), dtype=torch.bfloat16, device=dev), None,
                          torch.zeros(4, dtype=torch.int32, device=dev), 4, 3)
