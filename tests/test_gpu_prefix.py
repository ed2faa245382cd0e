"""GPU parity of fs_beam_prefix_attn against the fp64 oracle (Appendix A,
Eq. 2 and Eq. 3): a prefix shared by the beams of a sample plus per-beam
generated tokens, one softmax over both.  Also the invariants: the prefix
passed once per sample gives the same bits as the prefix replicated per beam,
beams permute, padding is never read, and with no generated token the result
equals the encoder-decoder form bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2106_04718_amd import api, workloads

from _gpu import assert_attn_close, bits, device, say, to_dev

pytestmark = pytest.mark.gpu


def run(d: dict, ws=None) -> torch.Tensor:
    o = api.beam_prefix_attn(to_dev(d["q"]), to_dev(d["Kp"]), to_dev(d["Vp"]),
                             to_dev(np.asarray(d["prefix_len"], np.int32)), to_dev(d["Kt"]),
                             to_dev(d["Vt"]), d["t"], workspace=ws)
    torch.cuda.synchronize()
    return o


def ref(d: dict) -> np.ndarray:
    return oracle.prefix_attn(d["q"], d["Kp"], d["Vp"], d["prefix_len"], d["Kt"], d["Vt"], d["t"])


def case(B, k, H, N, T, D, dtype, plen, t, seed):
    rng = np.random.default_rng(seed)

    def draw(shape):
        x = rng.standard_normal(shape).astype(np.float32)
        return x if dtype == "f32" else workloads.f32_to_bf16_bits(x)

    return {"q": draw((B, k, H, D)), "Kp": draw((B, H, N, D)), "Vp": draw((B, H, N, D)),
            "prefix_len": np.asarray(plen, np.int32), "Kt": draw((B * k, H, T, D)),
            "Vt": draw((B * k, H, T, D)), "t": t}


@pytest.mark.parametrize("name", ["tiny_prefix", "gpt2"])
def test_config_parity(name):
    say(f"[prefix parity] config={name}")
    d = workloads.prefix_inputs(name)
    err = assert_attn_close(run(d), ref(d), name)
    say(f"[prefix parity] config={name} max_abs_err={err:.3e}")


@pytest.mark.parametrize("t", [0, 1, 63, 64, 65, 140, 300])
def test_generated_lengths(t):
    d = case(3, 4, 2, 700, 300, 64, "bf16", [700, 256, 1], t, seed=t)
    say(f"[prefix edge] t={t}")
    assert_attn_close(run(d), ref(d), f"t={t}")


def test_no_prefix_and_no_key_at_all():
    d = case(3, 2, 2, 64, 20, 32, "f32", [0, 0, 5], 7, seed=1)
    say("[prefix edge] empty prefix")
    assert_attn_close(run(d), ref(d), "empty prefix")
    d0 = dict(d, t=0)
    out = bits(run(d0))
    assert np.all(out[0] == 0) and np.all(out[1] == 0)       # P = 0 and t = 0: zero rows
    assert_attn_close(run(d0), ref(d0), "t = 0")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("D", [16, 32, 64, 128])
def test_head_dims(dtype, D):
    d = case(4, 3, 2, 301, 80, D, dtype, [301, 257, 64, 0], 70, seed=D)
    say(f"[prefix edge] dtype={dtype} D={D}")
    assert_attn_close(run(d), ref(d), f"{dtype} D={D}")


@pytest.mark.parametrize("k", [1, 2, 5, 8])
def test_beam_counts(k):
    d = case(2, k, 3, 200, 40, 64, "bf16", [200, 33], 40, seed=10 + k)
    say(f"[prefix edge] k={k}")
    assert_attn_close(run(d), ref(d), f"k={k}")


def test_without_generated_tokens_equals_encoder_decoder_form_bitwise():
    d = case(4, 4, 2, 700, 16, 64, "bf16", [700, 513, 64, 1], 0, seed=5)
    say("[prefix invariant] t=0 vs fs_beam_cross_attn")
    a = bits(run(d))
    b = api.beam_cross_attn(to_dev(d["q"]), to_dev(d["Kp"]), to_dev(d["Vp"]), to_dev(d["prefix_len"]))
    torch.cuda.synchronize()
    assert np.array_equal(a, bits(b))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_shared_prefix_equals_replicated_prefix_bitwise(dtype):
    B, k, H, N, T, D = 3, 4, 2, 600, 100, 64
    d = case(B, k, H, N, T, D, dtype, [600, 300, 2], 90, seed=7)
    rep = {"q": d["q"].reshape(B * k, 1, H, D), "Kp": np.repeat(d["Kp"], k, axis=0),
           "Vp": np.repeat(d["Vp"], k, axis=0), "prefix_len": np.repeat(d["prefix_len"], k),
           "Kt": d["Kt"], "Vt": d["Vt"], "t": d["t"]}
    say(f"[prefix invariant] shared == replicated {dtype}")
    assert np.array_equal(bits(run(d)).reshape(B * k, 1, H, D), bits(run(rep)))


def test_beam_permutation_determinism_and_padding():
    B, k = 2, 4
    d = case(B, k, 3, 333, 50, 64, "bf16", [333, 100], 45, seed=9)
    say("[prefix invariant] permutation / padding")
    base = bits(run(d))
    perm = np.array([2, 0, 3, 1])
    hyp = (np.arange(B)[:, None] * k + perm[None, :]).ravel()
    dp = dict(d, q=np.ascontiguousarray(d["q"][:, perm]), Kt=np.ascontiguousarray(d["Kt"][hyp]),
              Vt=np.ascontiguousarray(d["Vt"][hyp]))
    assert np.array_equal(bits(run(dp)), base[:, perm])
    assert np.array_equal(bits(run(d)), base)
    dn = {kk: (v.copy() if isinstance(v, np.ndarray) else v) for kk, v in d.items()}
    nan = workloads.BF16_NAN
    for b, P in enumerate(d["prefix_len"]):
        dn["Kp"][b, :, P:] = nan
        dn["Vp"][b, :, P:] = nan
    dn["Kt"][:, :, d["t"]:] = nan
    dn["Vt"][:, :, d["t"]:] = nan
    assert np.array_equal(bits(run(dn)), base)


def test_workspace_reused_across_sizes_and_entry_points():
    # Zero-filled once, then shared by calls of both entry points whose
    # record counts differ: each must take only the records it wrote.
    dev = device()
    need = api.beam_prefix_attn_workspace_bytes(3, 4, 2, 700, 100, 64, torch.bfloat16)
    ws = api.new_workspace(need, dev)
    for rep in range(4):
        d = case(3, 4, 2, 700, 100, 64, "bf16", [700 - 100 * rep, 50 * rep, 256], 30 * rep, seed=20 + rep)
        say(f"[prefix workspace reuse] rep={rep}")
        assert_attn_close(run(d, ws=ws), ref(d), f"rep {rep}")
        o = api.beam_cross_attn(to_dev(d["q"]), to_dev(d["Kp"]), to_dev(d["Vp"]),
                                to_dev(d["prefix_len"]), workspace=ws)
        torch.cuda.synchronize()
        assert_attn_close(o, ref(dict(d, t=0)), f"rep {rep}, encoder-decoder form")


@pytest.mark.parametrize("dtype,D,k,t", [("bf16", 64, 4, 64), ("bf16", 64, 4, 0), ("f32", 32, 5, 140),
                                         ("bf16", 128, 8, 65), ("f32", 16, 1, 9)])
def test_decompositions_give_identical_bits(dtype, D, k, t):
    # Split-KV with a generated-token record, and the one-workgroup-per-row
    # kernel, fold the same states in the same order: identical bits.
    d = case(3, k, 2, 1100, 150, D, dtype, [1100, 0, 513], t, seed=90 + D + t)
    say(f"[prefix paths] dtype={dtype} D={D} k={k} t={t}")
    outs = {}
    for p in ("split", "whole1", "whole2", "whole4"):
        with api.attn_path(p):
            outs[p] = bits(run(d))
    assert np.array_equal(outs["whole1"], outs["split"])
    assert np.array_equal(outs["whole2"], outs["split"])
    assert np.array_equal(outs["whole4"], outs["split"])
    assert_attn_close(run(d), ref(d), f"paths {dtype} D={D} k={k} t={t}")
