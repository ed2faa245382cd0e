"""fs_beam_decode_step_noalloc, the decode step for callers that cannot
allocate, called through the C ABI: its outputs equal fs_beam_decode_step's
(with a caller workspace) bit for bit, on two calls in a row, the second
smaller, on the decomposition that keeps records in the library's scratch
array and on one that keeps none.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2106_04718_amd import _native as N
from paper_2106_04718_amd import api, workloads

from _gpu import bits, device, say, to_dev

pytestmark = pytest.mark.gpu


def case(rng, B, k, H, S, D, rows_t, vocab):
    def draw(shape):
        return workloads.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32))
    lens = rng.integers(0, S + 1, size=B).astype(np.int32)
    lens[0] = S
    tokens = workloads.plant_repeats(rng.integers(0, 30, size=(B * k, rows_t)).astype(np.int32), 3, rows_t, rng,
                                     per_row=2)
    return {"q": draw((B, k, H, D)), "K": draw((B, H, S, D)), "V": draw((B, H, S, D)), "src_len": lens,
            "tokens": tokens, "logits": rng.standard_normal((B * k, vocab)).astype(np.float32)}


def run_both(d, n=3):
    q, K, V = to_dev(d["q"]), to_dev(d["K"]), to_dev(d["V"])
    lens, tok = to_dev(d["src_len"]), to_dev(d["tokens"])
    B, k, H, D = q.shape
    S = K.shape[2]
    rows, t = tok.shape
    lg_ref, lg_new = to_dev(d["logits"]), to_dev(d["logits"])
    out_ref = api.beam_decode_step(q, K, V, lens, tok, n, lg_ref)
    out_new = torch.empty_like(q)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    st = N.lib().fs_beam_decode_step_noalloc(
        q.data_ptr(), K.data_ptr(), V.data_ptr(), lens.data_ptr(), out_new.data_ptr(), B, k, H, S, D, N.FS_BF16,
        tok.data_ptr(), t, t, n, lg_new.data_ptr(), lg_new.shape[1], stream)
    assert st == N.FS_OK, N.last_error()
    torch.cuda.synchronize()
    return (bits(out_ref), bits(lg_ref)), (bits(out_new), bits(lg_new))


@pytest.mark.parametrize("sizes", [
    # (B, k, H, S, D): fewer than 128 rows take the split-KV form, whose
    # partial records live in the scratch array; then a smaller second call
    [(3, 4, 4, 1100, 64), (2, 4, 4, 300, 64)],
    [(2, 8, 3, 700, 128), (1, 5, 2, 257, 32)],
    # 128 rows and more: one workgroup per row, no records at all
    [(8, 4, 16, 900, 64), (4, 4, 32, 400, 64)],
])
def test_noalloc_step_equals_the_workspace_step(sizes):
    device()
    rng = np.random.default_rng(sum(sum(s) for s in sizes))
    for call, (B, k, H, S, D) in enumerate(sizes):
        d = case(rng, B, k, H, S, D, 40, 300)
        say(f"[noalloc] call {call}: B={B} k={k} H={H} S={S} D={D}")
        ref, new = run_both(d)
        assert np.array_equal(new[0], ref[0]), f"attention bits, call {call}"
        assert np.array_equal(new[1], ref[1]), f"n-gram bits, call {call}"


def test_noalloc_refuses_records_beyond_the_scratch_array():
    # 127 rows of 64 chunks: the split-KV records need about 67 MB
    lib = N.lib()
    fake = 1 << 20
    st = lib.fs_beam_decode_step_noalloc(fake, fake * 2, fake * 3, fake * 4, fake * 5, 1, 8, 127, 8192, 128,
                                         N.FS_BF16, fake * 6, 8, 8, 3, fake * 7, 100, None)
    assert st == N.FS_ERR_UNSUPPORTED and "scratch array" in N.last_error()


def test_noalloc_step_replays_from_a_graph():
    """The no-allocation step captured into a HIP graph (its split-KV records
    in the library's scratch array, tagged by the array's counters): every
    replay, on inputs refreshed in place, gives the bits of the workspace
    step run eagerly on the same inputs."""
    dev = device()
    rng = np.random.default_rng(23)
    B, k, H, S, D, t, n, vocab = 3, 4, 4, 900, 64, 40, 3, 300
    q = torch.empty((B, k, H, D), dtype=torch.bfloat16, device=dev)
    K = torch.empty((B, H, S, D), dtype=torch.bfloat16, device=dev)
    V = torch.empty_like(K)
    lens = torch.empty((B,), dtype=torch.int32, device=dev)
    tok = torch.empty((B * k, t), dtype=torch.int32, device=dev)
    lg = torch.empty((B * k, vocab), dtype=torch.float32, device=dev)
    out = torch.empty_like(q)

    def fill():
        d = case(rng, B, k, H, S, D, t, vocab)
        for dst, key in ((q, "q"), (K, "K"), (V, "V"), (lens, "src_len"), (tok, "tokens"), (lg, "logits")):
            dst.copy_(to_dev(d[key]))
        return d

    def noalloc_step():
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        st = N.lib().fs_beam_decode_step_noalloc(
            q.data_ptr(), K.data_ptr(), V.data_ptr(), lens.data_ptr(), out.data_ptr(), B, k, H, S, D, N.FS_BF16,
            tok.data_ptr(), t, t, n, lg.data_ptr(), vocab, stream)
        assert st == N.FS_OK, N.last_error()

    fill()
    torch.cuda.synchronize()
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        noalloc_step()
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    say("[noalloc] capture the no-allocation step")
    with torch.cuda.graph(g):
        noalloc_step()
    torch.cuda.synchronize()
    for rep in range(4):
        say(f"[noalloc] replay {rep}")
        d = fill()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (bits(out).copy(), bits(lg).copy())
        ref, _ = run_both(d)
        assert np.array_equal(got[0], ref[0]), f"attention bits, replay {rep}"
        assert np.array_equal(got[1], ref[1]), f"n-gram bits, replay {rep}"
