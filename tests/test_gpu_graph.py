"""The decode step under HIP graph capture.

The cross-attention with one workgroup per row and the n-gram step keep no
state between calls, so a captured step replays like an eager one: each
replay, on inputs changed in place between replays (with eager work and
synchronisations in between), must give the eager call's bits.  Calls whose
workgroups exchange tagged records (the split-KV attention, the selection
step) tag them, when captured, by counters in their workspaces that each
replay advances, and replay like eager calls as well.
"""
import numpy as np
import pytest
import torch

from paper_2106_04718_amd import _native, api, workloads

from _gpu import bits, device, say

pytestmark = pytest.mark.gpu


def draw(rng, shape):
    return torch.from_numpy(workloads.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32)).view(np.int16))


def fill_inputs(rng, bufs, S, V):
    """New values in place (host-drawn, copied in), the way a decoder
    refreshes its buffers between steps."""
    q, K, Vv, lens, tokens, logits = bufs
    q.copy_(draw(rng, tuple(q.shape)).view(torch.bfloat16))
    K.copy_(draw(rng, tuple(K.shape)).view(torch.bfloat16))
    Vv.copy_(draw(rng, tuple(Vv.shape)).view(torch.bfloat16))
    lens.copy_(torch.from_numpy(rng.integers(0, S + 1, size=lens.shape[0]).astype(np.int32)))
    tk = rng.integers(0, 40, size=tuple(tokens.shape)).astype(np.int32)
    tokens.copy_(torch.from_numpy(tk))
    logits.copy_(torch.from_numpy(rng.standard_normal(tuple(logits.shape)).astype(np.float32)))


def test_captured_step_replays_like_eager_calls():
    dev = device()
    B, k, H, S, D, Vsz, t, n = 8, 4, 16, 700, 64, 3000, 60, 3   # 128 rows: one workgroup per row
    rng = np.random.default_rng(17)
    q = torch.empty((B, k, H, D), dtype=torch.bfloat16, device=dev)
    K = torch.empty((B, H, S, D), dtype=torch.bfloat16, device=dev)
    Vv = torch.empty_like(K)
    lens = torch.empty((B,), dtype=torch.int32, device=dev)
    tokens = torch.empty((B * k, t), dtype=torch.int32, device=dev)
    logits = torch.empty((B * k, Vsz), dtype=torch.float32, device=dev)
    bufs = (q, K, Vv, lens, tokens, logits)
    out = torch.empty_like(q)
    ws = api.new_workspace(api.beam_cross_attn_workspace_bytes(B, k, H, S, D, torch.bfloat16), dev)
    fill_inputs(rng, bufs, S, Vsz)
    torch.cuda.synchronize()

    def step():
        api.beam_cross_attn(q, K, Vv, lens, out=out, workspace=ws)
        api.ngram_block(tokens, n, logits)

    # warm the kernels on a side stream before capture, as torch asks
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    say("[graph] capture cross-attention + n-gram")
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    for rep in range(4):
        say(f"[graph] replay {rep}")
        fill_inputs(rng, bufs, S, Vsz)
        logits0 = logits.clone()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got_out, got_logits = bits(out).copy(), bits(logits).copy()
        # the same inputs, eager, into fresh outputs
        logits.copy_(logits0)
        ref_out = api.beam_cross_attn(q, K, Vv, lens, workspace=ws)
        api.ngram_block(tokens, n, logits)
        torch.cuda.synchronize()
        assert np.array_equal(got_out, bits(ref_out)), f"attention, replay {rep}"
        assert np.array_equal(got_logits, bits(logits)), f"n-gram, replay {rep}"


def test_record_exchanging_calls_replay_like_eager_calls():
    """The split-KV attention (2 rows), the split-cache attention over those
    rows, a fused step in the split-KV form and the selection step exchange
    tagged records through their workspaces.  Captured, they tag them by the
    workspaces' counters: every replay (back to back, and with eager calls
    on the same workspaces in between) gives the eager calls' bits."""
    dev = device()
    rng = np.random.default_rng(5)
    B, k, H, S, D, Vsz, t, n, c, T, tg = 2, 4, 1, 600, 64, 500, 12, 3, 8, 16, 9
    q = torch.empty((B, k, H, D), dtype=torch.bfloat16, device=dev)
    K = torch.empty((B, H, S, D), dtype=torch.bfloat16, device=dev)
    Vv = torch.empty_like(K)
    lens = torch.empty((B,), dtype=torch.int32, device=dev)
    tokens = torch.empty((B * k, t), dtype=torch.int32, device=dev)
    logits = torch.empty((B * k, Vsz), dtype=torch.float32, device=dev)
    bufs = (q, K, Vv, lens, tokens, logits)
    Kt = torch.empty((B * k, H, T, D), dtype=torch.bfloat16, device=dev)
    Vt = torch.empty_like(Kt)
    scores = torch.empty((B * k,), dtype=torch.float32, device=dev)
    step_logits = torch.empty_like(logits)
    ws = [api.new_workspace(api.beam_cross_attn_workspace_bytes(B, k, H, S, D, torch.bfloat16), dev),
          api.new_workspace(api.beam_prefix_attn_workspace_bytes(B, k, H, S, T, D, torch.bfloat16), dev),
          api.new_workspace(api.beam_cross_attn_workspace_bytes(B, k, H, S, D, torch.bfloat16), dev),
          api.new_workspace(api.beam_select_workspace_bytes(B, k, Vsz, c), dev)]

    def new_outs():
        return (torch.empty_like(q), torch.empty_like(q), torch.empty_like(q),
                (torch.empty((B, c), dtype=torch.float32, device=dev), torch.empty((B, c), dtype=torch.int32, device=dev),
                 torch.empty((B, c), dtype=torch.int32, device=dev)))

    def fill():
        fill_inputs(rng, bufs, S, Vsz)
        Kt.copy_(draw(rng, tuple(Kt.shape)).view(torch.bfloat16))
        Vt.copy_(draw(rng, tuple(Vt.shape)).view(torch.bfloat16))
        scores.copy_(torch.from_numpy(-np.abs(rng.standard_normal(B * k)).astype(np.float32)))
        step_logits.copy_(logits)

    def step(o):
        api.beam_cross_attn(q, K, Vv, lens, out=o[0], workspace=ws[0])
        api.beam_prefix_attn(q, K, Vv, lens, Kt, Vt, tg, out=o[1], workspace=ws[1])
        api.beam_decode_step(q, K, Vv, lens, tokens, n, step_logits, out=o[2], workspace=ws[2])
        api.beam_select(logits, scores, k, c, tokens=tokens, n=n, out=o[3], workspace=ws[3])

    def snapshot(o):
        return [bits(o[0]).copy(), bits(o[1]).copy(), bits(o[2]).copy(), bits(step_logits).copy(),
                *(bits(x).copy() for x in o[3])]

    graph_outs = new_outs()
    fill()
    torch.cuda.synchronize()
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        step(graph_outs)
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    say("[graph] capture split-KV attention, split-cache attention, fused step, selection")
    with torch.cuda.graph(g):
        step(graph_outs)
    torch.cuda.synchronize()

    names = ["attention", "split cache", "fused step", "fused step n-gram", "select scores", "select beams",
             "select tokens"]
    for rep in range(6):
        say(f"[graph] replay {rep}")
        fill()
        saved = step_logits.clone()
        torch.cuda.synchronize()
        g.replay()
        if rep % 2:   # every other time, a second replay right after (same inputs, fresh logits)
            torch.cuda.synchronize()
            step_logits.copy_(saved)
            g.replay()
        torch.cuda.synchronize()
        got = snapshot(graph_outs)
        # the same inputs, eager, on the same workspaces
        step_logits.copy_(saved)
        ref_outs = new_outs()
        step(ref_outs)
        torch.cuda.synchronize()
        ref = snapshot(ref_outs)
        for name, a, b in zip(names, got, ref):
            assert np.array_equal(a, b), f"{name}, replay {rep}"
        assert np.all((ref[0] & 0x7f80) != 0x7f80), "attention output not finite"   # bf16 exponent bits


def test_fused_step_replays_like_eager_calls():
    dev = device()
    B, k, H, S, D, Vsz, t, n = 8, 4, 16, 700, 64, 3000, 60, 3   # 128 rows: one workgroup per row
    rng = np.random.default_rng(11)
    q = torch.empty((B, k, H, D), dtype=torch.bfloat16, device=dev)
    K = torch.empty((B, H, S, D), dtype=torch.bfloat16, device=dev)
    Vv = torch.empty_like(K)
    lens = torch.empty(B, dtype=torch.int32, device=dev)
    tokens = torch.empty((B * k, t), dtype=torch.int32, device=dev)
    logits = torch.empty((B * k, Vsz), dtype=torch.float32, device=dev)
    bufs = (q, K, Vv, lens, tokens, logits)
    out = torch.empty_like(q)
    ws = api.new_workspace(api.beam_cross_attn_workspace_bytes(B, k, H, S, D, torch.bfloat16), dev)
    fill_inputs(rng, bufs, S, Vsz)
    api.beam_decode_step(q, K, Vv, lens, tokens, n, logits, out=out, workspace=ws)   # warm-up outside capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    say("[graph] capture of the fused step")
    with torch.cuda.graph(g):
        api.beam_decode_step(q, K, Vv, lens, tokens, n, logits, out=out, workspace=ws)
    for rep in range(4):
        fill_inputs(rng, bufs, S, Vsz)
        lg0 = logits.clone()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got_out, got_lg = bits(out), bits(logits)
        logits.copy_(lg0)
        eager = api.beam_decode_step(q, K, Vv, lens, tokens, n, logits)
        torch.cuda.synchronize()
        assert np.array_equal(got_out, bits(eager)), f"attention, replay {rep}"
        assert np.array_equal(got_lg, bits(logits)), f"n-gram, replay {rep}"


def test_validate_mode_is_refused_under_capture():
    # Debug mode copies the lengths to the host, which a capturing stream
    # cannot do: the call is refused before any HIP call and the capture
    # stays intact.  Outside capture it accepts valid lengths and rejects
    # an out-of-range one (the kernel never sees it).
    dev = device()
    B, k, H, S, D = 8, 4, 16, 300, 64          # 128 rows: the capturable form
    rng = np.random.default_rng(1)
    q = draw(rng, (B, k, H, D)).view(torch.bfloat16).to(dev)
    K = draw(rng, (B, H, S, D)).view(torch.bfloat16).to(dev)
    Vv = draw(rng, (B, H, S, D)).view(torch.bfloat16).to(dev)
    lens = torch.from_numpy(rng.integers(1, S + 1, size=B).astype(np.int32)).to(dev)
    tok = torch.zeros((B * k, 8), dtype=torch.int32, device=dev)
    logits = torch.zeros((B * k, 50), dtype=torch.float32, device=dev)
    out = torch.empty_like(q)
    ws = api.new_workspace(api.beam_cross_attn_workspace_bytes(B, k, H, S, D, torch.bfloat16), dev)
    say("[graph] debug mode under capture")
    with api.validate_lengths():
        api.beam_cross_attn(q, K, Vv, lens, out=out, workspace=ws)    # valid lengths: accepted
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        errs = []
        with torch.cuda.graph(g):
            api.ngram_block(tok, 3, logits)
            for call in (lambda: api.beam_cross_attn(q, K, Vv, lens, out=out, workspace=ws),
                         lambda: api.beam_decode_step(q, K, Vv, lens, tok, 3, logits, out=out, workspace=ws)):
                try:
                    call()
                except _native.NativeError as e:
                    errs.append((e.status, str(e)))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert len(errs) == 2, errs
        assert all(st == _native.FS_ERR_UNSUPPORTED and "FS_VALIDATE" in msg for st, msg in errs), errs
        bad = lens.clone()
        bad[3] = S + 1
        with pytest.raises(_native.NativeError) as ei:
            api.beam_cross_attn(q, K, Vv, bad, out=out, workspace=ws)
        assert ei.value.status == _native.FS_ERR_INVALID_ARG and "src_len[3]" in str(ei.value)
