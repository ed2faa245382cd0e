"""GPU parity of fs_beam_select against the oracle (one beam-search selection
step, Section 2.1, with the n-gram bans of Section 4.2, Algorithm 1).

The GPU computes in fp32 and the oracle in fp64, so where two candidates are
closer than the fp32 error the two may rank them differently; that is the
only freedom allowed.  Each check:
  * the GPU's c picks per source are distinct, in range, and best first;
  * each pick's value is the fp64 value of that (beam, token) within TOL;
  * the picks are the oracle's c best up to candidates within 2*TOL of the
    oracle's c-th value (near-ties at the boundary);
  * with no near-tie at all, the (beam, token) lists equal the oracle's.
TOL = 1e-5 * (1 + |value|): the fp32 log-normaliser over V ~ 5e4 terms
(per-slice sums, then the slices) is within a few ulp of ~11, and
beam_score + (x - lse) adds two roundings at |value| ~ 30, so the error is a
few 1e-6; 1e-5 relative keeps a margin and still flags any wrong normaliser,
beam score or token.
"""
import numpy as np
import pytest
import torch
from scipy.special import logsumexp

import oracle
from paper_2106_04718_amd import api, workloads

from _gpu import device, say

pytestmark = pytest.mark.gpu


def tol(v):
    return 1e-5 * (1.0 + np.abs(v))


def fp64_values(logits, beam_scores, tokens, t, n, k, b, beam, token):
    """fp64 value of candidate (beam, token) of source b (banned: -inf)."""
    r = b * k + beam
    x = logits[r].astype(np.float64)
    lse = logsumexp(x) if np.isfinite(x).any() else -np.inf
    banned = np.zeros(logits.shape[1], bool)
    if n > 0:
        banned = np.isneginf(oracle.ngram_block(tokens[r:r + 1], n, np.zeros((1, logits.shape[1]), np.float32),
                                                t)[0])
    if banned[token] or not np.isfinite(lse):
        return -np.inf
    return beam_scores[r] + x[token] - lse


def run(d, k, c, n, t, ws=None):
    dev = device()
    lg = torch.from_numpy(np.ascontiguousarray(d["logits"])).to(dev)
    bs = torch.from_numpy(np.ascontiguousarray(d["beam_scores"])).to(dev)
    tok = torch.from_numpy(np.ascontiguousarray(d["tokens"])).to(dev) if n > 0 else None
    s, i, v = api.beam_select(lg, bs, k, c, tokens=tok, n=n, t=t, workspace=ws)
    torch.cuda.synchronize()
    return s.cpu().numpy(), i.cpu().numpy(), v.cpu().numpy()


def check(d, k, c, n, t, what, sources=None, ws=None):
    say(f"[select parity] {what}")
    gs, gi, gv = run(d, k, c, n, t, ws=ws)
    lg, bs, tok = d["logits"], d["beam_scores"], d["tokens"]
    B = lg.shape[0] // k
    V = lg.shape[1]
    idx = np.arange(B) if sources is None else np.asarray(sources)
    rows = (idx[:, None] * k + np.arange(k)[None, :]).reshape(-1)
    sub = (lg[rows], bs[rows], tok[rows] if n > 0 else None)
    cc = min(c + 1, k * V)
    rs, ri, rv = oracle.beam_select(sub[0], sub[1], sub[2], t, n, k, cc)
    exact = 0
    for jb, b in enumerate(idx):
        assert np.all((gi[b] >= 0) & (gi[b] < k) & (gv[b] >= 0) & (gv[b] < V)), f"{what}: b={b} out of range"
        flat = gi[b].astype(np.int64) * V + gv[b]
        assert len(set(flat.tolist())) == c, f"{what}: b={b} repeated pick"
        assert np.all(np.diff(gs[b][np.isfinite(gs[b])]) <= 0), f"{what}: b={b} not best first"
        val = np.array([fp64_values(lg, bs, tok, t, n, k, b, int(i), int(v)) for i, v in zip(gi[b], gv[b])])
        fin = np.isfinite(val)
        assert np.array_equal(np.isfinite(gs[b]), fin), f"{what}: b={b} -inf mismatch"
        assert np.all(np.abs(gs[b][fin] - val[fin]) <= tol(val[fin])), \
            f"{what}: b={b} value error {np.max(np.abs(gs[b][fin] - val[fin]))}"
        ref_vals, ref_flat = rs[jb][:c], ri[jb][:c].astype(np.int64) * V + rv[jb][:c]
        tau = ref_vals[c - 1]
        if np.isfinite(tau):
            sure = ref_flat[ref_vals > tau + 2 * tol(tau)]
            assert set(sure.tolist()) <= set(flat.tolist()), f"{what}: b={b} missed a clear candidate"
            assert np.all(val[fin] >= tau - 2 * tol(tau)), f"{what}: b={b} picked below the c-th value"
        gaps = np.diff(rs[jb])
        near = np.any(np.abs(gaps[np.isfinite(gaps)]) <= 4 * tol(rs[jb][1:][np.isfinite(gaps)]))
        if not near:
            assert np.array_equal(flat, ref_flat), f"{what}: b={b} order differs with no near-tie"
            exact += 1
    return exact


@pytest.mark.parametrize("name", ["tiny", "bart", "t5", "prophetnet"])
def test_config_parity(name):
    d = workloads.select_inputs(name)
    exact = check(d, d["k"], d["c"], d["n"], d["t"], f"config={name}")
    say(f"[select parity] config={name}: {exact} of {d['B']} sources compared exactly")


def test_large_config_every_source():
    d = workloads.select_inputs("large")
    exact = check(d, d["k"], d["c"], d["n"], d["t"], "config=large")
    say(f"[select parity] config=large: {exact} of {d['B']} sources compared exactly")


def random_case(B, k, V, t, seed, neg_inf=0.0):
    rng = np.random.default_rng(seed)
    lg = rng.standard_normal((B * k, V)).astype(np.float32)
    if neg_inf:
        lg[rng.random(lg.shape) < neg_inf] = -np.inf
    tok = rng.integers(0, max(2, min(V, 6)), size=(B * k, max(t, 1))).astype(np.int32)
    bs = (-rng.random(B * k) * 4).astype(np.float32)
    return {"logits": lg, "beam_scores": bs, "tokens": tok}


@pytest.mark.parametrize("k,c", [(1, 1), (1, 16), (2, 3), (3, 16), (5, 10), (8, 16), (16, 16), (16, 1)])
def test_beam_and_candidate_counts(k, c):
    d = random_case(6, k, 3001, 20, seed=100 + k * 17 + c)
    check(d, k, c, 3, 20, f"k={k} c={c}")


@pytest.mark.parametrize("V", [1, 2, 3, 7, 63, 255, 1023, 1025, 4099, 16383, 16384, 16385, 50001])
def test_vocabulary_sizes_and_ragged_slices(V):
    k = 4
    c = min(8, k * V)
    d = random_case(5, k, V, 12, seed=V)
    check(d, k, c, 2, 12, f"V={V}")


def test_bans_without_and_with_history():
    d = random_case(4, 4, 700, 40, seed=7)
    for n in (0, 1, 2, 3, 5):
        check(d, 4, 8, n, 40, f"n={n}")
    check(d, 4, 8, 3, 2, "t < n")   # no window: nothing banned


@pytest.mark.parametrize("shift", [1, 2, 3])
def test_logits_not_on_a_16_byte_boundary(shift):
    # each slice reads the aligned 16-byte window around it; a base pointer
    # 4, 8 or 12 bytes past an aligned address moves every window
    dev = device()
    k, c, n, t, V, B = 4, 8, 2, 30, 5003, 6
    d = random_case(B, k, V, t, seed=40 + shift)
    flat = torch.empty(B * k * V + shift, dtype=torch.float32, device=dev)
    lg = flat[shift:].view(B * k, V)
    lg.copy_(torch.from_numpy(d["logits"]))
    assert lg.data_ptr() % 16 == 4 * shift
    say(f"[select parity] logits at +{4 * shift} bytes")
    bs = torch.from_numpy(d["beam_scores"]).to(dev)
    tok = torch.from_numpy(d["tokens"]).to(dev)
    s, i, v = api.beam_select(lg, bs, k, c, tokens=tok, n=n, t=t)
    torch.cuda.synchronize()
    ref = run(d, k, c, n, t)
    assert np.array_equal(i.cpu().numpy(), ref[1]) and np.array_equal(v.cpu().numpy(), ref[2])
    np.testing.assert_allclose(s.cpu().numpy(), ref[0], rtol=0, atol=1e-5)
    check(d, k, c, n, t, f"aligned copy for +{4 * shift}")


def test_equal_logits_take_the_smallest_flat_indices():
    # every value ties, so the tie rule decides end to end; with 256 rows the
    # slices hold ~13k equal values each, more than the collection buffer, and
    # take the exact c-round path
    for B, V in ((3, 5000), (64, 40000)):
        lg = np.zeros((B * 4, V), np.float32)
        d = {"logits": lg, "beam_scores": np.zeros(B * 4, np.float32), "tokens": np.zeros((B * 4, 1), np.int32)}
        say(f"[select ties] B={B} V={V}")
        gs, gi, gv = run(d, 4, 16, 0, 0)
        assert np.array_equal(gi * V + gv, np.tile(np.arange(16), (B, 1))), f"V={V}"
        assert np.all(gs == gs[0, 0])


def test_neg_inf_logits_and_dead_rows():
    d = random_case(3, 4, 900, 10, seed=11, neg_inf=0.3)
    d["logits"][2] = -np.inf            # a row with every logit -inf
    d["logits"][4:8] = -np.inf          # a source with no finite candidate
    check(d, 4, 8, 2, 10, "-inf logits")
    gs, gi, gv = run(d, 4, 8, 2, 10)
    assert np.all(np.isneginf(gs[1])) and np.array_equal(gi[1] * 900 + gv[1], np.arange(8))


def test_many_bans_low_entropy_rows():
    rng = np.random.default_rng(13)
    d = random_case(4, 4, 64, 200, seed=13)
    d["tokens"] = rng.integers(0, 40, size=(16, 200)).astype(np.int32)
    check(d, 4, 8, 1, 200, "n=1 bans up to 40 ids per row")
    check(d, 4, 8, 2, 200, "n=2 on low-entropy rows")


def test_deterministic_bits_and_workspace_reuse():
    dev = device()
    ws = api.new_workspace(api.beam_select_workspace_bytes(64, 4, 32128, 16), dev)
    d = workloads.select_inputs("t5")
    a = run(d, 4, 8, 3, 200, ws=ws)
    b = run(d, 4, 8, 3, 200, ws=ws)
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
    small = random_case(2, 4, 999, 8, seed=17)
    check(small, 4, 8, 2, 8, "smaller problem, same workspace", ws=ws)
    check(d, 4, 8, 3, 200, "t5 again after it", ws=ws)


def test_rejects_unsupported_sizes_on_device_tensors():
    dev = device()
    lg = torch.zeros((8, 100), dtype=torch.float32, device=dev)
    bs = torch.zeros(8, dtype=torch.float32, device=dev)
    with pytest.raises(Exception, match="c=17"):
        api.beam_select(lg, bs, 4, 17)
    with pytest.raises(Exception, match="k=17"):
        api.beam_select(torch.zeros((17, 100), dtype=torch.float32, device=dev),
                        torch.zeros(17, dtype=torch.float32, device=dev), 17, 4)
    with pytest.raises(ValueError):
        api.beam_select(lg, bs, 3, 4)      # rows not a multiple of k
