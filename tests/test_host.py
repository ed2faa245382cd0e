"""Host-side logic without a GPU: the seeded input recipe, the algorithmic
byte counts the roofline figures are built on, and the benchmark's contract
(one GPU only; traffic figures used only while the kernel sources match).
"""
import dataclasses
import json
import subprocess
import sys
from pathlib import Path

import numpy as np
import pytest
import torch

from paper_2106_04718_amd import workloads

ROOT = Path(__file__).resolve().parents[1]
sys.path.insert(0, str(ROOT))
import bench  # noqa: E402


# ---- bf16 rounding -----------------------------------------------------------

def test_bf16_rounding_is_round_to_nearest_even():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 20000),
                        np.array([0.0, -0.0, 1.0, -1.0, 3.0e38, -3.0e38, np.finfo(np.float32).max,
                                  np.finfo(np.float32).tiny], np.float32)])
    # ties: the halfway points between bf16 neighbours round to the even one
    base = rng.integers(0x0080, 0x7F00, 2000).astype(np.uint32) << 16
    ties = (base | 0x8000).view(np.float32)
    x = np.concatenate([x, ties, -ties])
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(workloads.f32_to_bf16_bits(x), want)
    t = workloads.f32_to_bf16_bits(ties)
    assert np.all((t & 1) == 0), "a tie went to the odd neighbour"


# ---- the Zipf token law ------------------------------------------------------

def test_zipf_tokens_follow_the_power_law():
    rng = np.random.default_rng(1)
    V, s, n = 6, 1.1, 300_000
    ids = workloads.zipf_tokens(rng, (n,), V, s)
    assert ids.dtype == np.int32 and ids.min() >= 0 and ids.max() < V
    p = np.arange(1, V + 1, dtype=np.float64) ** -s
    p /= p.sum()
    freq = np.bincount(ids, minlength=V) / n
    # each frequency within 5 standard errors of its probability
    assert np.all(np.abs(freq - p) <= 5 * np.sqrt(p * (1 - p) / n)), (freq, p)


# ---- the seeded configs -------------------------------------------------------

@pytest.mark.parametrize("name", ["tiny", "bart", "t5"])
def test_inputs_are_deterministic_and_shaped(name):
    cfg = workloads.get(name)
    # the same recipe at a size the host builds in moments
    small = cfg if cfg.name == "tiny" else dataclasses.replace(
        cfg, B=min(cfg.B, 3), S=min(cfg.S, 256), len_hi=min(cfg.len_hi, 256), len_lo=min(cfg.len_lo, 200))
    a, b = workloads.attn_inputs(small), workloads.attn_inputs(small)
    for key in ("q", "K", "V", "src_len"):
        np.testing.assert_array_equal(a[key], b[key])
    assert a["q"].shape == (small.B, small.k, small.H, small.D)
    assert a["K"].shape == (small.B, small.H, small.S, small.D)
    lens = a["src_len"]
    assert lens.dtype == np.int32
    if small.fixed_lens:   # the tiny config's lengths are given, 64 and 40
        assert lens.tolist() == list(small.fixed_lens)
    else:
        assert np.all(lens >= small.len_lo) and np.all(lens <= small.len_hi) and np.all(lens <= small.S)
    for bb, L in enumerate(lens):   # padding rows are zero
        assert not np.any(a["K"][bb, :, L:]) and not np.any(a["V"][bb, :, L:])
    r1 = workloads.attn_inputs(small, rep=1)   # a rotation set: new K/V, same q and lengths
    np.testing.assert_array_equal(r1["q"], a["q"])
    np.testing.assert_array_equal(r1["src_len"], lens)
    assert not np.array_equal(r1["K"], a["K"])


def test_the_bart_config_is_the_papers_shape():
    cfg = workloads.get("bart")
    assert (cfg.B, cfg.k, cfg.H, cfg.D, cfg.S) == (32, 4, 16, 64, 1024)
    assert (cfg.len_lo, cfg.len_hi, cfg.t, cfg.V, cfg.n, cfg.dtype) == (400, 1024, 140, 50264, 3, "bf16")
    lens = workloads.source_lengths(cfg)
    assert lens.shape == (32,) and lens.min() >= 400 and lens.max() <= 1024


# ---- algorithmic bytes ---------------------------------------------------------

def test_attention_bytes_count_valid_rows_queries_and_lengths():
    cfg = workloads.get("bart")
    lens = np.array([400, 1024, 0, 777] + [512] * 28, np.int32)
    want = 0
    for L in lens:                                   # K and V rows of every head
        want += 2 * int(L) * cfg.H * cfg.D * 2
    want += 2 * cfg.B * cfg.k * cfg.H * cfg.D * 2    # q and out
    want += 4 * cfg.B                                # src_len
    assert bench.attn_bytes(cfg, lens) == want


def test_reorder_bytes_against_a_brute_force_count():
    rng = np.random.default_rng(4)
    for k in (1, 2, 4, 5):
        parent = rng.integers(-1, k + 1, size=6 * k)
        reads = writes = 0
        for src in range(6):
            p = parent[src * k:(src + 1) * k]
            moved = [j for j in range(k) if 0 <= p[j] < k and p[j] != j]
            writes += len(moved)
            reads += len({int(p[j]) for j in moved})
        assert bench.reorder_bytes(parent, k, 100, tensors=2) == (reads + writes) * 100 * 2
    ident = np.tile(np.arange(4), 3)
    assert bench.reorder_bytes(ident, 4, 100) == 0


def test_select_and_ngram_bytes():
    assert bench.select_bytes(128, 50264, 140, 32, 8) == 128 * 50264 * 4 + 128 * 140 * 4 + 128 * 4 + 32 * 8 * 12
    assert bench.ngram_bytes(128, 140, 7) == 128 * 140 * 4 + 7 * 4


# ---- the benchmark's contract -----------------------------------------------------

def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_figures_are_used_only_for_the_measured_sources(tmp_path):
    sha = bench.kernel_source_sha()
    p = tmp_path / "traffic.json"
    p.write_text(json.dumps({"bart": {"kernel_source_sha": sha, "bytes_per_launch": 123},
                             "gpt2": {"kernel_source_sha": "0" * 16, "bytes_per_launch": 456}}))
    assert bench.load_traffic(str(p), "bart") == 123
    assert bench.load_traffic(str(p), "gpt2") is None          # taken on other sources
    assert bench.load_traffic(str(p), "t5") is None            # never taken
    assert bench.load_traffic(str(tmp_path / "missing.json"), "bart") is None

