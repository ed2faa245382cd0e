"""GPU checks of the asynchronous post-processing (Section 4.3): the text a
PostProcessor writes while the GPU keeps working equals, byte for byte, the
synchronous detokenisation of the oracle, in submission order."""
import numpy as np
import pytest
import torch

import oracle
from paper_2106_04718_amd import api, workloads

from _gpu import device, say, to_dev

pytestmark = pytest.mark.gpu


def setup(name="bart", batches=5, V=None):
    cfg = workloads.get(name)
    V = V or cfg.V
    vocab = workloads.byte_vocab(V, seed=cfg.index)
    tok = workloads.finished_batches(cfg, batches, seed=1)
    tok = np.where(tok >= V - 1, tok % (V - 1), tok).astype(np.int32)   # a smaller vocabulary than the config's
    ends = np.random.default_rng(2).integers(cfg.t // 2, cfg.t + 1, size=tok.shape[:2])
    for b in range(tok.shape[0]):
        for r in range(tok.shape[1]):
            if ends[b, r] < cfg.t:
                tok[b, r, ends[b, r]] = V - 1
    return cfg, vocab, tok


@pytest.mark.parametrize("slots", [1, 2, 4])
def test_async_output_equals_synchronous_detokenisation(slots):
    device()
    cfg, vocab, tok = setup(batches=5, V=50264)
    eos = len(vocab) - 1
    say(f"[postproc] {tok.shape[0]} batches of {cfg.rows} rows, slots={slots}")
    work = torch.empty((2048, 2048), device="cuda")
    with api.PostProcessor(vocab, eos, cfg.rows, cfg.t, slots=slots) as pp:
        for b in range(tok.shape[0]):
            d = to_dev(tok[b])
            pp.submit(d)
            d.fill_(0)                       # later work on the stream must not reach the copy
            work.normal_()                   # and the GPU keeps busy meanwhile
            torch.mm(work, work)
        pp.flush()
        got = pp.output()
        busy = pp.busy_seconds()
    want = b"".join(oracle.detokenize(tok[b], vocab, eos) for b in range(tok.shape[0]))
    assert got == want
    assert got.count(b"\n") == tok.shape[0] * cfg.rows
    assert busy > 0.0


def test_file_output_and_leading_dimension(tmp_path):
    device()
    cfg, vocab, tok = setup("t5", batches=3, V=32128)
    eos = len(vocab) - 1
    path = tmp_path / "out.txt"
    wide = np.zeros((tok.shape[1], cfg.t + 37), np.int32)
    with api.PostProcessor(vocab, eos, cfg.rows, cfg.t, slots=2, path=str(path)) as pp:
        for b in range(tok.shape[0]):
            wide[:, :cfg.t] = tok[b]
            wide[:, cfg.t:] = 7              # columns past t are never read
            pp.submit(to_dev(wide), t=cfg.t)
        pp.flush()
    want = b"".join(oracle.detokenize(tok[b], vocab, eos) for b in range(tok.shape[0]))
    assert path.read_bytes() == want


def test_empty_batches_and_short_rows():
    device()
    vocab = ["a", "Ġb", "</s>"]
    with api.PostProcessor(vocab, 2, 4, 6, slots=2) as pp:
        pp.submit(torch.zeros((0, 6), dtype=torch.int32, device="cuda"))
        rows = np.array([[0, 1, 2, 0, 0, 0], [1, 1, 1, 1, 1, 1], [2, 0, 0, 0, 0, 0]], np.int32)
        pp.submit(to_dev(rows), t=6)
        pp.submit(to_dev(rows), t=0)
        pp.flush()
        assert pp.output() == oracle.detokenize(rows, vocab, 2) + b"\n\n\n"
