"""Pins for the oracle's post-processing of finished hypotheses (Section
4.3): byte-level detokenisation, one line per row up to the end-of-sequence
id.  Checked against a hand-worked example, the byte alphabet's hand values,
and a round trip from bytes through a tokenisation back to the same bytes.
"""
import numpy as np
from hypothesis import given, settings, strategies as st

import oracle
from paper_2106_04718_amd import workloads


def test_hand_example():
    # 'G'+dot-above (U+0120) is the symbol of the space byte 0x20, the 33rd
    # byte that is not printable (0x00..0x20), so it is 0x100 + 32
    vocab = ["ab", "Ġc", "xĀy", "</s>"]
    tokens = np.array([[0, 1, 3, 2], [2, 9, -1, 0], [3, 0, 0, 0]], np.int32)
    assert oracle.detokenize(tokens, vocab, eos=3) == b"ab c\nx\x00yab\n\n"


def test_alphabet_hand_values():
    table = oracle._symbol_bytes()
    assert len(table) == 256 and sorted(table.values()) == list(range(256))
    assert table[0x41] == 0x41 and table[0xFF] == 0xFF and table[0xA1] == 0xA1
    assert table[0x100] == 0x00 and table[0x120] == 0x20       # 33 bytes 0x00..0x20 first
    assert table[0x121] == 0x7F and table[0x142] == 0xA0       # then 0x7F..0xA0 (34 bytes)
    assert table[0x143] == 0xAD                                # then 0xAD, the last one
    assert 0x144 not in table and 0x20 not in table


@settings(max_examples=150, deadline=None)
@given(data=st.binary(min_size=0, max_size=200), cuts=st.lists(st.integers(1, 7), min_size=1, max_size=60))
def test_round_trip_from_bytes(data, cuts):
    # tokenise the bytes into pieces, write each piece in the byte alphabet,
    # and detokenise: the bytes come back (no newline inside the data)
    data = data.replace(b"\n", b"n")
    pieces, i, c = [], 0, 0
    while i < len(data):
        n = cuts[c % len(cuts)]
        pieces.append(data[i:i + n])
        i, c = i + n, c + 1
    vocab = sorted(set(pieces)) + [b"</s>"]
    sym = [workloads._SYMBOLS[b] for b in range(256)]
    vstr = ["".join(sym[b] for b in p) for p in vocab[:-1]] + ["</s>"]
    ids = [vocab.index(p) for p in pieces]
    eos = len(vocab) - 1
    row = np.array([ids + [eos, 0, 1]], np.int32)
    assert oracle.detokenize(row, vstr, eos) == data + b"\n"


def test_rows_end_at_their_first_eos_and_skip_unknown_ids():
    vocab = ["a", "b", "c"]
    tok = np.array([[0, 5, 1, 2, 0], [2, 2, 2, 2, 2], [-3, 0, 1, 0, 1]], np.int32)
    assert oracle.detokenize(tok, vocab, eos=2) == b"ab\n\nabab\n"
    assert oracle.detokenize(np.zeros((0, 4), np.int32), vocab, eos=2) == b""


def test_synthetic_vocabulary_is_made_of_the_alphabet():
    vocab = workloads.byte_vocab(2000, seed=3)
    table = oracle._symbol_bytes()
    assert vocab[-1] == "</s>" and len(vocab) == 2000
    assert all(len(s) >= 1 and all(ord(ch) in table for ch in s) for s in vocab[:-1])
    data, off = workloads.vocab_utf8(vocab)
    assert off[0] == 0 and off[-1] == len(data) and np.all(np.diff(off) >= 1)
