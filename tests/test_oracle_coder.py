"""Pins of the oracle's arithmetic coder (CacheGen Sec. 5.2 "Arithmetic coding" step), checked
against facts that do not come from the oracle itself: hand-worked streams, Kraft's
inequality and distinctness over every short sequence, and the Shannon bound."""
import itertools
import math

import numpy as np
import pytest

import oracle
from conftest import golden_rows


def three_symbol_table(f0, f1, f2):
    """A 255-symbol cumulative table whose only non-empty symbols are 252, 253, 254."""
    assert f0 + f1 + f2 == 65536
    t = np.zeros(256, np.uint16)
    t[253] = f0
    t[254] = f0 + f1
    return t


TABLES = {"A": three_symbol_table(32768, 16384, 16384),
          "B": three_symbol_table(16384, 32768, 16384)}


@pytest.mark.parametrize("row", golden_rows("ac_hand_streams.txt"), ids=lambda r: "_".join(r))
def test_hand_worked_streams(row):
    table, syms, nbits, word = row
    seq = [] if syms == "-" else [int(s) for s in syms.split("_")]
    words, bits = oracle.ac_encode(seq, TABLES[table])
    assert bits == int(nbits)
    assert len(words) == 1 and int(words[0]) == int(word, 16)
    assert list(oracle.ac_decode(words, len(seq), TABLES[table])) == seq


BRUTE = {"dyadic": (32768, 16384, 16384), "near_uniform": (21846, 21845, 21845),
         "extreme": (65534, 1, 1)}


def _bitstring(words, nbits):
    return "".join(format(int(w), "032b") for w in words)[:nbits]


@pytest.mark.parametrize("name", list(BRUTE))
def test_brute_force_short_sequences(name):
    freqs = BRUTE[name]
    table = three_symbol_table(*freqs)
    p = [f / 65536 for f in freqs]
    for n in range(0, 7):
        codes = set()
        kraft = 0.0
        for seq in itertools.product(range(3), repeat=n):
            sym = [252 + s for s in seq]
            words, bits = oracle.ac_encode(sym, table)
            # round trip
            assert list(oracle.ac_decode(words, n, table)) == sym
            # within 2 bits (plus the per-symbol truncation loss) of the model's ideal length
            ideal = -sum(math.log2(p[s]) for s in seq)
            assert bits <= ideal + 2 + 1e-4 * n + 1e-9, (seq, bits, ideal)
            code = _bitstring(words, bits)
            codes.add(code)
            kraft += 2.0 ** (-bits)
        # distinct sequences of one length give distinct, prefix-free codewords
        assert len(codes) == 3 ** n
        for a in codes:
            for b in codes:
                if a != b:
                    assert not b.startswith(a)
        assert kraft <= 1.0 + 1e-12


def test_random_full_alphabet_shannon_and_round_trip():
    rng = np.random.default_rng(123)
    for trial in range(20):
        counts = rng.integers(0, 50, size=255) * (rng.random(255) < 0.3)
        table = oracle.normalize(counts)
        c32 = oracle.cum32(table)
        freq = np.diff(c32.astype(np.int64))
        assert freq.min() >= 1 and c32[255] == 65536
        n = int(rng.integers(1, 3000))
        sym = rng.choice(255, size=n, p=freq / 65536.0).astype(np.uint8)
        words, bits = oracle.ac_encode(sym, table)
        ideal = float(-np.log2(freq[sym] / 65536.0).sum())
        assert ideal - 1e-6 <= bits + 1e-9            # no code beats the model's information
        assert bits <= ideal + 2 + 1e-4 * n           # and WNC stays within 2 bits of it
        out = oracle.ac_decode(words, n, table)
        assert np.array_equal(out, sym)


def test_worst_case_bound_all_rare_symbols():
    """Symbols of frequency 1 cost at most 18 shifts each: the encoder's slot bound."""
    counts = np.zeros(255, np.int64)
    counts[127] = 10**9
    table = oracle.normalize(counts)
    n = 400
    sym = np.array([0, 254] * (n // 2), np.uint8)
    words, bits = oracle.ac_encode(sym, table)
    assert bits <= 18 * n + 2
    assert bits >= 16 * n - 1
    assert np.array_equal(oracle.ac_decode(words, n, table), sym)


def test_zero_fill_past_end_and_truncation():
    """Decoding reads zeros past the stream end; the coder's termination makes the stored
    words alone sufficient (the padding bits and beyond are irrelevant)."""
    rng = np.random.default_rng(7)
    counts = rng.integers(1, 100, size=255)
    table = oracle.normalize(counts)
    sym = rng.integers(0, 255, size=500).astype(np.uint8)
    words, bits = oracle.ac_encode(sym, table)
    padded = np.concatenate([words, rng.integers(0, 2**32, size=3, dtype=np.uint32)])
    # garbage after the last word must not matter when the decoder is told the length
    assert np.array_equal(oracle.ac_decode(words, 500, table), sym)
    # and garbage following the codeword's last bit must not matter either
    tail_bits = len(words) * 32 - bits
    w2 = words.copy()
    if tail_bits > 0:
        w2[-1] |= np.uint32((1 << tail_bits) - 1)
    assert np.array_equal(oracle.ac_decode(w2, 500, table), sym)
    assert np.array_equal(oracle.ac_decode(padded, 500, table), sym)


def test_per_symbol_tables_switch():
    """Anchor and delta positions use different tables inside one stream."""
    rng = np.random.default_rng(9)
    ta = oracle.normalize(rng.integers(0, 20, size=255))
    cd = np.zeros(255, np.int64)
    cd[120:135] = rng.integers(1, 1000, size=15)
    td = oracle.normalize(cd)
    n = 257
    tabs = [ta if j % 10 == 0 else td for j in range(n)]
    sym = np.array([rng.integers(0, 255) if j % 10 == 0 else rng.integers(120, 135)
                    for j in range(n)], np.uint8)
    words, bits = oracle.ac_encode(sym, tabs)
    assert np.array_equal(oracle.ac_decode(words, n, tabs), sym)
    ideal = sum(-math.log2((int(oracle.cum32(t)[s + 1]) - int(oracle.cum32(t)[s])) / 65536)
                for t, s in zip(tabs, sym))
    assert bits <= ideal + 2 + 1e-4 * n
