"""Oracle frequency table and interleaved rANS coder.

Pins: exact states and words of closed-form chains, brute-force losslessness
over every short sequence, the terminal invariant, the Gibbs inequality for
the normalised table, and the code length against the information content
sum(log2(2^P / f)) within rANS's rounding bound.
"""
import itertools
import math

import numpy as np
import pytest

import oracle


def _counts(d):
    c = np.zeros(256, dtype=np.uint64)
    for k, v in d.items():
        c[k] = v
    return c


def test_freq_table_sums_and_floors():
    r = np.random.default_rng(4)
    for P in (1, 4, 8, 12):
        for K in (1, 2, 3, 17, min(2 ** P, 200)):
            if K > 2 ** P:
                continue
            codes = r.choice(256, K, replace=False)
            c = np.zeros(256, dtype=np.uint64)
            c[codes] = r.integers(1, 10 ** 6, K)
            sym, freq = oracle.freq_table(c, P)
            assert list(sym) == sorted(codes)
            assert int(freq.astype(np.int64).sum()) == 2 ** P
            assert (freq >= 1).all()
            if K == 1:
                assert freq[0] == 2 ** P


def test_freq_table_rejects_more_symbols_than_slots():
    with pytest.raises(ValueError):
        oracle.freq_table(_counts({1: 5, 2: 5, 3: 5}), 1)


def test_freq_table_exact_when_proportional():
    sym, freq = oracle.freq_table(_counts({3: 300, 9: 100, 200: 600}), 10)
    # 1024 * (0.3, 0.1, 0.6) = 307.2, 102.4, 614.4 -> floors 307, 102, 614 (sum 1023).
    # Remainders are .2, .4, .4; codes 9 and 200 tie at .4 and the lower code
    # comes first, so the missing unit goes to code 9.
    assert list(sym) == [3, 9, 200]
    assert list(freq) == [307, 103, 614]


def test_freq_table_gibbs():
    r = np.random.default_rng(5)
    c = np.zeros(256, dtype=np.uint64)
    c[:40] = (1e6 * r.dirichlet(np.full(40, 0.3))).astype(np.uint64) + 1
    sym, freq = oracle.freq_table(c, 12)
    n = c.sum()
    p = c[sym] / n
    cost = -(p * np.log2(freq / 4096.0)).sum()          # bits/symbol under the table
    assert cost >= oracle.entropy_counts(c) - 1e-12       # Gibbs
    assert cost <= oracle.entropy_counts(c) + 0.02


def test_closed_form_chain_p12():
    """One symbol B with f = 1, cum = 2^P - 1 in every lane: each encode maps
    x -> (x + 1) 2^P - 1, and a word is pushed whenever x >= 2^(32-P).  From
    x = 2^16 with P = 12 and four steps per lane: x1 = 65537*4096 - 1 (no
    push), then three pushes of the low 16 bits (each 4095), ending at
    17*4096 - 1 = 69631."""
    sym = np.array([0x00, 0x38], dtype=np.uint8)
    freq = np.array([4095, 1], dtype=np.uint16)
    q = np.full(64 * 4, 0x38, dtype=np.uint8)
    words, states = oracle.rans_encode(q, 64, 12, sym, freq)
    assert (states == 69631).all()
    assert words.size == 3 * 64 and (words == 4095).all()
    rc, back = oracle.rans_decode(words, states, q.size, 64, 12, sym, freq)
    assert rc == oracle.OK and (back == q).all()


def test_closed_form_chain_p4_no_push_then_push():
    """P = 4: x -> 16(x+1) - 1 gives 1048591, 16777471, 268439551 (no push,
    all < 2^28); the fourth encode pushes 268439551 mod 2^16 = 4095 and
    continues from 4096 to 65551."""
    sym = np.array([0x10, 0x38], dtype=np.uint8)
    freq = np.array([15, 1], dtype=np.uint16)
    for T, st, nw in ((1, 1048591, 0), (2, 16777471, 0), (3, 268439551, 0), (4, 65551, 1)):
        q = np.full(64 * T, 0x38, dtype=np.uint8)
        words, states = oracle.rans_encode(q, 64, 4, sym, freq)
        assert (states == st).all() and words.size == 64 * nw
        assert (words == 4095).all()


def test_single_symbol_alphabet_costs_nothing():
    sym = np.array([0x00], dtype=np.uint8)
    freq = np.array([4096], dtype=np.uint16)
    q = np.zeros(4096 + 13, dtype=np.uint8)
    words, states = oracle.rans_encode(q, 64, 12, sym, freq)
    assert words.size == 0 and (states == 65536).all()
    rc, back = oracle.rans_decode(words, states, q.size, 64, 12, sym, freq)
    assert rc == oracle.OK and (back == 0).all()


@pytest.mark.parametrize("P,freqs", [(2, [1, 3]), (3, [5, 2, 1]), (12, [4000, 90, 6]),
                                     (12, [1, 1, 4094])])
def test_brute_force_short_sequences(P, freqs):
    sym = np.array([0x00, 0x38, 0xC5][: len(freqs)], dtype=np.uint8)
    freq = np.array(freqs, dtype=np.uint16)
    for n in range(1, 7):
        for seq in itertools.product(range(len(freqs)), repeat=n):
            q = sym[list(seq)]
            words, states = oracle.rans_encode(q, 64, P, sym, freq)
            rc, back = oracle.rans_decode(words, states, n, 64, P, sym, freq)
            assert rc == oracle.OK and (back == q).all(), (P, seq)


def _random_stream(r, n, K, skew=0.7):
    p = skew ** np.arange(K)
    p /= p.sum()
    codes = np.sort(r.choice(np.arange(1, 127), K, replace=False)).astype(np.uint8)
    return codes[r.choice(K, size=n, p=p)]


@pytest.mark.parametrize("lanes", [64, 128, 256])
@pytest.mark.parametrize("n", [1, 63, 64, 65, 4095, 4096, 4097, 20000])
def test_round_trip_and_code_length(lanes, n):
    r = np.random.default_rng(n * 7 + lanes)
    q = _random_stream(r, n, 23)
    counts = np.bincount(q, minlength=256).astype(np.uint64)
    P = 12
    sym, freq = oracle.freq_table(counts, P)
    words, states = oracle.rans_encode(q, lanes, P, sym, freq)
    rc, back = oracle.rans_decode(words, states, n, lanes, P, sym, freq)
    assert rc == oracle.OK and (back == q).all()
    # information content under the table vs. bits actually produced
    f = dict(zip(sym.tolist(), freq.tolist()))
    info = sum(math.log2(4096 / f[c]) for c in q.tolist())
    used = 16 * words.size + sum(math.log2(s / 65536.0) for s in states.tolist())
    slack = n * math.log2(1 + 2 ** (P - 16)) + 17 * min(n, lanes)
    assert abs(used - info) <= slack
    if n >= 4096:
        assert abs(used - info) <= 0.01 * info + 17 * lanes


def test_decode_detects_corruption():
    r = np.random.default_rng(9)
    q = _random_stream(r, 8192, 30)
    sym, freq = oracle.freq_table(np.bincount(q, minlength=256).astype(np.uint64), 12)
    words, states = oracle.rans_encode(q, 64, 12, sym, freq)
    for trial in range(40):
        bad = words.copy()
        k = r.integers(bad.size)
        bad[k] ^= np.uint16(1 << int(r.integers(16)))
        rc, back = oracle.rans_decode(bad, states, q.size, 64, 12, sym, freq)
        # ANS decoding is a bijection: a changed stream cannot reproduce the
        # symbols and pass the terminal check at the same time
        assert rc == oracle.ECORRUPT or not (back == q).all()
    rc, _ = oracle.rans_decode(words[:-1], states, q.size, 64, 12, sym, freq)
    assert rc == oracle.ECORRUPT
    st = states.copy()
    st[3] += 1
    rc, back = oracle.rans_decode(words, st, q.size, 64, 12, sym, freq)
    assert rc == oracle.ECORRUPT or not (back == q).all()
