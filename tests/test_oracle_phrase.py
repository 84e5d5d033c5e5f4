"""Pins of the oracle's container version 2 (tile order, phrase alphabet,
rANS at M = 2^16): hand-worked cases, closed-form coder chains, properties
that determine the greedy parse uniquely, brute-force round trips and the
code-length bound.  These are checked against what the definitions fix,
not against a second copy of the oracle's code."""
import itertools
import math

import numpy as np
import pytest

import oracle
import synth
from synth.configs import small_spec


def le(codes):
    v = 0
    for i, c in enumerate(codes):
        v |= int(c) << (8 * i)
    return v


# ---- frequency normalisation ----

def test_freq_norm_worked_and_invariants():
    # 3:1 over 2^10 slots splits exactly
    assert list(oracle.freq_norm([3, 1], 10)) == [768, 256]
    # floor(c * 1024 / 7) = 146, 292, 585 (sum 1023) with remainders 2, 4, 1:
    # the one missing slot goes to the largest remainder
    assert list(oracle.freq_norm([1, 2, 4], 10)) == [146, 293, 585]
    # excess: 1000 symbols of count 1 and one large at R = 10: every f clamped
    # to 1 (1000 slots), the large one gets the rest
    f = oracle.freq_norm([1] * 1000 + [10**9], 10)
    assert f[-1] == 24 and (f[:-1] == 1).all()
    r = np.random.default_rng(1)
    for _ in range(50):
        n = int(r.integers(1, 300))
        c = r.integers(1, 10**6, size=n) ** r.integers(1, 3, size=n)
        f = oracle.freq_norm(c, 12)
        assert f.sum() == 4096 and (f >= 1).all()
        # each share within one slot of proportional, unless clamped at 1 or reduced
        prop = c / c.sum() * 4096
        assert (f <= np.floor(prop) + 1 + (f == 1)).all()
    # agrees with the byte-alphabet rule of version 1 on byte histograms
    counts = np.zeros(256, dtype=np.uint64)
    counts[[0, 3, 200, 255]] = [1000, 7, 1, 50000]
    sym, freq = oracle.freq_table(counts, 12)
    assert np.array_equal(oracle.freq_norm(counts[sym], 12), freq)
    with pytest.raises(ValueError):
        oracle.freq_norm([1, 0, 2], 12)  # a symbol that never occurs
    with pytest.raises(ValueError):
        oracle.freq_norm(np.ones(4097), 12)  # more symbols than slots


def test_tile_geometry():
    # 300 x 1000 in 64 x 256 tiles: 5 x 4 tiles, the last ones cut
    assert oracle.tile_geometry(300, 1000, 64, 256, 0) == (0, 0, 64, 256)
    assert oracle.tile_geometry(300, 1000, 64, 256, 3) == (0, 768, 64, 232)
    assert oracle.tile_geometry(300, 1000, 64, 256, 4) == (64, 0, 64, 256)
    assert oracle.tile_geometry(300, 1000, 64, 256, 19) == (256, 768, 44, 232)


# ---- parse ----

DQ = sorted([le([1, 2, 3, 4]), le([0, 0, 0, 0])])
DP = sorted([le([5, 6]), le([0, 0])])


def expand(tokens, quads, pairs, singles):
    out = []
    for t in tokens:
        if t < len(quads):
            out += [(quads[t] >> (8 * e)) & 255 for e in range(4)]
        elif t < len(quads) + len(pairs):
            v = pairs[t - len(quads)]
            out += [v & 255, v >> 8]
        else:
            out.append(int(singles[t - len(quads) - len(pairs)]))
    return out


def test_parse_worked_example():
    singles = np.array([1, 5, 7, 9], dtype=np.uint8)
    u = [9, 1, 2, 3, 4, 5, 6, 7, 0, 0, 0, 0, 0, 0, 5]
    t = oracle.phrase_parse(np.array(u, dtype=np.uint8), DQ, DP, singles)
    # single 9; quad 1234 (at position 1: the parse is not bound to block
    # positions); pair 56; single 7; quad 0000; pair 00; single 5 (at the end a
    # quad or pair does not fit)
    nq, np_ = len(DQ), len(DP)
    s = {c: nq + np_ + i for i, c in enumerate(singles)}
    assert list(t) == [s[9], DQ.index(le([1, 2, 3, 4])), nq + DP.index(le([5, 6])), s[7],
                       DQ.index(0), nq + DP.index(0), s[5]]
    assert expand(t, DQ, DP, singles) == u
    with pytest.raises(ValueError):  # 8 is neither in a phrase nor a single
        oracle.phrase_parse(np.array([8], dtype=np.uint8), DQ, DP, singles)


def test_parse_is_the_greedy_parse():
    """The token sequence reproduces the segment, and at every token start the
    longest phrase that starts there and is in the dictionary was taken --
    properties that fix the greedy parse uniquely."""
    r = np.random.default_rng(7)
    for trial in range(200):
        K = int(r.integers(1, 5))
        u = r.integers(0, K, size=int(r.integers(1, 40))).astype(np.uint8)
        quads = sorted({le(r.integers(0, K, size=4)) for _ in range(int(r.integers(0, 6)))})
        pairs = sorted({le(r.integers(0, K, size=2)) for _ in range(int(r.integers(0, 5)))})
        singles = np.arange(K, dtype=np.uint8)
        t = oracle.phrase_parse(u, quads, pairs, singles)
        assert expand(t, quads, pairs, singles) == list(u)
        j = 0
        for tok in t:
            q_here = j + 4 <= len(u) and le(u[j:j + 4]) in quads
            p_here = j + 2 <= len(u) and le(u[j:j + 2]) in pairs
            if tok < len(quads):
                j += 4
            elif tok < len(quads) + len(pairs):
                assert not q_here
                j += 2
            else:
                assert not q_here and not p_here
                j += 1


# ---- dictionary rule ----

def test_dictionary_share_rule_and_caps():
    """R = 10: a quad enters DQ when count * 2^12 >= tau * blocks.  One row of
    65536 codes in 64-column tiles has 16384 blocks: a quad seen 4 times
    passes at tau = 1 (4 * 4096 = 16384) and fails at tau = 2; one seen 3
    times fails.  Pairs use tau = 1 over the 32768 pairs: 8 are needed."""
    N = 65536
    q = np.full((1, N), 9, dtype=np.uint8)  # filler quad 9999 (and pair 99)
    A, B = [1, 2, 3, 4], [4, 3, 2, 1]
    for blk in (0, 100, 200, 300):
        q[0, 4 * blk:4 * blk + 4] = A
    for blk in (400, 500, 600):
        q[0, 4 * blk:4 * blk + 4] = B
    # pair 77 eight times, pair 88 seven times, at even positions inside blocks of
    # (7, 7, 9, 9) / (8, 8, 9, 9) so the quads stay rare
    for i in range(8):
        q[0, 4 * (1000 + i):4 * (1000 + i) + 2] = 7
    for i in range(7):
        q[0, 4 * (2000 + i):4 * (2000 + i) + 2] = 8
    quads, pairs = oracle.phrase_dict(q, 64, 64, R=10, tau=1)
    assert le(A) in quads and le(B) not in quads and le([9] * 4) in quads
    assert le([7, 7]) in pairs and le([8, 8]) not in pairs and le([9, 9]) in pairs
    quads2, _ = oracle.phrase_dict(q, 64, 64, R=10, tau=2)
    assert le(A) not in quads2 and le([9] * 4) in quads2
    assert list(quads) == sorted(quads) and list(pairs) == sorted(pairs)
    # cap: 2^(R-1) = 512 quads at most, the most frequent kept (ties: lower value)
    r = np.random.default_rng(3)
    q = r.integers(0, 7, size=(64, 4096)).astype(np.uint8)  # 7^4 = 2401 candidates
    quads, pairs = oracle.phrase_dict(q, 64, 256, R=10, tau=1)
    assert len(quads) == 512 and len(pairs) <= 256
    blocks = q.reshape(-1, 4)
    vals, cnt = np.unique([le(b) for b in blocks], return_counts=True)
    order = sorted(zip(-cnt, vals))[:512]
    assert sorted(v for _, v in order) == list(quads)


# ---- rANS at M = 2^16 ----

def test_prans_closed_form_chain():
    """One state, three symbols of frequency 1 (F = 16 at R = 12, slot
    offsets c1, c2, c3): each step consumes 12 bits, so the encoder pushes the
    low word twice and the final state is 2^20 + c1, with words [c2, c3]."""
    freq = np.array([1, 1, 4094], dtype=np.uint16)  # CUM = 0, 16, 32
    seq = [1, 0, 1]
    c = [16 * 1, 0, 16 * 1]
    words, states = oracle.prans_encode([seq], freq, 12)
    assert states[0] == (1 << 20) + c[0]
    assert list(words) == [c[1], c[2]]
    rc, out = oracle.prans_decode(words, states, [3], freq, np.array([1, 1, 1], np.uint8), 12)
    assert rc == oracle.OK and list(out[0]) == seq


def test_prans_single_symbol_costs_nothing():
    freq = np.array([4096], dtype=np.uint16)
    words, states = oracle.prans_encode([[0] * 50, [0] * 3, []], freq, 12)
    assert words.size == 0 and (states == 65536).all()
    rc, out = oracle.prans_decode(words, states, [200, 12, 0], freq, np.array([4], np.uint8), 12)
    assert rc == oracle.OK and [len(o) for o in out] == [50, 3, 0]


def test_prans_brute_force_round_trip():
    """Every sequence of length <= 5 over 3 symbols, on one state and beside
    other states of different lengths: exact round trip, terminal states."""
    freq = np.array([3000, 1000, 96], dtype=np.uint16)
    plen = np.array([1, 2, 4], dtype=np.uint8)
    r = np.random.default_rng(11)
    for n in range(6):
        for seq in itertools.product(range(3), repeat=n):
            others = [list(r.integers(0, 3, size=int(r.integers(0, 7)))) for _ in range(3)]
            toks = [list(seq)] + others
            words, states = oracle.prans_encode(toks, freq, 12)
            need = [int(sum(plen[t] for t in s)) for s in toks]
            rc, out = oracle.prans_decode(words, states, need, freq, plen, 12)
            assert rc == oracle.OK
            assert [list(o) for o in out] == toks


def test_prans_code_length_bound():
    """Words used vs I = sum log2(2^16 / F): each step changes log2 x by
    log2(2^16 / F) up to a factor (1 +- F / x), F / x <= 2^-4 ... bounded
    by n log2(1 + 2^-4) in the worst case; in practice within 1%, plus the
    final states (32 bits each)."""
    r = np.random.default_rng(5)
    freq = np.array([2048, 1024, 512, 256, 128, 64, 32, 16, 8, 4, 2, 1, 1], dtype=np.uint16)
    p = freq / freq.sum()
    toks = [list(r.choice(len(freq), size=int(r.integers(2000, 3000)), p=p)) for _ in range(64)]
    words, states = oracle.prans_encode(toks, freq, 12)
    info = sum(math.log2(4096 / freq[t]) for s in toks for t in s)
    bits = 16 * words.size + 32 * len(toks)
    n = sum(len(s) for s in toks)
    assert abs(bits - info) <= n * math.log2(1 + 2 ** -4) + 32 * len(toks) + 16
    assert abs(16 * words.size - info) <= 0.01 * info + 32 * len(toks)


def test_prans_corruption_detected():
    freq = np.array([3000, 1000, 96], dtype=np.uint16)
    plen = np.array([1, 1, 1], dtype=np.uint8)
    r = np.random.default_rng(2)
    toks = [list(r.integers(0, 3, size=300)) for _ in range(4)]
    words, states = oracle.prans_encode(toks, freq, 12)
    need = [len(s) for s in toks]
    flagged = 0
    for trial in range(20):
        bad = words.copy()
        bad[int(r.integers(bad.size))] ^= np.uint16(1 << int(r.integers(16)))
        rc, out = oracle.prans_decode(bad, states, need, freq, plen, 12)
        if rc == oracle.ECORRUPT:
            flagged += 1
        else:
            assert [list(o) for o in out] == toks
    assert flagged >= 15
    rc, _ = oracle.prans_decode(words[:-1], states, need, freq, plen, 12)
    assert rc == oracle.ECORRUPT


# ---- container version 2 ----

SHAPES = [
    # M, N, TR, TC
    (300, 1000, 64, 256),   # ragged in both directions
    (37, 1283, 128, 64),    # fewer rows than a tile; N not a multiple of 4
    (5, 7, 64, 4),
    (1, 1, 64, 4),          # a single code
    (64, 4096, 64, 64),
    (3, 13, 256, 8),
]


@pytest.mark.parametrize("M,N,TR,TC", SHAPES)
def test_container2_round_trip(M, N, TR, TC):
    w = synth.weights(small_spec(M, N, seed=M * 31 + N))
    alpha, _ = oracle.alpha_search(w, 2.5)
    blob = oracle.container2_build(w, alpha, TR, TC)
    info = oracle.container2_info(blob)
    assert info.n_chunks == ((M + TR - 1) // TR) * ((N + TC - 1) // TC)
    rc, q = oracle.container2_decode(blob)
    assert rc == oracle.OK
    assert np.array_equal(q, oracle.quantize(w, oracle.container_scales(blob)))
    for c in range(info.n_chunks):
        rc, t = oracle.container2_decode_chunk(blob, c)
        r0, c0, rows, cols = oracle.tile_geometry(M, N, TR, TC, c)
        assert rc == oracle.OK and np.array_equal(t, q[r0:r0 + rows, c0:c0 + cols])
    rc, qp = oracle.container2_decode_par(blob)
    assert rc == oracle.OK and np.array_equal(qp, q)


def test_container2_single_phrase():
    """An all-zero matrix: one phrase (the zero quad) of frequency 2^R: no
    words, every state stays at 2^16."""
    w = np.zeros((70, 512), dtype=np.uint16)
    blob = oracle.container2_build(w, 1.0, 64, 256)
    info = oracle.container2_info(blob)
    assert (info.n_quads, info.n_pairs, info.n_singles, info.total_words) == (1, 0, 0, 0)
    states = np.frombuffer(blob[info.off_chunk_state:info.off_chunk_state + 4 * 64 *
                                info.n_chunks].tobytes(), dtype=np.uint32)
    assert (states == 65536).all()
    rc, q = oracle.container2_decode(blob)
    assert rc == oracle.OK and not q.any()


def test_container2_chooses_the_cheapest_alphabet():
    """tau is the one of 8, 4, 2, 1 whose alphabet needs the fewest bits,
    sum count * log2(2^R / f), recomputed here from the dictionary, the
    greedy parse and the normalisation."""
    w = synth.weights(small_spec(128, 2048, seed=4))
    alpha, _ = oracle.alpha_search(w, 2.0)
    blob = oracle.container2_build(w, alpha, 64, 256)
    info = oracle.container2_info(blob)
    q = oracle.quantize(w, oracle.container_scales(blob))
    costs = {}
    for tau in (8, 4, 2, 1):
        quads, pairs = oracle.phrase_dict(q, 64, 256, 12, tau)
        toks = []
        allsingles = np.arange(256, dtype=np.uint8)
        for c in range(info.n_chunks):
            r0, c0, rows, cols = oracle.tile_geometry(128, 2048, 64, 256, c)
            for s in range(rows):
                toks.append(oracle.phrase_parse(q[r0 + s, c0:c0 + cols], quads, pairs, allsingles))
        toks = np.concatenate(toks)
        _, cnt = np.unique(toks, return_counts=True)
        # alphabet order: used quads, used pairs, used singles = ascending token index
        f = oracle.freq_norm(cnt, 12)
        costs[tau] = float(np.sum(cnt * np.log2(4096.0 / f)))
    best = min(costs, key=lambda t: (costs[t], -t))
    assert info.tau == best, costs
    assert abs(16 * info.total_words - costs[best]) <= 0.01 * costs[best] + 32 * 64 * info.n_chunks


def test_container2_coded_size_near_entropy():
    """Payload bits per code of a 2-bit config-like layer: above what the
    symbol statistics allow minus the state bits, within 5% of the empirical
    entropy of the codes (the phrase alphabet cannot use all of the order-0
    statistics; measured 1-3% on the synthetic configurations)."""
    w = synth.weights(small_spec(512, 4096, seed=6))
    alpha, h = oracle.alpha_search(w, 2.0)
    blob = oracle.container2_build(w, alpha, 64, 256)
    info = oracle.container2_info(blob)
    payload = 16 * info.total_words / w.size
    assert 0.9 * info.entropy_bits <= payload <= 1.05 * info.entropy_bits


def test_container2_int8_and_header_checks():
    w = synth.weights(small_spec(40, 640, seed=9))
    alpha, _ = oracle.alpha_search(w, 2.0, oracle.INT8)
    blob = oracle.container2_build(w, alpha, 64, 128, fmt=oracle.INT8)
    info = oracle.container2_info(blob)
    assert info.base_format == oracle.INT8
    rc, q = oracle.container2_decode(blob)
    assert rc == oracle.OK
    assert np.array_equal(q, oracle.quantize(w, oracle.container_scales(blob), oracle.INT8))
    for off, val in ((4, 3), (36, 9), (84, 6), (32, 96), (40, info.n_syms + 1)):
        bad = blob.copy()
        bad[off:off + 4] = np.frombuffer(np.uint32(val).tobytes(), dtype=np.uint8)
        with pytest.raises(ValueError):
            oracle.container2_info(bad)
    with pytest.raises(ValueError):
        oracle.container2_build(w, alpha, 96, 128)   # tile rows not 64/128/256
    with pytest.raises(ValueError):
        oracle.container2_build(w, alpha, 64, 126)   # tile columns not a multiple of 4


# ---- row order (eq_phrase.c, item 4) ----

def _row_costs(blob, q):
    """Phrases of each matrix row's greedy parse, summed over its tile
    segments: a plain loop over the container's dictionary (quads first,
    then pairs, then the single code)."""
    info = oracle.container2_info(blob)
    codes, plen, _ = oracle.container2_phrases(blob)
    quads = {tuple(int(v) for v in codes[k][:4]) for k in range(len(plen)) if plen[k] == 4}
    pairs = {tuple(int(v) for v in codes[k][:2]) for k in range(len(plen)) if plen[k] == 2}
    M, N = q.shape
    TC = info.tile_cols
    cost = []
    for r in range(M):
        n = 0
        for c0 in range(0, N, TC):
            u = [int(v) for v in q[r, c0:c0 + TC]]
            j = 0
            while j < len(u):
                if j + 4 <= len(u) and tuple(u[j:j + 4]) in quads:
                    j += 4
                elif j + 2 <= len(u) and tuple(u[j:j + 2]) in pairs:
                    j += 2
                else:
                    j += 1
                n += 1
        cost.append(n)
    return np.array(cost)


@pytest.mark.parametrize("M,N,TR,TC", SHAPES)
def test_container2_row_order_round_trip(M, N, TR, TC):
    """Tiles cut over the rows in their stored order: every tile's codes are
    the stored rows' codes, and the whole decode is the quantised matrix."""
    w = synth.weights(small_spec(M, N, seed=M * 31 + N))
    alpha, _ = oracle.alpha_search(w, 2.5)
    blob = oracle.container2_build(w, alpha, TR, TC, row_order=True)
    info = oracle.container2_info(blob)
    assert info.flags == 1
    order = oracle.container2_row_order(blob)
    assert sorted(order.tolist()) == list(range(M))
    rc, q = oracle.container2_decode(blob)
    assert rc == oracle.OK
    assert np.array_equal(q, oracle.quantize(w, oracle.container_scales(blob)))
    for c in range(info.n_chunks):
        rc, t = oracle.container2_decode_chunk(blob, c)
        r0, c0, rows, cols = oracle.tile_geometry(M, N, TR, TC, c)
        assert rc == oracle.OK and np.array_equal(t, q[order[r0:r0 + rows], c0:c0 + cols])
    rc, qp = oracle.container2_decode_par(blob)
    assert rc == oracle.OK and np.array_equal(qp, q)


def test_container2_row_order_sorts_by_phrase_count():
    """The stored order is the rows by ascending phrase count, ties by lower
    row index, with the counts from a plain greedy parse; rows of very
    different code ranges (a few near-zero rows, a few with a large scale)
    make the order far from the identity."""
    M, N = 300, 1024
    w = synth.weights(small_spec(M, N, seed=12)).copy()
    w[::7] = 0                                      # all-zero rows: the cheapest
    w[3::11, 5] = np.uint16(0x4480)                 # one large weight: codes near zero
    alpha, _ = oracle.alpha_search(w, 2.0)
    blob = oracle.container2_build(w, alpha, 64, 256, row_order=True)
    rc, q = oracle.container2_decode(blob)
    assert rc == oracle.OK
    cost = _row_costs(blob, q)
    assert len(set(cost.tolist())) > 10
    want = sorted(range(M), key=lambda r: (cost[r], r))
    order = oracle.container2_row_order(blob)
    assert order.tolist() == want
    assert cost[order[0]] == N // 4                # an all-zero row: zero quads only


def _sections(blob):
    info = oracle.container2_info(blob)
    n_st = 4 * info.n_chunks * info.lanes
    return {
        "phr": blob[info.off_phr:info.off_phr + 4 * info.n_syms].tobytes(),
        "freq": blob[info.off_freq:info.off_freq + 2 * info.n_syms].tobytes(),
        "off": blob[info.off_chunk_off:info.off_chunk_off + 4 * (info.n_chunks + 1)].tobytes(),
        "state": blob[info.off_chunk_state:info.off_chunk_state + n_st].tobytes(),
        "words": blob[info.off_words:info.off_words + 2 * info.total_words].tobytes(),
        "tau": info.tau,
    }


def test_container2_row_order_is_the_row_permuted_container():
    """With a row order, the container codes exactly the row-permuted
    matrix: alphabet, chunk offsets, states and words equal those of the
    matrix-order container of w[order] (with its scales permuted alike),
    and the scales stay in matrix order."""
    w = synth.weights(small_spec(200, 520, seed=21)).copy()
    w[::5] = 0
    alpha, _ = oracle.alpha_search(w, 2.0)
    blob = oracle.container2_build(w, alpha, 64, 128, row_order=True)
    order = oracle.container2_row_order(blob)
    scale = oracle.container_scales(blob)
    assert np.array_equal(scale, oracle.row_scales(w, alpha))
    ref = oracle.container2_build(w[order], 0.0, 64, 128, scale=scale[order])
    assert oracle.container2_info(ref).flags == 0
    assert _sections(blob) == _sections(ref)


def test_container2_row_order_checks():
    """A damaged order section (a repeated row, a row out of range), an
    unknown flag, or an order offset without the flag is refused."""
    w = synth.weights(small_spec(70, 256, seed=3))
    alpha, _ = oracle.alpha_search(w, 2.0)
    blob = oracle.container2_build(w, alpha, 64, 128, row_order=True)
    info = oracle.container2_info(blob)
    o = info.off_order
    for k, val in ((1, int(oracle.container2_row_order(blob)[0])), (5, 70)):
        bad = blob.copy()
        bad[o + 4 * k:o + 4 * k + 4] = np.frombuffer(np.uint32(val).tobytes(), dtype=np.uint8)
        with pytest.raises(ValueError):
            oracle.container2_info(bad)
    bad = blob.copy()
    bad[44:48] = np.frombuffer(np.uint32(3).tobytes(), dtype=np.uint8)
    with pytest.raises(ValueError):
        oracle.container2_info(bad)
    bad = blob.copy()
    bad[44:48] = 0                                  # offset present, flag clear
    with pytest.raises(ValueError):
        oracle.container2_info(bad)
    plain = oracle.container2_build(w, alpha, 64, 128)
    assert oracle.container2_info(plain).off_order == 0
    assert np.array_equal(oracle.container2_row_order(plain), np.arange(70))
