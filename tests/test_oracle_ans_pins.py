"""Pins for the oracle's entropy coder on the exception section (Section
3.1: the changed exponents travel ANS-coded), each against something other
than the oracle's own code:
  - hand-worked quantisation cases and two hand-worked chunks
    (tests/golden/ans_chunk_*.txt), one with a renormalisation word;
  - closed forms: a one-symbol alphabet costs nothing (every state stays at
    L), and the section layout follows from E alone;
  - the information identity of range ANS: over a chunk,
    16 W + sum_l log2 x_l = 64 * 16 + sum_i log2(M / f_{s_i}) + drift, where
    each symbol's drift is below log2(1 + 1/16) (x >= 16 f before coding);
  - decode(encode(x)) == x for every length up to a chunk and for whole
    shards, with malformed sections rejected.
The stream layout itself (64 interleaved states, chunking, section order) is
a reading of the paper, which names nvCOMP's ANS without its format.
"""
import math
import os

import numpy as np
import pytest

from tests import ieee_ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
M, L = 4096, 65536


def _expand(tok):
    out = []
    for t in tok.split():
        if "*" in t:
            k, v = t.split("*")
            out += [int(v, 0)] * int(k)
        else:
            out.append(int(t, 0))
    return out


def _read_chunk_fixture(name):
    f = {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if line:
                k, v = (s.strip() for s in line.split("=", 1))
                f[k] = v
    sym = np.array(_expand(f["symbols"]), np.uint8)
    freq = np.zeros(256, np.uint32)
    for kv in f["freq"].split():
        s, v = kv.split(":")
        freq[int(s)] = int(v)
    states = _expand(f["states"])
    words = [int(w, 16) for w in f.get("words", "").split()]
    stream = b"".join(x.to_bytes(4, "little") for x in states) + \
        b"".join(w.to_bytes(2, "little") for w in words)
    return sym, freq, np.frombuffer(stream, np.uint8)


# ------------------------------------------------------------ quantising ----

def test_normalize_hand_cases(orc):
    # h5 = 2, h9 = 1: floors 2730 and 1365, deficit 1 to the more frequent 5
    f = orc.ans_normalize(np.bincount([5, 5, 9], minlength=256))
    assert (f[5], f[9], f.sum()) == (2731, 1365, 4096)
    # three equal counts: floors 1365 each, deficit 1 to the lowest symbol
    f = orc.ans_normalize(np.bincount([3, 7, 8], minlength=256))
    assert (f[3], f[7], f[8]) == (1366, 1365, 1365)
    # 10000 of symbol 0 and 200 singletons (E = 10200): f0 = 4015 and the 200
    # singletons are raised to 1 (sum 4215); the excess 119 comes off f0
    h = np.zeros(256, np.uint64)
    h[0] = 10000
    h[1:201] = 1
    f = orc.ans_normalize(h)
    assert f[0] == 4015 - 119 and np.all(f[1:201] == 1) and f.sum() == 4096
    # one symbol takes the whole range
    f = orc.ans_normalize(np.bincount([7] * 100, minlength=256))
    assert f[7] == 4096 and f.sum() == 4096


def test_normalize_invariants(orc):
    rng = np.random.default_rng(21)
    for trial in range(300):
        k = int(rng.integers(1, 257))
        h = np.zeros(256, np.uint64)
        idx = rng.choice(256, k, replace=False)
        # heavy-tailed counts, many rare symbols
        h[idx] = (rng.pareto(0.7, k) * 3 + 1).astype(np.uint64)
        f = orc.ans_normalize(h)
        assert f.sum() == M
        np.testing.assert_array_equal(f > 0, h > 0)


# ---------------------------------------------------------------- chunks ----

@pytest.mark.parametrize("name", ["ans_chunk_three_symbols.txt",
                                  "ans_chunk_one_word.txt"])
def test_hand_worked_chunks(orc, name):
    sym, freq, stream = _read_chunk_fixture(name)
    got = orc.ans_encode_chunk(sym, freq)
    np.testing.assert_array_equal(got, stream)
    dec, used = orc.ans_decode_chunk(stream, sym.size, freq)
    np.testing.assert_array_equal(dec, sym)
    assert used == stream.size


def test_one_symbol_alphabet_costs_nothing(orc):
    for n in (1, 63, 64, 65, 4096):
        sym = np.full(n, 200, np.uint8)
        f = orc.ans_normalize(np.bincount(sym, minlength=256))
        st = orc.ans_encode_chunk(sym, f)
        assert st.size == 256
        assert np.all(st.view(np.uint32) == L)


def _cost_bits(sym, freq):
    return float(np.sum(np.log2(M / freq[sym].astype(np.float64))))


def test_information_identity(orc):
    """16 W + sum log2(final states) - 64 * 16 equals the symbols' ideal cost
    within log2(1 + 1/16) bits per symbol (the per-step rounding of
    floor(x / f) M + x mod f + c against x M / f, with x >= 16 f)."""
    rng = np.random.default_rng(22)
    for trial in range(40):
        n = int(rng.integers(1, 4097))
        p = rng.dirichlet(np.full(int(rng.integers(2, 40)), 0.4))
        sym = rng.choice(len(p), n, p=p).astype(np.uint8) + np.uint8(100)
        f = orc.ans_normalize(np.bincount(sym, minlength=256))
        st = orc.ans_encode_chunk(sym, f)
        states = st[:256].view(np.uint32).astype(np.float64)
        W = (st.size - 256) // 2
        info = 16 * W + float(np.sum(np.log2(states))) - 64 * 16
        ideal = _cost_bits(sym, f)
        assert abs(info - ideal) <= n * math.log2(1 + 1 / 16) + 1e-6, \
            (n, info, ideal)
        # and in practice the coder is within 0.5% of the ideal
        assert abs(info - ideal) <= 0.005 * ideal + 64


def test_chunk_round_trip_every_length(orc):
    rng = np.random.default_rng(23)
    for n in list(range(1, 200)) + [1000, 4095, 4096]:
        sym = rng.choice([118, 119, 120, 121, 122, 3, 255], n,
                         p=[.3, .3, .2, .1, .07, .02, .01]).astype(np.uint8)
        f = orc.ans_normalize(np.bincount(sym, minlength=256))
        st = orc.ans_encode_chunk(sym, f)
        dec, used = orc.ans_decode_chunk(st, n, f)
        np.testing.assert_array_equal(dec, sym)
        assert used == st.size


# ------------------------------------------------------ section and shard ----

def test_section_layout(orc):
    rng = np.random.default_rng(24)
    for E in (1, 4095, 4096, 4097, 3 * 4096 + 5, 20000):
        exc = rng.choice([120, 121, 122, 123], E, p=[.4, .3, .2, .1]
                         ).astype(np.uint8)
        sec = orc.ans_code_section(exc)
        K = -(-E // 4096)
        assert int(sec[0:4].view(np.uint32)[0]) == K
        assert int(sec[4:8].view(np.uint32)[0]) == 4096
        freq = sec[8:520].view(np.uint16).astype(np.uint32)
        np.testing.assert_array_equal(
            freq, orc.ans_normalize(np.bincount(exc, minlength=256)))
        ends = sec[520:520 + 4 * K].view(np.uint32).astype(np.int64)
        assert np.all(np.diff(np.concatenate([[0], ends])) >= 256)
        assert np.all(ends % 4 == 0)
        assert 520 + 4 * K + int(ends[-1]) == sec.size
        # each chunk is a stand-alone chunk stream of its 4096 symbols
        streams = sec[520 + 4 * K:]
        start = 0
        for c in range(K):
            part = exc[c * 4096:(c + 1) * 4096]
            st = orc.ans_encode_chunk(part, freq)
            np.testing.assert_array_equal(streams[start:start + st.size], st)
            assert not streams[start + st.size:ends[c]].any()
            start = int(ends[c])
        np.testing.assert_array_equal(orc.ans_decode_section(sec, E), exc)


def _shard(orc, n, B, rate, seed):
    rng = np.random.default_rng(seed)
    w = (rng.normal(0, 0.02, n).astype(np.float32).view(np.uint32)
         >> 16).astype(np.uint16)
    w2 = w.copy()
    flip = rng.random(n) < rate
    w2[flip] ^= np.uint16(0x0080)
    return w, w2


@pytest.mark.parametrize("B", [1, 16, 512, 4096])
def test_coded_shard_round_trip_and_sizes(orc, B):
    a16 = lambda x: -(-x // 16) * 16
    for i, (n, rate) in enumerate([(5000, 0.01), (70001, 0.002),
                                   (200003, 0.02), (4096 * 8, 0.0)]):
        w, w2 = _shard(orc, n, B, rate, 100 + i)
        cache = ieee_ref.exponent_field(w)
        enc = orc.encode(w2, cache, B)
        h = orc.header(enc)
        bm = -(-(-(-n // B)) // 8)
        exc = enc[64 + a16(n) + a16(bm):][:h["E"]]
        C = orc.ans_code_section(exc).size
        coded = orc.ans_code(enc, n)
        hc = orc.header(coded)
        if C < h["E"]:
            assert hc["mode"] == 2 and hc["P"] == n + bm + C
            assert hc["total"] == 64 + a16(n) + a16(bm) + a16(C) == coded.size
            assert hc["E"] == h["E"]
            np.testing.assert_array_equal(coded[:64 + a16(n) + a16(bm)][64:],
                                          enc[64:64 + a16(n) + a16(bm)])
            assert not coded[64 + a16(n) + a16(bm) + C:].any()
        else:
            np.testing.assert_array_equal(coded, enc)
        c2 = cache.copy()
        np.testing.assert_array_equal(orc.decode(coded, n, c2), w2)
        np.testing.assert_array_equal(c2, ieee_ref.exponent_field(w2))
        c3 = cache.copy()
        orc.update_cache(c3, coded, n)
        np.testing.assert_array_equal(c3, ieee_ref.exponent_field(w2))


def test_coding_pays_on_natural_exponents(orc):
    """Whole changed blocks of N(0, 0.02) weights carry about 3 bits of
    exponent entropy: the coded section is well under half of E."""
    w, w2 = _shard(orc, 1 << 20, 512, 0.001, 7)
    enc = orc.encode(w2, ieee_ref.exponent_field(w), 512)
    coded = orc.ans_code(enc, 1 << 20)
    h, hc = orc.header(enc), orc.header(coded)
    assert hc["mode"] == 2
    C = hc["P"] - (1 << 20) - (-(-(1 << 20) // 512) // 8)
    assert C < 0.45 * h["E"]


def test_malformed_sections_are_rejected(orc):
    rng = np.random.default_rng(25)
    exc = rng.choice([120, 121, 122], 9000, p=[.5, .3, .2]).astype(np.uint8)
    sec = orc.ans_code_section(exc)
    bad = sec.copy()
    bad[8 + 2 * 120] ^= 1  # frequencies no longer sum to 4096
    with pytest.raises(ValueError):
        orc.ans_decode_section(bad, exc.size)
    with pytest.raises(ValueError):  # truncated
        orc.ans_decode_section(sec[:-4], exc.size)
    with pytest.raises(ValueError):  # wrong chunk count for E
        orc.ans_decode_section(sec, exc.size + 4096)
    bad = sec.copy()
    bad[520 + 4 * 3 + 100] ^= 0x40  # a state or word flipped
    with pytest.raises(ValueError):
        orc.ans_decode_section(bad, exc.size)
