"""Pins for the CPU oracle, each against something other than the oracle:
IEEE-754 value semantics, brute force over every bf16 pattern, the paper's
closed-form sizes (Section 3.2), its reuse model (Section 2.3), hand-worked
fixtures under tests/golden/ and hand-computed gains."""
import math
import os

import numpy as np
import pytest

from tests import ieee_ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _ceil_div(a, b):
    return -(-a // b)


def _a16(x):
    return _ceil_div(x, 16) * 16


def _changed_block_lengths(e_new, cache, B):
    """Per-block element counts of blocks holding any differing exponent,
    computed independently of the oracle (numpy reduce over a padded view)."""
    n = e_new.size
    nb = _ceil_div(n, B)
    diff = np.zeros(nb * B, bool)
    diff[:n] = e_new != cache
    changed = diff.reshape(nb, B).any(axis=1)
    lengths = np.full(nb, B, np.int64)
    if nb:
        lengths[-1] = n - (nb - 1) * B
    return changed, lengths


# ---------------------------------------------------------------- split ----

def test_split_matches_ieee_semantics(orc):
    """Algorithm 1 SplitExpMant on all 65,536 bf16 patterns: the exponent byte
    is the biased exponent of the value, the other byte is sign<<7 | mantissa."""
    w = ieee_ref.all_bf16_patterns()
    e, sm = orc.split(w)
    np.testing.assert_array_equal(e, ieee_ref.exponent_field(w))
    sign = ieee_ref.sign_bit(w)
    np.testing.assert_array_equal(sm >> 7, sign)
    mant = ieee_ref.mantissa7(w)
    finite = mant >= 0
    np.testing.assert_array_equal((sm & 0x7F)[finite], mant[finite])
    # non-finite: exponent 255, and the value is Inf iff the fraction is zero
    nf = ~finite
    assert np.all(e[nf] == 255)
    inf = np.isinf(ieee_ref.bf16_to_f32(w[nf]))
    np.testing.assert_array_equal((sm[nf] & 0x7F) == 0, inf)


def test_every_pattern_against_every_cached_exponent(orc):
    """Brute force over all 65,536 x 256 (new value, old exponent) pairs. Only
    the old exponent matters to the codec, so this is every old/new pair. At
    B=1 the exception list is exactly {new exponent != old}; both B=1 and
    B=512 reconstruct every value bit for bit and leave the new exponents in
    the cache."""
    w = ieee_ref.all_bf16_patterns()
    n = w.size
    e_ref = ieee_ref.exponent_field(w)
    for old in range(256):
        cache = np.full(n, old, np.uint8)
        enc = orc.encode(w, cache, 1)
        h = orc.header(enc)
        changed = e_ref != old
        assert h["E"] == int(changed.sum())
        assert h["changed_blocks"] == int(changed.sum())
        bm = np.frombuffer(enc[64 + _a16(n): 64 + _a16(n) + n // 8].tobytes(),
                           np.uint8)
        bits = np.unpackbits(bm, bitorder="little").astype(bool)
        np.testing.assert_array_equal(bits, changed)
        exc0 = 64 + _a16(n) + _a16(n // 8)
        np.testing.assert_array_equal(enc[exc0: exc0 + h["E"]], e_ref[changed])
        c2 = cache.copy()
        np.testing.assert_array_equal(orc.decode(enc, n, c2), w)
        np.testing.assert_array_equal(c2, e_ref)
        if old % 17 == 0:
            c3 = cache.copy()
            enc512 = orc.encode(w, cache, 512)
            np.testing.assert_array_equal(orc.decode(enc512, n, c3), w)
            np.testing.assert_array_equal(c3, e_ref)


# --------------------------------------------------------------- golden ----

def _read_golden(name):
    fields, raw_bytes = {}, []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            k, v = (s.strip() for s in line.split("=", 1))
            if k == "bytes":
                raw_bytes += [int(t, 16) for t in v.split()]
            else:
                fields[k] = v
    return fields, np.array(raw_bytes, np.uint8)


@pytest.mark.parametrize("name", ["worked_example_b2.txt",
                                  "worked_example_raw.txt"])
def test_hand_worked_example(orc, name):
    f, expect = _read_golden(name)
    w = np.array([int(t, 16) for t in f["values_bits"].split()], np.uint16)
    cache = np.array([int(t, 16) for t in f["cache"].split()], np.uint8)
    raw = f.get("raw", "0") == "1"
    enc = orc.encode(w, None if raw else cache, int(f["B"]), raw=raw)
    h = orc.header(enc)
    for k in ("magic", "version", "mode", "B", "n", "changed_blocks", "E",
              "P", "total"):
        assert h[k] == int(f["header." + k], 0), k
    np.testing.assert_array_equal(enc, expect)
    c2 = cache.copy()
    np.testing.assert_array_equal(orc.decode(enc, w.size, c2), w)
    after = np.array([int(t, 16) for t in f["cache_after"].split()], np.uint8)
    np.testing.assert_array_equal(c2, after)


# ------------------------------------------------------- sizes and shape ----

SIZES = [0, 1, 7, 8, 15, 16, 17, 63, 64, 65, 511, 512, 513, 4095, 4096, 4097,
         16383, 16384, 16385, 100003]
BLOCKS = [1, 3, 16, 64, 512, 4096]


@pytest.mark.parametrize("B", BLOCKS)
def test_payload_closed_form_and_round_trip(orc, B):
    """Section 3.2: payload = S_{s+m} + S_bm + (changed-block exponent bytes)
    with S_b = ceil(n/B), S_bm = ceil(S_b/8); sections 16-byte aligned; the
    shard decodes exactly against ANY cache (not only exp(W)), and afterwards
    the cache holds the new exponents."""
    rng = np.random.default_rng(1000 + B)
    for n in SIZES:
        w = rng.integers(0, 65536, n, dtype=np.uint32).astype(np.uint16)
        e_new = ieee_ref.exponent_field(w)
        cache = e_new.copy()
        flip = rng.random(n) < 0.01
        cache[flip] = rng.integers(0, 256, int(flip.sum()), dtype=np.uint8)
        enc = orc.encode(w, cache, B)
        h = orc.header(enc)
        changed, lengths = _changed_block_lengths(e_new, cache, B)
        S_b = _ceil_div(n, B)
        S_bm = _ceil_div(S_b, 8)
        E = int(lengths[changed].sum())
        assert h["n"] == n and h["B"] == B and h["mode"] == 0
        assert h["changed_blocks"] == int(changed.sum())
        assert h["E"] == E
        assert h["P"] == n + S_bm + E
        assert h["total"] == 64 + _a16(n) + _a16(S_bm) + _a16(E) == enc.size
        # padding bytes are zero
        body = enc[64:]
        assert not body[n:_a16(n)].any()
        assert not body[_a16(n) + S_bm:_a16(n) + _a16(S_bm)].any()
        assert not enc[64 + _a16(n) + _a16(S_bm) + E:].any()
        c2 = cache.copy()
        np.testing.assert_array_equal(orc.decode(enc, n, c2), w)
        np.testing.assert_array_equal(c2, e_new)
        c3 = cache.copy()
        orc.update_cache(c3, enc, n)
        np.testing.assert_array_equal(c3, e_new)


def test_zero_exceptions_when_no_exponent_changed(orc):
    """Algorithm 1: with no block flagged there is no exception payload; the
    wire holds the sign+mantissa plane and an all-zero bitmap only."""
    rng = np.random.default_rng(7)
    for n, B in [(1 << 20, 512), (12345, 64), (999, 1)]:
        w = rng.integers(0, 65536, n, dtype=np.uint32).astype(np.uint16)
        cache = ieee_ref.exponent_field(w)
        enc = orc.encode(w, cache, B)
        h = orc.header(enc)
        bm = _ceil_div(_ceil_div(n, B), 8)
        assert h["E"] == 0 and h["changed_blocks"] == 0
        assert h["P"] == n + bm
        assert not enc[64 + _a16(n):].any()


def test_raw_mode(orc):
    rng = np.random.default_rng(3)
    for n in [0, 1, 17, 4097]:
        w = rng.integers(0, 65536, n, dtype=np.uint32).astype(np.uint16)
        enc = orc.encode(w, None, 512, raw=True)
        h = orc.header(enc)
        assert h["mode"] == 1 and h["P"] == 2 * n
        assert h["total"] == 64 + _a16(2 * n) == enc.size
        np.testing.assert_array_equal(enc[64:64 + 2 * n].view(np.uint16), w)
        cache = rng.integers(0, 256, n, dtype=np.uint8)
        c2 = cache.copy()
        np.testing.assert_array_equal(orc.decode(enc, n, cache), w)
        np.testing.assert_array_equal(cache, ieee_ref.exponent_field(w))
        # the cache update alone seeds the same exponents
        orc.update_cache(c2, enc, n)
        np.testing.assert_array_equal(c2, ieee_ref.exponent_field(w))


def test_special_values_round_trip(orc):
    """Lossless on +-0, subnormals, +-Inf and every NaN payload."""
    specials = [0x0000, 0x8000, 0x0001, 0x8001, 0x007F, 0x807F, 0x0080,
                0x7F7F, 0xFF7F, 0x7F80, 0xFF80]
    nans = list(range(0x7F81, 0x8000)) + list(range(0xFF81, 0x10000))
    w = np.array(specials + nans, np.uint16)
    for B in (1, 16, 512):
        cache = np.random.default_rng(B).integers(0, 256, w.size,
                                                  dtype=np.uint8)
        enc = orc.encode(w, cache, B)
        c2 = cache.copy()
        np.testing.assert_array_equal(orc.decode(enc, w.size, c2), w)


def test_bad_headers_rejected(orc):
    w = np.arange(100, dtype=np.uint16)
    enc = orc.encode(w, np.zeros(100, np.uint8), 16)
    for pos, val in [(0, 0x00), (4, 0x02), (6, 0x05), (16, 99)]:
        bad = enc.copy()
        bad[pos] = val
        with pytest.raises(ValueError):
            orc.decode(bad, 100, np.zeros(100, np.uint8))
    with pytest.raises(ValueError):
        orc.decode(enc, 101, np.zeros(101, np.uint8))
    # a bitmap that flags more blocks than the exception list holds
    bad = enc.copy()
    bad[64 + _a16(100)] ^= 0x01
    with pytest.raises(ValueError):
        orc.decode(bad, 100, np.zeros(100, np.uint8))


# ------------------------------------------------ change structure pins ----

def test_forced_exact_k(orc):
    """Exactly K forced exponent moves: E(B=1) = K and the changed-block
    count at B=512 is the number of distinct blocks the moves hit."""
    import torch
    from paper_2609_04609_amd import synth
    n, K = 131072, 1311
    w = synth.normal_bf16_bits(n, 0.02, 11)
    w2, idx = synth.forced_exact_k_bits(w, K, 12)
    wn, w2n = w.numpy().view(np.uint16), w2.numpy().view(np.uint16)
    cache = ieee_ref.exponent_field(wn)
    h1 = orc.header(orc.encode(w2n, cache, 1))
    assert h1["E"] == K
    h512 = orc.header(orc.encode(w2n, cache, 512))
    assert h512["changed_blocks"] == len(set((idx // 512).tolist()))
    assert isinstance(idx, torch.Tensor)


@pytest.mark.parametrize("B,c", [(64, 0.003), (512, 0.001), (512, 0.0005),
                                 (4096, 0.0002)])
def test_block_change_rate_matches_reuse_model(orc, B, c):
    """Section 2.3: with independent per-element change probability c, a block
    of B values stays reusable with probability (1-c)^B; the oracle's changed
    block fraction lies within 5 sigma of 1 - (1-c)^B."""
    from paper_2609_04609_amd import synth
    n = 1 << 22
    w = synth.normal_bf16_bits(n, 0.02, 21)
    w2 = synth.forced_bernoulli_bits(w, c, 22)
    wn, w2n = w.numpy().view(np.uint16), w2.numpy().view(np.uint16)
    h = orc.header(orc.encode(w2n, ieee_ref.exponent_field(wn), B))
    nb = n // B
    q = 1.0 - (1.0 - c) ** B
    sigma = math.sqrt(q * (1 - q) / nb)
    assert abs(h["changed_blocks"] / nb - q) < 5 * sigma + 1e-12


def test_multi_step_chain_sender_and_receiver_caches_agree(orc):
    """A small mirror of the paper's bitwise-correctness run (Section 4.6):
    over T updates, the sender's cache and every receiver's cache stay equal
    and every gathered shard decodes exactly."""
    from paper_2609_04609_amd import synth
    R, n, B, T = 4, 5000, 64, 6
    ws = [synth.normal_bf16_bits(n, 0.02, 100 + j).numpy().view(np.uint16)
          for j in range(R)]
    # step 0: raw gather seeds every cache
    send_cache = [np.zeros(n, np.uint8) for _ in range(R)]
    recv_cache = np.zeros(R * n, np.uint8)
    for t in range(T):
        encs = []
        for j in range(R):
            if t == 0:
                e = orc.encode(ws[j], None, B, raw=True)
            else:
                e = orc.encode(ws[j], send_cache[j], B)
            orc.update_cache(send_cache[j], e, n)
            encs.append(e)
        offs = np.cumsum([0] + [e.size for e in encs[:-1]]).astype(np.uint64)
        gathered = np.concatenate(encs)
        out = orc.decode_gathered(gathered, offs, n, recv_cache)
        np.testing.assert_array_equal(out, np.concatenate(ws))
        np.testing.assert_array_equal(recv_cache, np.concatenate(send_cache))
        import torch
        ws = [synth.natural_update_bits(torch.from_numpy(x.view(np.int16)),
                                        3e-4, 1000 * t + j).numpy()
              .view(np.uint16) for j, x in enumerate(ws)]
