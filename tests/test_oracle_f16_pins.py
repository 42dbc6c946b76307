"""Pins for the oracle's fp16 shards (the paper's second precision, Table 2;
sizes S_e = 5n/8, S_{s+m} = 11n/8), against IEEE binary16 semantics, a
hand-worked fixture, brute force over every fp16 pattern and closed-form
sizes. The bit-plane sections are unpacked here with numpy, not with the
oracle's own loops."""
import os

import numpy as np
import pytest

from tests import ieee_ref
from tests.test_oracle_pins import _read_golden

ALL = np.arange(65536, dtype=np.uint32).astype(np.uint16)


def a16(x):
    return -(-x // 16) * 16


def _unpack_groups(buf, count, planes):
    """Values whose bit p is bit k of byte planes*g + p (group g = i // 8)."""
    groups = -(-count // 8)
    b = np.asarray(buf[:planes * groups], np.uint8).reshape(groups, planes)
    bits = np.unpackbits(b, axis=1, bitorder="little").reshape(
        groups, planes, 8)  # [group, plane, k]
    v = np.zeros((groups, 8), np.int64)
    for p in range(planes):
        v |= bits[:, p, :].astype(np.int64) << p
    return v.ravel()[:count]


def test_split_matches_binary16_semantics(orc):
    e, lo, hi = orc.split_f16(ALL)
    np.testing.assert_array_equal(e, ieee_ref.exponent_field_f16(ALL))
    np.testing.assert_array_equal(hi >> 2, ieee_ref.sign_f16(ALL))
    mant = ieee_ref.mantissa10_f16(ALL)
    fin = mant >= 0
    np.testing.assert_array_equal(((hi.astype(np.int64) & 3) << 8 | lo)[fin],
                                  mant[fin])
    # non-finite: exponent 31, Inf iff the fraction is zero
    nf = ~fin
    inf = np.isinf(ieee_ref.f16_values(ALL[nf]))
    np.testing.assert_array_equal((((hi[nf] & 3).astype(int) << 8) | lo[nf])
                                  == 0, inf)


def test_hand_worked_fp16_example(orc):
    f, expect = _read_golden("worked_example_f16_b2.txt")
    w = np.array([int(t, 16) for t in f["values_bits"].split()], np.uint16)
    cache = np.array([int(t, 16) for t in f["cache"].split()], np.uint8)
    enc = orc.encode_f16(w, cache, int(f["B"]))
    h = orc.header(enc)
    assert h["dtype"] == 1
    for k in ("magic", "version", "mode", "B", "n", "changed_blocks", "E",
              "P", "total"):
        assert h[k] == int(f["header." + k], 0), k
    np.testing.assert_array_equal(enc, expect)
    c2 = cache.copy()
    np.testing.assert_array_equal(orc.decode_f16(enc, w.size, c2), w)
    after = np.array([int(t, 16) for t in f["cache_after"].split()], np.uint8)
    np.testing.assert_array_equal(c2, after)


def test_every_pattern_against_every_old_exponent(orc):
    """All 65,536 patterns x all 32 old exponents: at B = 1 the exception
    list is exactly the differing exponents (unpacked here from the planes),
    and B = 1, 16, 512 rebuild every value and leave the new exponents."""
    n = ALL.size
    e_ref = ieee_ref.exponent_field_f16(ALL)
    S_sm = n + 3 * (n // 8)
    for old in range(32):
        cache = np.full(n, old, np.uint8)
        enc = orc.encode_f16(ALL, cache, 1)
        h = orc.header(enc)
        changed = e_ref != old
        assert h["E"] == int(changed.sum())
        exc0 = 64 + a16(S_sm) + a16(n // 8)
        got = _unpack_groups(enc[exc0:], h["E"], 5)
        np.testing.assert_array_equal(got, e_ref[changed])
        for B in (1, 16, 512):
            e2 = enc if B == 1 else orc.encode_f16(ALL, cache, B)
            c2 = cache.copy()
            np.testing.assert_array_equal(orc.decode_f16(e2, n, c2), ALL)
            np.testing.assert_array_equal(c2, e_ref)


@pytest.mark.parametrize("B", [1, 3, 16, 64, 512, 4096])
def test_sizes_planes_and_round_trip(orc, B):
    rng = np.random.default_rng(40 + B)
    for n in [0, 1, 7, 8, 9, 63, 64, 65, 511, 513, 4097, 20011]:
        w = rng.integers(0, 65536, n, dtype=np.uint32).astype(np.uint16)
        e_new = ieee_ref.exponent_field_f16(w)
        cache = e_new.copy()
        flip = rng.random(n) < 0.02
        cache[flip] = rng.integers(0, 32, int(flip.sum()), dtype=np.uint8)
        enc = orc.encode_f16(w, cache, B)
        h = orc.header(enc)
        nb = -(-n // B)
        diff = np.zeros(nb * B, bool)
        diff[:n] = e_new != cache
        ch = diff.reshape(nb, B).any(axis=1) if nb else np.zeros(0, bool)
        lens = np.full(nb, B)
        if nb:
            lens[-1] = n - (nb - 1) * B
        E = int(lens[ch].sum())
        bm = -(-nb // 8)
        S_sm = n + 3 * (-(-n // 8))
        S_exc = 5 * (-(-E // 8))
        assert h["E"] == E and h["changed_blocks"] == int(ch.sum())
        assert h["P"] == S_sm + bm + S_exc
        assert h["total"] == 64 + a16(S_sm) + a16(bm) + a16(S_exc) == enc.size
        body = enc[64:]
        # low mantissa bytes and the sign/high-mantissa planes, by numpy
        np.testing.assert_array_equal(body[:n], (w & 0xFF).astype(np.uint8))
        hi = _unpack_groups(body[n:S_sm], n, 3)
        np.testing.assert_array_equal(
            hi, (ieee_ref.sign_f16(w).astype(np.int64) << 2) |
            ((w.astype(np.int64) >> 8) & 3))
        # zero padding
        assert not body[S_sm:a16(S_sm)].any()
        assert not body[a16(S_sm) + bm:a16(S_sm) + a16(bm)].any()
        assert not enc[64 + a16(S_sm) + a16(bm) + S_exc:].any()
        c2 = cache.copy()
        np.testing.assert_array_equal(orc.decode_f16(enc, n, c2), w)
        np.testing.assert_array_equal(c2, e_new)
        c3 = cache.copy()
        orc.update_cache_f16(c3, enc, n)
        np.testing.assert_array_equal(c3, e_new)


def test_raw_fp16_and_dtype_checks(orc):
    rng = np.random.default_rng(41)
    w = rng.integers(0, 65536, 1000, dtype=np.uint32).astype(np.uint16)
    enc = orc.encode_f16(w, None, 512, raw=True)
    assert orc.header(enc)["dtype"] == 1 and orc.header(enc)["mode"] == 1
    c = np.zeros(1000, np.uint8)
    np.testing.assert_array_equal(orc.decode_f16(enc, 1000, c), w)
    np.testing.assert_array_equal(c, ieee_ref.exponent_field_f16(w))
    # a bf16 decoder refuses an fp16 shard and the other way round
    with pytest.raises(ValueError):
        orc.decode(enc, 1000, np.zeros(1000, np.uint8))
    enc16 = orc.encode(w, np.zeros(1000, np.uint8), 512)
    with pytest.raises(ValueError):
        orc.decode_f16(enc16, 1000, np.zeros(1000, np.uint8))
