"""Pins for the oracle's sender-side block hash (Section 3.1: Hash128 built
from two SplitMix64 hashes, HashCache on the sender).

What fixes the hash, independently of the oracle's C code:
  - the SplitMix64 finaliser is the mixing step of pandas' hash_array on
    uint64 data (a library routine);
  - GAMMA is the odd integer nearest to 2^64 / golden ratio, computed here
    with exact integer square roots;
  - the two seeds are the first 128 bits of the binary fraction of pi,
    computed here with Machin's formula in integer arithmetic;
  - a one-word block of zeros hashes to the first SplitMix64 output of each
    seed, so GAMMA, the seeds and the word index enter as published.
How a block's words combine into H_t is a reading (the paper leaves it open);
it is pinned through its decisions: the hashed encoder must emit exactly the
bytes of the exact-compare encoder on every case below, and a block counts as
unchanged only when both 64-bit halves match.
"""
import math

import numpy as np
import pandas as pd
import pytest

from tests import ieee_ref

M64 = (1 << 64) - 1


def _pandas_mix(vals):
    a = np.asarray(vals, dtype=np.uint64)
    return [int(x) for x in pd.util.hash_array(a, categorize=False)]


def _gamma():
    # 2^64 / phi = 2^63 (sqrt 5 - 1); take the nearest odd integer
    r = math.isqrt(5 << 126) - (1 << 63)   # floor(2^63 sqrt 5) - 2^63
    return r if r & 1 else r + 1


def _pi_fraction_words(count):
    """First `count` 64-bit words of the binary fraction of pi (Machin:
    pi = 16 atan(1/5) - 4 atan(1/239)), exact integer arithmetic."""
    bits = 64 * count + 64
    one = 1 << bits

    def atan_inv(x):
        total, term, k, x2 = 0, one // x, 1, x * x
        while term:
            total += term // k if (k // 2) % 2 == 0 else -(term // k)
            term //= x2
            k += 2
        return total
    pi = 16 * atan_inv(5) - 4 * atan_inv(239)
    frac = pi - 3 * one
    return [(frac >> (bits - 64 * (i + 1))) & M64 for i in range(count)]


GAMMA = _gamma()
SEEDS = _pi_fraction_words(2)


def test_constants_have_their_published_values():
    assert GAMMA == 0x9E3779B97F4A7C15
    assert SEEDS == [0x243F6A8885A308D3, 0x13198A2E03707344]


def test_finaliser_matches_library_routine(orc):
    rng = np.random.default_rng(11)
    vals = rng.integers(0, 1 << 63, 4000, dtype=np.uint64) * np.uint64(2) \
        + rng.integers(0, 2, 4000, dtype=np.uint64)
    vals = np.concatenate([vals, np.array([0, 1, M64, GAMMA], np.uint64)])
    want = _pandas_mix(vals)
    got = [orc.sm64_mix(int(v)) for v in vals]
    assert got == want
    # the first output of SplitMix64 seeded with 0
    assert orc.sm64_mix(GAMMA) == 0xE220A8397B1DCDAF


def test_single_word_blocks_are_splitmix64_outputs(orc):
    """len <= 8: H_t = mix(u_0 XOR (s_t + GAMMA)); for u_0 = 0 that is the
    first SplitMix64 output of seed s_t; a two-word zero block sums the first
    two outputs."""
    for t in range(2):
        assert orc.block_hash(np.zeros(8, np.uint8))[t] == \
            _pandas_mix([(SEEDS[t] + GAMMA) & M64])[0]
        two = _pandas_mix([(SEEDS[t] + GAMMA) & M64,
                           (SEEDS[t] + 2 * GAMMA) & M64])
        assert orc.block_hash(np.zeros(16, np.uint8))[t] == sum(two) & M64
    rng = np.random.default_rng(12)
    for ln in (1, 3, 7, 8):
        e = rng.integers(0, 256, ln, dtype=np.uint8)
        u = int.from_bytes(bytes(e) + bytes(8 - ln), "little")
        for t in range(2):
            assert orc.block_hash(e)[t] == \
                _pandas_mix([u ^ ((SEEDS[t] + GAMMA) & M64)])[0]


def _exps_like(e):
    """bf16 patterns whose exponent bytes are e (sign and mantissa 0)."""
    return (np.asarray(e, np.uint16) << 7).astype(np.uint16)


@pytest.mark.parametrize("B", [8, 16, 64, 512, 4096])
def test_hashed_encode_equals_exact_compare(orc, B):
    """Same bytes as the exact-compare encoder (any change flagged, nothing
    else), and the HashCache afterwards equals the new weights' hashes."""
    rng = np.random.default_rng(100 + B)
    for n in (0, 1, 7, 8, 9, 511, 512, 513, 4097, 20011):
        w_old = rng.integers(0, 65536, n, dtype=np.uint32).astype(np.uint16)
        w_new = w_old.copy()
        for rate in (0.0, 0.001, 0.05, 1.0):
            flip = rng.random(n) < rate
            w_new = w_old.copy()
            # +-1 exponent steps and whole-pattern changes
            w_new[flip] ^= np.uint16(0x0080)
            cache = ieee_ref.exponent_field(w_old)
            h_old = orc.hash_blocks(w_old, B)
            enc_h, h_new = orc.encode_hashed(w_new, h_old, B)
            np.testing.assert_array_equal(enc_h, orc.encode(w_new, cache, B))
            np.testing.assert_array_equal(h_new, orc.hash_blocks(w_new, B))


def test_brute_force_every_pattern_against_old_exponents(orc):
    """All 65,536 bf16 patterns against a cache holding one old exponent:
    the hashed encoder flags exactly the blocks the exact compare flags."""
    w = ieee_ref.all_bf16_patterns()
    for old in (0, 1, 126, 127, 128, 200, 254, 255):
        w_old = _exps_like(np.full(w.size, old))
        cache = np.full(w.size, old, np.uint8)
        for B in (16, 512):
            enc_h, _ = orc.encode_hashed(w, orc.hash_blocks(w_old, B), B)
            np.testing.assert_array_equal(enc_h, orc.encode(w, cache, B))


def test_every_single_byte_change_is_detected(orc):
    """One exponent byte changed anywhere in a block: one word's term
    changes and the finaliser is a bijection, so both halves change."""
    rng = np.random.default_rng(13)
    e = rng.integers(0, 255, 512, dtype=np.uint8)
    h0 = orc.block_hash(e)
    for k in range(512):
        e2 = e.copy()
        e2[k] = (int(e2[k]) + 1 + int(rng.integers(0, 254))) % 256
        h1 = orc.block_hash(e2)
        assert h1[0] != h0[0] and h1[1] != h0[1]


def test_both_halves_must_match(orc):
    """HashCache semantics: a block is reused only when all 128 bits match;
    a stored hash differing in either half flags the block."""
    rng = np.random.default_rng(14)
    n, B = 4096, 512
    w = rng.integers(0, 65536, n, dtype=np.uint32).astype(np.uint16)
    h = orc.hash_blocks(w, B)
    enc, _ = orc.encode_hashed(w, h, B)
    assert orc.header(enc)["changed_blocks"] == 0
    for half, blk in ((0, 2), (1, 5)):
        h2 = h.copy()
        h2[2 * blk + half] ^= np.uint64(1 << 40)
        enc2, hout = orc.encode_hashed(w, h2, B)
        hd = orc.header(enc2)
        assert hd["changed_blocks"] == 1 and hd["E"] == B
        np.testing.assert_array_equal(hout, h)
        c = ieee_ref.exponent_field(w)
        c[blk * B] ^= 1
        np.testing.assert_array_equal(enc2, orc.encode(w, c, B))
