"""Do the pins catch plausible mistakes in the oracle?

Each case plants one mistake in a copy of oracle/ciera_oracle.c (on the CPU
only), builds it with gcc, and runs a condensed set of the pins against it:
IEEE-semantics field extraction, brute force over old exponents, the
hand-worked wire fixtures, closed-form sizes and zero padding, the raw form,
a hand-computed gain and a hand-ranked selection, the block-hash pins,
the rANS pins and the fp16 pins. Every mutant must fail at
least one of them; the real oracle must pass all of them.
"""
import os
import subprocess
import sys

import numpy as np
import pytest

from tests import ieee_ref
from tests.test_oracle_pins import _read_golden

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "ciera_oracle.c")

# (name, text in the source, planted replacement)
MUTANTS = [
    ("exponent shift", "uint8_t expo = (uint8_t)((x >> 7) & 0xFFu);",
     "uint8_t expo = (uint8_t)((x >> 8) & 0xFFu);"),
    ("sign bit position", "sm[k] = (uint8_t)((sign << 7) | mant);",
     "sm[k] = (uint8_t)((sign << 6) | mant);"),
    ("mantissa mask", "uint8_t mant = (uint8_t)(x & 0x7Fu);",
     "uint8_t mant = (uint8_t)(x & 0x3Fu);"),
    ("merge drops the sign", "return (uint16_t)((sign << 15) | ((uint16_t)expo << 7) | mant);",
     "return (uint16_t)(((uint16_t)expo << 7) | mant);"),
    ("change test ignores decreases", "if (expo[k] != cache[k]) {",
     "if (expo[k] > cache[k]) {"),
    ("bitmap bit order", "bitmap[b / 8u] = (uint8_t)(bitmap[b / 8u] | (1u << (b % 8u)));",
     "bitmap[b / 8u] = (uint8_t)(bitmap[b / 8u] | (0x80u >> (b % 8u)));"),
    ("last partial block dropped", "  uint64_t nblk = num_blocks(n, B);\n  uint8_t *changed",
     "  uint64_t nblk = n / B;\n  uint8_t *changed"),
    ("exceptions of the first element only", "for (uint64_t k = lo; k < hi; k++) exc[E++] = expo[k];",
     "for (uint64_t k = lo; k < lo + 1; k++) exc[E++] = expo[k];"),
    ("bitmap size floors", "return ceil_div(num_blocks(n, B), 8u);",
     "return num_blocks(n, B) / 8u;"),
    ("padding rounds wrong", "static uint64_t round16(uint64_t x) { return (x + 15u) / 16u * 16u; }",
     "static uint64_t round16(uint64_t x) { return (x + 16u) / 16u * 16u; }"),
    ("payload omits the bitmap", "uint64_t P = n + bm + E;", "uint64_t P = n + E;"),
    ("header swaps E and count", "put_u64(out + 32, E);", "put_u64(out + 32, changed);"),
    ("padding left unwritten",
     "  memset(out, 0, total);\n  write_header(out, OR_MODE_COMPRESSED, B, n, nchanged",
     "  write_header(out, OR_MODE_COMPRESSED, B, n, nchanged"),
    ("decode patches only the first value of a block",
     "for (uint64_t k = lo; k < hi; k++) cache[k] = exc[j++];",
     "cache[lo] = exc[j]; j += hi - lo;"),
    ("raw cache from the wrong field", "cache[k] = (uint8_t)((x >> 7) & 0xFFu);\n    }\n    return 0;\n  }\n  return patch_cache",
     "cache[k] = (uint8_t)((x >> 6) & 0xFFu);\n    }\n    return 0;\n  }\n  return patch_cache"),
    ("raw decode seeds the wrong field",
     "      out[k] = x;\n      cache[k] = (uint8_t)((x >> 7) & 0xFFu);",
     "      out[k] = x;\n      cache[k] = (uint8_t)((x >> 8) & 0xFFu);"),
    ("decode skips the patch", "  if (E > 0 && patch_cache(enc, n, B, cache)) return -4;",
     "  if (E > n && patch_cache(enc, n, B, cache)) return -4;"),
    ("ans emission bound", "(uint64_t)((OR_ANS_L >> OR_ANS_SCALE) << 16) * f;",
     "(uint64_t)((OR_ANS_L >> OR_ANS_SCALE) << 15) * f;"),
    ("ans decoder drops the cumulative",
     "x[l] = freq[s] * (x[l] >> OR_ANS_SCALE) + slot - cum[s];",
     "x[l] = freq[s] * (x[l] >> OR_ANS_SCALE) + slot;"),
    ("ans words in emission order", "emitted[nw - 1u - k]", "emitted[k]"),
    ("ans deficit tie to the last symbol", "if (hist[s] > hist[best]) best = s;",
     "if (hist[s] >= hist[best]) best = s;"),
    ("ans chunk size", "#define OR_ANS_CHUNK 4096u", "#define OR_ANS_CHUNK 2048u"),
    ("ans codes when not smaller", "  if (C < E) {", "  if (C < E + 100000u) {"),
    ("gain counts R hops", "double comm_raw = alpha_s + (double)(R - 1) * S / bw_Bps;",
     "double comm_raw = alpha_s + (double)R * S / bw_Bps;"),
    ("gain ignores overlap flag", "double sender = overlapped ? 0.0 : (t_hash_s + t_cmp_s);",
     "double sender = 0.0;"),
    ("gain drops the decode time", "return comm_raw - (comm_cmp + sender + t_decmp_s);",
     "return comm_raw - (comm_cmp + sender);"),
    ("fp16 gain counts bf16 exponent bytes", "5.0 * octets, n, B, q, R,",
     "8.0 * octets, n, B, q, R,"),
    ("fp16 gain drops the bit planes", "(double)n + 3.0 * octets,",
     "(double)n,"),
    ("hash word index off by one", "(j + 1u) * OR_SM64_GAMMA",
     "j * OR_SM64_GAMMA"),
    ("hash decision reads one half",
     "h[0] != hash_in[2u * b] || h[1] != hash_in[2u * b + 1u]",
     "h[0] != hash_in[2u * b]"),
    ("hash adds the word to the state", "oracle_sm64_mix(u ^ state)",
     "oracle_sm64_mix(u + state)"),
    ("hash drops the last partial word", "uint64_t words = ceil_div(len, 8u);",
     "uint64_t words = len / 8u;"),
    ("finaliser shift", "z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;",
     "z = (z ^ (z >> 28)) * 0x94D049BB133111EBull;"),
    ("fp16 exponent shift", "e[k] = (uint8_t)((x >> 10) & 0x1Fu);",
     "e[k] = (uint8_t)((x >> 11) & 0x1Fu);"),
    ("fp16 high mantissa bits", "hi3[k] = (uint8_t)((sign << 2) | ((x >> 8) & 0x3u));",
     "hi3[k] = (uint8_t)((sign << 2) | ((x >> 9) & 0x3u));"),
    ("fp16 exception group stride", "out[off_exc + 5u * (i / 8u) + p] |=",
     "out[off_exc + 4u * (i / 8u) + p] |="),
    ("fp16 sign+mantissa size floors",
     "static uint64_t f16_sm_bytes(uint64_t n) { return n + 3u * ceil_div(n, 8u); }",
     "static uint64_t f16_sm_bytes(uint64_t n) { return n + 3u * (n / 8u); }"),
    ("select sorts ascending", "if (ry >= rx) break;", "if (ry <= rx) break;"),
    ("select keeps non-positive gains", "if (gain[i] > 0.0) order[m++] = i;",
     "if (gain[i] >= 0.0) order[m++] = i;"),
]


def _build(src_text, out_dir, tag):
    c = os.path.join(out_dir, f"m_{tag}.c")
    so = os.path.join(out_dir, f"libm_{tag}.so")
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-w", "-fPIC", "-shared",
                           "-I" + os.path.join(ROOT, "oracle"), "-o", so, c])
    return so


def _pins(o):
    """Returns the list of pins the oracle object fails (empty = all pass)."""
    failed = []

    def check(name, fn):
        try:
            if not fn():
                failed.append(name)
        except Exception:  # an exception is a detection too
            failed.append(name)

    allw = ieee_ref.all_bf16_patterns()
    e_ref = ieee_ref.exponent_field(allw)

    def split_ieee():
        e, sm = o.split(allw)
        mant = ieee_ref.mantissa7(allw)
        fin = mant >= 0
        return (np.array_equal(e, e_ref)
                and np.array_equal(sm >> 7, ieee_ref.sign_bit(allw))
                and np.array_equal((sm & 0x7F)[fin], mant[fin]))
    check("split", split_ieee)

    def brute_force():
        n = allw.size
        a16 = lambda x: -(-x // 16) * 16
        for old in (0, 1, 126, 127, 128, 200, 255):
            cache = np.full(n, old, np.uint8)
            enc = o.encode(allw, cache, 1)
            h = o.header(enc)
            changed = e_ref != old
            if h["E"] != int(changed.sum()):
                return False
            exc0 = 64 + a16(n) + a16(n // 8)
            if not np.array_equal(enc[exc0:exc0 + h["E"]], e_ref[changed]):
                return False
            c2 = cache.copy()
            if not np.array_equal(o.decode(enc, n, c2), allw):
                return False
            if not np.array_equal(c2, e_ref):
                return False
            c3 = cache.copy()
            if not np.array_equal(o.decode(o.encode(allw, cache, 512), n, c3),
                                  allw):
                return False
        return True
    check("brute force", brute_force)

    def golden():
        for name in ("worked_example_b2.txt", "worked_example_raw.txt"):
            f, expect = _read_golden(name)
            w = np.array([int(t, 16) for t in f["values_bits"].split()],
                         np.uint16)
            cache = np.array([int(t, 16) for t in f["cache"].split()],
                             np.uint8)
            raw = f.get("raw", "0") == "1"
            enc = o.encode(w, None if raw else cache, int(f["B"]), raw=raw)
            if not np.array_equal(enc, expect):
                return False
        return True
    check("golden", golden)

    def sizes():
        rng = np.random.default_rng(3)
        a16 = lambda x: -(-x // 16) * 16
        for n in (1, 17, 511, 513, 4097, 10007):
            for B in (1, 16, 512, 4096):
                w = rng.integers(0, 65536, n, dtype=np.uint32).astype(np.uint16)
                e_new = ieee_ref.exponent_field(w)
                cache = e_new.copy()
                flip = rng.random(n) < 0.05
                cache[flip] = rng.integers(0, 256, int(flip.sum()),
                                           dtype=np.uint8)
                enc = o.encode(w, cache, B)
                h = o.header(enc)
                nb = -(-n // B)
                diff = np.zeros(nb * B, bool)
                diff[:n] = e_new != cache
                ch = diff.reshape(nb, B).any(axis=1)
                lens = np.full(nb, B)
                lens[-1] = n - (nb - 1) * B
                E = int(lens[ch].sum())
                bm = -(-nb // 8)
                if h["E"] != E or h["P"] != n + bm + E:
                    return False
                if h["changed_blocks"] != int(ch.sum()):
                    return False
                if h["total"] != 64 + a16(n) + a16(bm) + a16(E) != enc.size:
                    return False
                if enc[64 + n:64 + a16(n)].any() or enc[64 + a16(n) + bm:
                                                         64 + a16(n) + a16(bm)].any():
                    return False
                if enc[64 + a16(n) + a16(bm) + E:].any():
                    return False
                c2 = cache.copy()
                if not np.array_equal(o.decode(enc, n, c2), w):
                    return False
                c3 = cache.copy()
                o.update_cache(c3, enc, n)
                if not np.array_equal(c3, e_new):
                    return False
        return True
    check("sizes", sizes)

    def raw_mode():
        w = np.random.default_rng(5).integers(0, 65536, 999, dtype=np.uint32
                                              ).astype(np.uint16)
        enc = o.encode(w, None, 512, raw=True)
        cache = np.zeros(999, np.uint8)
        c2 = cache.copy()
        ok = np.array_equal(o.decode(enc, 999, cache), w)
        o.update_cache(c2, enc, 999)
        e = ieee_ref.exponent_field(w)
        return ok and np.array_equal(cache, e) and np.array_equal(c2, e)
    check("raw", raw_mode)

    def gain_hand():
        g = o.gain(1_000_000, 512, 0.2, 16, 10e-6, 8e9, t_decmp_s=1e-3)
        g2 = o.gain(1_000_000, 512, 0.2, 16, 10e-6, 8e9, t_hash_s=2e-4,
                    t_cmp_s=4e-4, t_decmp_s=1e-3, overlapped=False)
        g3 = o.gain(1_000_000, 512, 0.2, 16, 10e-6, 8e9, t_decmp_s=1e-3,
                    fp16=True)
        return (abs(g - 0.000499420625) < 1e-12
                and abs(g2 - (0.000499420625 - 6e-4)) < 1e-12
                and abs(g3 + 0.000063079375) < 1e-12)
    check("gain", gain_hand)

    def hash_pins():
        from tests.test_oracle_hash_pins import GAMMA, SEEDS, _pandas_mix
        M = (1 << 64) - 1
        if o.sm64_mix(GAMMA) != 0xE220A8397B1DCDAF:
            return False
        e = np.array([3, 0, 250, 17, 9], np.uint8)
        u = int.from_bytes(bytes(e) + bytes(3), "little")
        for t in range(2):
            if o.block_hash(e)[t] != _pandas_mix([u ^ ((SEEDS[t] + GAMMA) & M)])[0]:
                return False
            if o.block_hash(np.zeros(16, np.uint8))[t] != sum(_pandas_mix(
                    [(SEEDS[t] + GAMMA) & M, (SEEDS[t] + 2 * GAMMA) & M])) & M:
                return False
        rng = np.random.default_rng(15)
        for n, B in ((20011, 512), (13, 8)):
            w_old = rng.integers(0, 65536, n, dtype=np.uint32).astype(np.uint16)
            w_new = w_old.copy()
            w_new[-1] ^= np.uint16(0x0080)
            w_new[n // 3] ^= np.uint16(0x0080)
            h = o.hash_blocks(w_old, B)
            enc, _ = o.encode_hashed(w_new, h, B)
            if not np.array_equal(enc, o.encode(
                    w_new, ieee_ref.exponent_field(w_old), B)):
                return False
            h2 = o.hash_blocks(w_new, B)
            h2[1] ^= np.uint64(1)
            enc, _ = o.encode_hashed(w_new, h2, B)
            if o.header(enc)["changed_blocks"] != 1:
                return False
        return True
    check("hash", hash_pins)

    def ans_pins():
        from tests.test_oracle_ans_pins import _read_chunk_fixture
        f = o.ans_normalize(np.bincount([3, 7, 8], minlength=256))
        if (f[3], f[7], f[8]) != (1366, 1365, 1365):
            return False
        f = o.ans_normalize(np.bincount([5, 5, 9], minlength=256))
        if (f[5], f[9]) != (2731, 1365):
            return False
        for name in ("ans_chunk_three_symbols.txt", "ans_chunk_one_word.txt"):
            sym, freq, stream = _read_chunk_fixture(name)
            if not np.array_equal(o.ans_encode_chunk(sym, freq), stream):
                return False
        rng = np.random.default_rng(26)
        sym = rng.choice([118, 119, 120, 121, 7], 3000,
                         p=[.4, .3, .2, .09, .01]).astype(np.uint8)
        f = o.ans_normalize(np.bincount(sym, minlength=256))
        dec, _ = o.ans_decode_chunk(o.ans_encode_chunk(sym, f), sym.size, f)
        if not np.array_equal(dec, sym):
            return False
        sec = o.ans_code_section(np.tile(sym, 3))
        if int(sec[4:8].view(np.uint32)[0]) != 4096 or \
                int(sec[0:4].view(np.uint32)[0]) != 3:
            return False
        n = 30011
        w = (rng.normal(0, 0.02, n).astype(np.float32).view(np.uint32)
             >> 16).astype(np.uint16)
        for rate in (0.01, 0.0):
            w2 = w.copy()
            w2[rng.random(n) < rate] ^= np.uint16(0x0080)
            cache = ieee_ref.exponent_field(w)
            enc = o.encode(w2, cache, 64)
            coded = o.ans_code(enc, n)
            E = o.header(enc)["E"]
            a16 = lambda x: -(-x // 16) * 16
            exc = enc[64 + a16(n) + a16(-(-(-(-n // 64)) // 8)):][:E]
            if (o.header(coded)["mode"] == 2) != \
                    (o.ans_code_section(exc).size < E):
                return False
            c2 = cache.copy()
            if not np.array_equal(o.decode(coded, n, c2), w2):
                return False
        return True
    check("ans", ans_pins)

    def f16_pins():
        from tests.test_oracle_f16_pins import ALL, _unpack_groups
        e, lo, hi = o.split_f16(ALL)
        if not np.array_equal(e, ieee_ref.exponent_field_f16(ALL)):
            return False
        f, expect = _read_golden("worked_example_f16_b2.txt")
        w = np.array([int(t, 16) for t in f["values_bits"].split()],
                     np.uint16)
        cache = np.array([int(t, 16) for t in f["cache"].split()], np.uint8)
        if not np.array_equal(o.encode_f16(w, cache, 2), expect):
            return False
        rng = np.random.default_rng(42)
        n = 20013
        w = rng.integers(0, 65536, n, dtype=np.uint32).astype(np.uint16)
        c = ieee_ref.exponent_field_f16(w)
        c[rng.random(n) < 0.01] ^= 1
        for B in (1, 64):
            enc = o.encode_f16(w, c, B)
            h = o.header(enc)
            S_sm = n + 3 * (-(-n // 8))
            if h["P"] != S_sm + (-(-(-(-n // B)) // 8)) + 5 * (-(-h["E"] // 8)):
                return False
            hi3 = _unpack_groups(enc[64 + n:64 + S_sm], n, 3)
            if not np.array_equal(hi3, (ieee_ref.sign_f16(w).astype(
                    np.int64) << 2) | ((w.astype(np.int64) >> 8) & 3)):
                return False
            c2 = c.copy()
            if not np.array_equal(o.decode_f16(enc, n, c2), w):
                return False
        return True
    check("fp16", f16_pins)

    def select_hand():
        # budget 6.5 MB: 3, 4, 0 fill 6 MB; the zero-gain shard 5 would fit
        g = [3e-3, 1e-3, -1e-3, 4e-3, 2e-3, 0.0]
        m = [3e6, 2e6, 1e6, 2e6, 1e6, 0.5e6]
        return list(o.select(g, m, 6.5e6)) == [True, False, False, True, True,
                                               False]
    check("select", select_hand)
    return failed


@pytest.fixture(scope="module")
def src_text():
    with open(SRC) as f:
        return f.read()


def test_real_oracle_passes_condensed_pins(orc):
    from oracle import oracle
    assert _pins(oracle.Oracle(oracle._LIB)) == []


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, src_text, name, old, new):
    """The pins run in a child process: a planted mistake that crashes the
    oracle (an overrun, say) is a detection too."""
    assert src_text.count(old) == 1, f"mutation site not found: {name}"
    so = _build(src_text.replace(old, new), str(tmp_path), "m")
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from oracle import oracle\n"
            "from tests.test_oracle_mutants import _pins\n"
            "failed = _pins(oracle.Oracle(%r))\n"
            "print('FAILED:', failed)\n"
            "sys.exit(3 if failed else 0)\n") % (ROOT, so)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode != 0, f"no pin catches the planted mistake: {name}"
