"""Python view of the CIERA reference oracle (plain C in ``ciera_oracle.c``).

TEST INFRASTRUCTURE ONLY. The product package never imports this module; only
the tests, the smoke check and the benchmark's CPU-baseline leg do. The oracle
shares no code with the HIP library: it is compiled from its own C source with
gcc and loaded here through ctypes, on host (numpy) buffers.

Every function follows the paper's Algorithm 1 (appendix) and Section 3.1/3.2;
the C file cites the step each part implements.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ciera_oracle.c")
_LIB = os.path.join(_HERE, "libciera_oracle.so")

_u8p = ctypes.POINTER(ctypes.c_uint8)
_u16p = ctypes.POINTER(ctypes.c_uint16)
_u32p = ctypes.POINTER(ctypes.c_uint32)
_u64p = ctypes.POINTER(ctypes.c_uint64)
_f64p = ctypes.POINTER(ctypes.c_double)

HEADER_BYTES = 64


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, no vector intrinsics)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call([
            "gcc", "-O2", "-std=c99", "-Wall", "-Wextra", "-fPIC", "-shared",
            "-o", tmp, _SRC,
        ])
        os.replace(tmp, _LIB)
    return _LIB


def _bind(lib):
    lib.oracle_encoded_bound.restype = ctypes.c_uint64
    lib.oracle_encoded_bound.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
    lib.oracle_split.restype = None
    lib.oracle_split.argtypes = [_u16p, ctypes.c_uint64, _u8p, _u8p]
    lib.oracle_encode.restype = ctypes.c_uint64
    lib.oracle_encode.argtypes = [_u16p, _u8p, ctypes.c_uint64,
                                  ctypes.c_uint64, ctypes.c_int, _u8p,
                                  ctypes.c_uint64]
    lib.oracle_decode.restype = ctypes.c_int
    lib.oracle_decode.argtypes = [_u8p, ctypes.c_uint64, _u8p, _u16p]
    lib.oracle_decode_gathered.restype = ctypes.c_int
    lib.oracle_decode_gathered.argtypes = [_u8p, _u64p, ctypes.c_uint64,
                                           ctypes.c_uint64, _u16p, _u8p]
    lib.oracle_update_cache.restype = ctypes.c_int
    lib.oracle_update_cache.argtypes = [_u8p, _u8p, ctypes.c_uint64]
    for fn in (lib.oracle_gain, lib.oracle_gain_f16):
        fn.restype = ctypes.c_double
        fn.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_double,
                       ctypes.c_uint64, ctypes.c_double, ctypes.c_double,
                       ctypes.c_double, ctypes.c_double, ctypes.c_double,
                       ctypes.c_int, ctypes.c_double]
    lib.oracle_select.restype = ctypes.c_uint64
    lib.oracle_select.argtypes = [_f64p, _f64p, ctypes.c_uint64,
                                  ctypes.c_double, ctypes.c_int, _u8p]
    lib.oracle_sm64_mix.restype = ctypes.c_uint64
    lib.oracle_sm64_mix.argtypes = [ctypes.c_uint64]
    lib.oracle_block_hash.restype = None
    lib.oracle_block_hash.argtypes = [_u8p, ctypes.c_uint64, _u64p]
    lib.oracle_hash_blocks.restype = ctypes.c_int
    lib.oracle_hash_blocks.argtypes = [_u16p, ctypes.c_uint64,
                                       ctypes.c_uint64, _u64p]
    lib.oracle_ans_normalize.restype = None
    lib.oracle_ans_normalize.argtypes = [_u64p, _u32p]
    lib.oracle_ans_encode_chunk.restype = ctypes.c_uint64
    lib.oracle_ans_encode_chunk.argtypes = [_u8p, ctypes.c_uint64, _u32p, _u8p]
    lib.oracle_ans_decode_chunk.restype = ctypes.c_int
    lib.oracle_ans_decode_chunk.argtypes = [_u8p, ctypes.c_uint64,
                                            ctypes.c_uint64, _u32p, _u8p,
                                            _u64p]
    lib.oracle_ans_section_bound.restype = ctypes.c_uint64
    lib.oracle_ans_section_bound.argtypes = [ctypes.c_uint64]
    lib.oracle_ans_code_section.restype = ctypes.c_uint64
    lib.oracle_ans_code_section.argtypes = [_u8p, ctypes.c_uint64, _u8p]
    lib.oracle_ans_decode_section.restype = ctypes.c_int
    lib.oracle_ans_decode_section.argtypes = [_u8p, ctypes.c_uint64,
                                              ctypes.c_uint64, _u8p]
    lib.oracle_ans_code_shard.restype = ctypes.c_uint64
    lib.oracle_ans_code_shard.argtypes = [_u8p, ctypes.c_uint64]
    lib.oracle_split_f16.restype = None
    lib.oracle_split_f16.argtypes = [_u16p, ctypes.c_uint64, _u8p, _u8p, _u8p]
    lib.oracle_encoded_bound_f16.restype = ctypes.c_uint64
    lib.oracle_encoded_bound_f16.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
    lib.oracle_encode_f16.restype = ctypes.c_uint64
    lib.oracle_encode_f16.argtypes = [_u16p, _u8p, ctypes.c_uint64,
                                      ctypes.c_uint64, ctypes.c_int, _u8p,
                                      ctypes.c_uint64]
    lib.oracle_decode_f16.restype = ctypes.c_int
    lib.oracle_decode_f16.argtypes = [_u8p, ctypes.c_uint64, _u8p, _u16p]
    lib.oracle_update_cache_f16.restype = ctypes.c_int
    lib.oracle_update_cache_f16.argtypes = [_u8p, _u8p, ctypes.c_uint64]
    lib.oracle_encode_hashed.restype = ctypes.c_uint64
    lib.oracle_encode_hashed.argtypes = [_u16p, _u64p, _u64p, ctypes.c_uint64,
                                         ctypes.c_uint64, _u8p,
                                         ctypes.c_uint64]
    return lib


def _ptr(a: np.ndarray, typ):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(typ)


class Oracle:
    """The oracle's functions bound to one compiled library (the default one,
    or a copy built from another source, as the mutation tests do)."""

    def __init__(self, lib_path: str):
        self._lib = _bind(ctypes.CDLL(lib_path))

    def encoded_bound(self, n: int, B: int) -> int:
        return int(self._lib.oracle_encoded_bound(n, B))

    def split(self, w: np.ndarray):
        """Algorithm 1 SplitExpMant: (exponent bytes, sign+mantissa bytes)."""
        w = np.ascontiguousarray(w, dtype=np.uint16)
        e = np.empty(w.size, np.uint8)
        sm = np.empty(w.size, np.uint8)
        self._lib.oracle_split(_ptr(w, _u16p), w.size, _ptr(e, _u8p),
                               _ptr(sm, _u8p))
        return e, sm

    def encode(self, w: np.ndarray, cache, B: int,
               raw: bool = False) -> np.ndarray:
        """Encode one shard; returns the encoded bytes (exactly ``total``
        long). The output buffer starts filled with 0xA5, so a byte the
        oracle forgets to write shows up."""
        w = np.ascontiguousarray(w, dtype=np.uint16).ravel()
        n = w.size
        cap = self.encoded_bound(n, B)
        out = np.full(cap, 0xA5, np.uint8)
        if cache is None:
            cptr = ctypes.cast(None, _u8p)
        else:
            cache = np.ascontiguousarray(cache, dtype=np.uint8).ravel()
            assert cache.size == n
            cptr = _ptr(cache, _u8p)
        total = self._lib.oracle_encode(_ptr(w, _u16p), cptr, n, B, int(raw),
                                        _ptr(out, _u8p), cap)
        if total == 0 or total > cap:
            raise ValueError("oracle_encode rejected its arguments")
        return out[:total].copy()

    def decode(self, enc: np.ndarray, n: int, cache: np.ndarray):
        """Decode one shard; ``cache`` is updated in place. Returns values."""
        enc = np.ascontiguousarray(enc, dtype=np.uint8)
        assert cache.dtype == np.uint8 and cache.flags["C_CONTIGUOUS"]
        out = np.empty(n, np.uint16)
        rc = self._lib.oracle_decode(_ptr(enc, _u8p), n, _ptr(cache, _u8p),
                                     _ptr(out, _u16p))
        if rc:
            raise ValueError(f"oracle_decode: bad shard ({rc})")
        return out

    def decode_gathered(self, gathered: np.ndarray, offsets, n_s: int,
                        cache: np.ndarray):
        gathered = np.ascontiguousarray(gathered, dtype=np.uint8)
        offs = np.ascontiguousarray(offsets, dtype=np.uint64)
        R = offs.size
        assert cache.size == R * n_s and cache.flags["C_CONTIGUOUS"]
        out = np.empty(R * n_s, np.uint16)
        rc = self._lib.oracle_decode_gathered(
            _ptr(gathered, _u8p), _ptr(offs, _u64p), R, n_s,
            _ptr(out, _u16p), _ptr(cache, _u8p))
        if rc:
            raise ValueError(f"oracle_decode_gathered: bad shard ({rc})")
        return out

    def update_cache(self, cache: np.ndarray, enc: np.ndarray, n: int):
        enc = np.ascontiguousarray(enc, dtype=np.uint8)
        assert cache.dtype == np.uint8 and cache.flags["C_CONTIGUOUS"]
        rc = self._lib.oracle_update_cache(_ptr(cache, _u8p), _ptr(enc, _u8p),
                                           n)
        if rc:
            raise ValueError(f"oracle_update_cache: bad shard ({rc})")

    def gain(self, n: int, B: int, q: float, R: int, alpha_s: float,
             bus_bw_Bps: float, t_hash_s: float = 0.0, t_cmp_s: float = 0.0,
             t_decmp_s: float = 0.0, overlapped: bool = True,
             header_bytes: float = HEADER_BYTES, fp16: bool = False) -> float:
        fn = self._lib.oracle_gain_f16 if fp16 else self._lib.oracle_gain
        return float(fn(n, B, q, R, alpha_s, bus_bw_Bps, t_hash_s, t_cmp_s,
                        t_decmp_s, int(overlapped), header_bytes))

    def should_compress(self, *args, **kw) -> bool:
        """Section 3.2: keep a shard only when its gain is positive."""
        return self.gain(*args, **kw) > 0.0

    def select(self, gains, mems, budget: float,
               stop_at_first_misfit: bool = False):
        g = np.ascontiguousarray(gains, dtype=np.float64)
        m = np.ascontiguousarray(mems, dtype=np.float64)
        sel = np.zeros(g.size, np.uint8)
        self._lib.oracle_select(_ptr(g, _f64p), _ptr(m, _f64p), g.size,
                                budget, int(stop_at_first_misfit),
                                _ptr(sel, _u8p))
        return sel.astype(bool)

    # ---- sender-side block hash (Section 3.1, Hash128 / HashCache) ----

    def sm64_mix(self, z: int) -> int:
        return int(self._lib.oracle_sm64_mix(z))

    def block_hash(self, e: np.ndarray):
        e = np.ascontiguousarray(e, dtype=np.uint8).ravel()
        h = np.zeros(2, np.uint64)
        self._lib.oracle_block_hash(_ptr(e, _u8p), e.size, _ptr(h, _u64p))
        return int(h[0]), int(h[1])

    def hash_blocks(self, w: np.ndarray, B: int) -> np.ndarray:
        """HashCache of a shard: uint64[2 * ceil(n/B)], (H_0, H_1) per block."""
        w = np.ascontiguousarray(w, dtype=np.uint16).ravel()
        nb = -(-w.size // B)
        h = np.zeros(max(2 * nb, 1), np.uint64)
        if self._lib.oracle_hash_blocks(_ptr(w, _u16p), w.size, B,
                                        _ptr(h, _u64p)):
            raise ValueError("oracle_hash_blocks rejected its arguments")
        return h[:2 * nb].copy()

    def encode_hashed(self, w: np.ndarray, hash_in: np.ndarray, B: int):
        """Encode against a HashCache; returns (encoded bytes, new HashCache)."""
        w = np.ascontiguousarray(w, dtype=np.uint16).ravel()
        n = w.size
        nb = -(-n // B)
        hin = np.ascontiguousarray(hash_in, dtype=np.uint64).ravel()
        assert hin.size == 2 * nb
        hin = np.concatenate([hin, np.zeros(1, np.uint64)])
        hout = np.full(2 * nb + 1, 0xA5A5A5A5A5A5A5A5, np.uint64)
        cap = self.encoded_bound(n, B)
        out = np.full(cap, 0xA5, np.uint8)
        total = self._lib.oracle_encode_hashed(
            _ptr(w, _u16p), _ptr(hin, _u64p), _ptr(hout, _u64p), n, B,
            _ptr(out, _u8p), cap)
        if total == 0 or total > cap:
            raise ValueError("oracle_encode_hashed rejected its arguments")
        return out[:total].copy(), hout[:2 * nb].copy()

    # ---- rANS on the exception section (Section 3.1) ----

    def ans_normalize(self, hist) -> np.ndarray:
        h = np.ascontiguousarray(hist, dtype=np.uint64)
        assert h.size == 256
        f = np.zeros(256, np.uint32)
        self._lib.oracle_ans_normalize(_ptr(h, _u64p), _ptr(f, _u32p))
        return f

    def ans_encode_chunk(self, sym, freq) -> np.ndarray:
        sym = np.ascontiguousarray(sym, dtype=np.uint8).ravel()
        f = np.ascontiguousarray(freq, dtype=np.uint32)
        buf = np.full(256 + 2 * sym.size, 0xA5, np.uint8)
        nb = self._lib.oracle_ans_encode_chunk(_ptr(sym, _u8p), sym.size,
                                               _ptr(f, _u32p), _ptr(buf, _u8p))
        return buf[:nb].copy()

    def ans_decode_chunk(self, stream, length, freq):
        """Returns (symbols, bytes consumed); raises on a malformed stream."""
        st = np.ascontiguousarray(stream, dtype=np.uint8)
        f = np.ascontiguousarray(freq, dtype=np.uint32)
        out = np.zeros(max(length, 1), np.uint8)
        used = np.zeros(1, np.uint64)
        rc = self._lib.oracle_ans_decode_chunk(
            _ptr(st, _u8p), st.size, length, _ptr(f, _u32p), _ptr(out, _u8p),
            _ptr(used, _u64p))
        if rc:
            raise ValueError("oracle_ans_decode_chunk: malformed stream")
        return out[:length].copy(), int(used[0])

    def ans_code_section(self, exc) -> np.ndarray:
        exc = np.ascontiguousarray(exc, dtype=np.uint8).ravel()
        cap = int(self._lib.oracle_ans_section_bound(exc.size))
        sec = np.full(cap, 0xA5, np.uint8)
        C = self._lib.oracle_ans_code_section(_ptr(exc, _u8p), exc.size,
                                              _ptr(sec, _u8p))
        return sec[:C].copy()

    def ans_decode_section(self, section, E) -> np.ndarray:
        sec = np.ascontiguousarray(section, dtype=np.uint8)
        out = np.zeros(max(E, 1), np.uint8)
        if self._lib.oracle_ans_decode_section(_ptr(sec, _u8p), sec.size, E,
                                               _ptr(out, _u8p)):
            raise ValueError("oracle_ans_decode_section: malformed section")
        return out[:E].copy()

    def ans_code(self, enc: np.ndarray, n: int) -> np.ndarray:
        """An encoded shard with its exception section rANS-coded when that
        is smaller (mode 2); otherwise the same bytes."""
        buf = np.array(enc, dtype=np.uint8, copy=True)
        total = self._lib.oracle_ans_code_shard(_ptr(buf, _u8p), n)
        if total == 0:
            raise ValueError("oracle_ans_code_shard: bad shard")
        return buf[:total].copy()

    # ---- FP16 shards (Table 2's second precision) ----

    def split_f16(self, w):
        """(5-bit exponents, low mantissa bytes, sign<<2 | mantissa bits 9..8)"""
        w = np.ascontiguousarray(w, dtype=np.uint16).ravel()
        e, lo, hi = (np.empty(w.size, np.uint8) for _ in range(3))
        self._lib.oracle_split_f16(_ptr(w, _u16p), w.size, _ptr(e, _u8p),
                                   _ptr(lo, _u8p), _ptr(hi, _u8p))
        return e, lo, hi

    def encoded_bound_f16(self, n, B):
        return int(self._lib.oracle_encoded_bound_f16(n, B))

    def encode_f16(self, w, cache, B, raw=False):
        w = np.ascontiguousarray(w, dtype=np.uint16).ravel()
        n = w.size
        cap = self.encoded_bound_f16(n, B)
        out = np.full(cap, 0xA5, np.uint8)
        if cache is None:
            cptr = ctypes.cast(None, _u8p)
        else:
            cache = np.ascontiguousarray(cache, dtype=np.uint8).ravel()
            assert cache.size == n
            cptr = _ptr(cache, _u8p)
        total = self._lib.oracle_encode_f16(_ptr(w, _u16p), cptr, n, B,
                                            int(raw), _ptr(out, _u8p), cap)
        if total == 0 or total > cap:
            raise ValueError("oracle_encode_f16 rejected its arguments")
        return out[:total].copy()

    def decode_f16(self, enc, n, cache):
        enc = np.ascontiguousarray(enc, dtype=np.uint8)
        assert cache.dtype == np.uint8 and cache.flags["C_CONTIGUOUS"]
        out = np.empty(n, np.uint16)
        if self._lib.oracle_decode_f16(_ptr(enc, _u8p), n, _ptr(cache, _u8p),
                                       _ptr(out, _u16p)):
            raise ValueError("oracle_decode_f16: bad shard")
        return out

    def update_cache_f16(self, cache, enc, n):
        enc = np.ascontiguousarray(enc, dtype=np.uint8)
        if self._lib.oracle_update_cache_f16(_ptr(cache, _u8p),
                                             _ptr(enc, _u8p), n):
            raise ValueError("oracle_update_cache_f16: bad shard")

    def decode_gathered_f16(self, gathered, offsets, n_s, cache):
        out = np.empty(len(offsets) * n_s, np.uint16)
        for j, off in enumerate(offsets):
            c = cache[j * n_s:(j + 1) * n_s]
            cj = np.ascontiguousarray(c)
            out[j * n_s:(j + 1) * n_s] = self.decode_f16(
                np.asarray(gathered)[int(off):], n_s, cj)
            cache[j * n_s:(j + 1) * n_s] = cj
        return out

    header = staticmethod(lambda enc: header(enc))


_default = None


def _oracle() -> Oracle:
    global _default
    if _default is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _default = Oracle(_LIB)
    return _default


def encoded_bound(n, B):
    return _oracle().encoded_bound(n, B)


def split(w):
    return _oracle().split(w)


def encode(w, cache, B, raw=False):
    return _oracle().encode(w, cache, B, raw)


def decode(enc, n, cache):
    return _oracle().decode(enc, n, cache)


def decode_gathered(gathered, offsets, n_s, cache):
    return _oracle().decode_gathered(gathered, offsets, n_s, cache)


def update_cache(cache, enc, n):
    return _oracle().update_cache(cache, enc, n)


def gain(*args, **kw):
    return _oracle().gain(*args, **kw)


def should_compress(*args, **kw):
    return _oracle().should_compress(*args, **kw)


def select(gains, mems, budget, stop_at_first_misfit=False):
    return _oracle().select(gains, mems, budget, stop_at_first_misfit)


def sm64_mix(z):
    return _oracle().sm64_mix(z)


def block_hash(e):
    return _oracle().block_hash(e)


def hash_blocks(w, B):
    return _oracle().hash_blocks(w, B)


def encode_hashed(w, hash_in, B):
    return _oracle().encode_hashed(w, hash_in, B)


def ans_normalize(hist):
    return _oracle().ans_normalize(hist)


def ans_encode_chunk(sym, freq):
    return _oracle().ans_encode_chunk(sym, freq)


def ans_decode_chunk(stream, length, freq):
    return _oracle().ans_decode_chunk(stream, length, freq)


def ans_code_section(exc):
    return _oracle().ans_code_section(exc)


def ans_decode_section(section, E):
    return _oracle().ans_decode_section(section, E)


def ans_code(enc, n):
    return _oracle().ans_code(enc, n)


# ---- header fields, read straight from the bytes (no oracle arithmetic) ----

def header(enc: np.ndarray) -> dict:
    h = np.ascontiguousarray(enc[:HEADER_BYTES], dtype=np.uint8)
    u64 = h.view(np.uint64)
    return {
        "magic": int(h[0:4].view(np.uint32)[0]),
        "version": int(h[4:6].view(np.uint16)[0]),
        "mode": int(h[6:8].view(np.uint16)[0]),
        "B": int(h[8:12].view(np.uint32)[0]),
        "dtype": int(h[12:16].view(np.uint32)[0]),
        "n": int(u64[2]),
        "changed_blocks": int(u64[3]),
        "E": int(u64[4]),
        "P": int(u64[5]),
        "total": int(u64[6]),
    }


def split_f16(w):
    return _oracle().split_f16(w)


def encoded_bound_f16(n, B):
    return _oracle().encoded_bound_f16(n, B)


def encode_f16(w, cache, B, raw=False):
    return _oracle().encode_f16(w, cache, B, raw)


def decode_f16(enc, n, cache):
    return _oracle().decode_f16(enc, n, cache)


def update_cache_f16(cache, enc, n):
    return _oracle().update_cache_f16(cache, enc, n)


def decode_gathered_f16(gathered, offsets, n_s, cache):
    return _oracle().decode_gathered_f16(gathered, offsets, n_s, cache)
