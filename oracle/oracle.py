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


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
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
        lib.oracle_gain.restype = ctypes.c_double
        lib.oracle_gain.argtypes = [ctypes.c_uint64, ctypes.c_uint64,
                                    ctypes.c_double, ctypes.c_uint64,
                                    ctypes.c_double, ctypes.c_double,
                                    ctypes.c_double, ctypes.c_double,
                                    ctypes.c_double, ctypes.c_int,
                                    ctypes.c_double]
        lib.oracle_select.restype = ctypes.c_uint64
        lib.oracle_select.argtypes = [_f64p, _f64p, ctypes.c_uint64,
                                      ctypes.c_double, ctypes.c_int, _u8p]
        _lib = lib
    return _lib


def _ptr(a: np.ndarray, typ):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(typ)


def encoded_bound(n: int, B: int) -> int:
    return int(_load().oracle_encoded_bound(n, B))


def split(w: np.ndarray):
    """Algorithm 1 SplitExpMant: (exponent bytes, sign+mantissa bytes)."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    e = np.empty(w.size, np.uint8)
    sm = np.empty(w.size, np.uint8)
    _load().oracle_split(_ptr(w, _u16p), w.size, _ptr(e, _u8p), _ptr(sm, _u8p))
    return e, sm


def encode(w: np.ndarray, cache: np.ndarray | None, B: int,
           raw: bool = False) -> np.ndarray:
    """Encode one shard; returns the encoded bytes (exactly ``total`` long)."""
    w = np.ascontiguousarray(w, dtype=np.uint16).ravel()
    n = w.size
    cap = encoded_bound(n, B)
    out = np.empty(cap, np.uint8)
    if cache is None:
        cptr = ctypes.cast(None, _u8p)
    else:
        cache = np.ascontiguousarray(cache, dtype=np.uint8).ravel()
        assert cache.size == n
        cptr = _ptr(cache, _u8p)
    total = _load().oracle_encode(_ptr(w, _u16p), cptr, n, B, int(raw),
                                  _ptr(out, _u8p), cap)
    if total == 0:
        raise ValueError("oracle_encode rejected its arguments")
    return out[:total].copy()


def decode(enc: np.ndarray, n: int, cache: np.ndarray):
    """Decode one shard; ``cache`` is updated in place. Returns the values."""
    enc = np.ascontiguousarray(enc, dtype=np.uint8)
    assert cache.dtype == np.uint8 and cache.flags["C_CONTIGUOUS"]
    out = np.empty(n, np.uint16)
    rc = _load().oracle_decode(_ptr(enc, _u8p), n, _ptr(cache, _u8p),
                               _ptr(out, _u16p))
    if rc:
        raise ValueError(f"oracle_decode: bad shard ({rc})")
    return out


def decode_gathered(gathered: np.ndarray, offsets, n_s: int,
                    cache: np.ndarray):
    gathered = np.ascontiguousarray(gathered, dtype=np.uint8)
    offs = np.ascontiguousarray(offsets, dtype=np.uint64)
    R = offs.size
    assert cache.size == R * n_s and cache.flags["C_CONTIGUOUS"]
    out = np.empty(R * n_s, np.uint16)
    rc = _load().oracle_decode_gathered(_ptr(gathered, _u8p), _ptr(offs, _u64p),
                                        R, n_s, _ptr(out, _u16p),
                                        _ptr(cache, _u8p))
    if rc:
        raise ValueError(f"oracle_decode_gathered: bad shard ({rc})")
    return out


def update_cache(cache: np.ndarray, enc: np.ndarray, n: int) -> None:
    enc = np.ascontiguousarray(enc, dtype=np.uint8)
    assert cache.dtype == np.uint8 and cache.flags["C_CONTIGUOUS"]
    rc = _load().oracle_update_cache(_ptr(cache, _u8p), _ptr(enc, _u8p), n)
    if rc:
        raise ValueError(f"oracle_update_cache: bad shard ({rc})")


def gain(n: int, B: int, q: float, R: int, alpha_s: float, bus_bw_Bps: float,
         t_hash_s: float = 0.0, t_cmp_s: float = 0.0, t_decmp_s: float = 0.0,
         overlapped: bool = True, header_bytes: float = HEADER_BYTES) -> float:
    return float(_load().oracle_gain(n, B, q, R, alpha_s, bus_bw_Bps, t_hash_s,
                                     t_cmp_s, t_decmp_s, int(overlapped),
                                     header_bytes))


def should_compress(*args, **kw) -> bool:
    """Section 3.2: keep a shard only when its gain is positive."""
    return gain(*args, **kw) > 0.0


def select(gains, mems, budget: float, stop_at_first_misfit: bool = False):
    g = np.ascontiguousarray(gains, dtype=np.float64)
    m = np.ascontiguousarray(mems, dtype=np.float64)
    sel = np.zeros(g.size, np.uint8)
    _load().oracle_select(_ptr(g, _f64p), _ptr(m, _f64p), g.size, budget,
                          int(stop_at_first_misfit), _ptr(sel, _u8p))
    return sel.astype(bool)


# ---- header fields, read straight from the bytes (no oracle arithmetic) ----

def header(enc: np.ndarray) -> dict:
    h = np.ascontiguousarray(enc[:HEADER_BYTES], dtype=np.uint8)
    u64 = h.view(np.uint64)
    return {
        "magic": int(h[0:4].view(np.uint32)[0]),
        "version": int(h[4:6].view(np.uint16)[0]),
        "mode": int(h[6:8].view(np.uint16)[0]),
        "B": int(h[8:12].view(np.uint32)[0]),
        "n": int(u64[2]),
        "changed_blocks": int(u64[3]),
        "E": int(u64[4]),
        "P": int(u64[5]),
        "total": int(u64[6]),
    }
