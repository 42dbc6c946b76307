"""ctypes binding of libciera (the C ABI in include/ciera.h).

Argument marshalling only: every function forwards to the library call of the
same name, and every step of the codec runs in the library's HIP kernels. The
``*_t`` helpers accept torch tensors and pass their device pointers and the
current HIP stream. Opening the library fails loudly when it is not built;
there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libciera.so")

OK, EINVAL, ENOSPC, EUNSUPPORTED, EFORMAT, EHIP = 0, -1, -2, -3, -4, -5
DEVERR_FORMAT, DEVERR_ALIGN, DEVERR_BOUNDS, DEVERR_NOSPACE = 1, 2, 4, 8
ENC_RAW = 0x1
FP16 = 0x2
ENC_UPDATE_CACHE = 0x4
WS_ANS = 0x1
SELECT_STOP_AT_MISFIT = 0x1
HEADER_BYTES = 64
STATUS_NAMES = {OK: "OK", EINVAL: "EINVAL", ENOSPC: "ENOSPC",
                EUNSUPPORTED: "EUNSUPPORTED", EFORMAT: "EFORMAT",
                EHIP: "EHIP"}


class CieraError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} returned {STATUS_NAMES.get(code, code)}")
        self.code = code


class ShardStats(ctypes.Structure):
    _fields_ = [("n_elems", ctypes.c_uint64), ("block_elems", ctypes.c_uint32),
                ("flags", ctypes.c_uint32), ("q", ctypes.c_double)]


class CostModel(ctypes.Structure):
    _fields_ = [("world_size", ctypes.c_uint32), ("alpha_s", ctypes.c_double),
                ("bus_bw_Bps", ctypes.c_double), ("t_hash_s", ctypes.c_double),
                ("t_cmp_s", ctypes.c_double), ("t_decmp_s", ctypes.c_double),
                ("header_bytes", ctypes.c_double), ("overlapped", ctypes.c_int)]


_vp, _u64, _u32, _i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int
_SIGS = {
    "ciera_encoded_bound": (_u64, [_u64, _u32, _u32]),
    "ciera_workspace_bytes": (_u64, [_u64, _u32, _u32, _u32]),
    "ciera_workspace_init": (_i32, [_vp, _u64, _vp]),
    "ciera_workspace_error": (_i32, [_vp, ctypes.POINTER(_u32), _i32, _vp]),
    "ciera_encode": (_i32, [_vp, _vp, _u64, _u32, _u32, _vp, _u64, _vp, _vp,
                            _u64, _vp]),
    "ciera_decode_gathered": (_i32, [_vp, _u64, _vp, _u32, _u64, _u32, _u32,
                                     _vp, _vp, _vp, _u64, _vp]),
    "ciera_update_cache": (_i32, [_vp, _vp, _u64, _u64, _u32, _u32, _vp, _u64,
                                  _vp]),
    "ciera_decode_gathered_noalloc": (_i32, [_vp, _u64, _vp, _u32, _u64,
                                             _u32, _u32, _vp, _vp, _vp,
                                             _vp]),
    "ciera_ans_code": (_i32, [_vp, _u64, _u32, _vp, _vp, _u64, _vp]),
    "ciera_hash_blocks": (_i32, [_vp, _u64, _u32, _vp, _vp]),
    "ciera_encode_hashed": (_i32, [_vp, _vp, _vp, _u64, _u32, _vp, _u64, _vp,
                                   _vp, _u64, _vp]),
    "ciera_should_compress": (_i32, [ctypes.POINTER(ShardStats),
                                     ctypes.POINTER(CostModel),
                                     ctypes.POINTER(ctypes.c_double)]),
    "ciera_select": (_i32, [ctypes.POINTER(ctypes.c_double),
                            ctypes.POINTER(ctypes.c_double), _u64,
                            ctypes.c_double, _u32,
                            ctypes.POINTER(ctypes.c_uint8)]),
}
EXPORTED = tuple(_SIGS)

_lib = None


def lib():
    """Open libciera.so (once). Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2609_04609_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(handle, name)
            f.restype, f.argtypes = res, args
        _lib = handle
    return _lib


def _check(fn, rc):
    if rc < 0:
        raise CieraError(fn, rc)
    return rc


# ---- the C ABI, name for name (pointers and the stream as integers) ----

def ciera_encoded_bound(n_elems, block_elems, flags=0):
    return lib().ciera_encoded_bound(n_elems, block_elems, flags)


def ciera_workspace_bytes(n_elems, nshards, block_elems, flags=0):
    return lib().ciera_workspace_bytes(n_elems, nshards, block_elems, flags)


def ciera_workspace_init(workspace, workspace_bytes, stream):
    return lib().ciera_workspace_init(workspace, workspace_bytes, stream)


def ciera_workspace_error(workspace, clear, stream):
    err = _u32(0)
    rc = lib().ciera_workspace_error(workspace, ctypes.byref(err), clear, stream)
    _check("ciera_workspace_error", rc)
    return err.value


def ciera_encode(w_new, exp_cache, n_elems, block_elems, flags, out,
                 out_capacity, out_bytes, workspace, workspace_bytes, stream):
    return lib().ciera_encode(w_new, exp_cache, n_elems, block_elems, flags,
                              out, out_capacity, out_bytes, workspace,
                              workspace_bytes, stream)


def ciera_decode_gathered(gathered, gathered_bytes, shard_offsets, nshards,
                          shard_elems, block_elems, out, exp_cache, workspace,
                          workspace_bytes, stream, flags=0):
    """The C call of the same name; `flags` (0 or FP16) comes last here."""
    return lib().ciera_decode_gathered(gathered, gathered_bytes,
                                       shard_offsets, nshards, shard_elems,
                                       block_elems, flags, out, exp_cache,
                                       workspace, workspace_bytes, stream)


def ciera_decode_gathered_noalloc(gathered, gathered_bytes, shard_offsets,
                                  nshards, shard_elems, block_elems, out,
                                  exp_cache, err, stream, flags=0):
    """The C call of the same name; `flags` (0 or FP16) comes last here."""
    return lib().ciera_decode_gathered_noalloc(
        gathered, gathered_bytes, shard_offsets, nshards, shard_elems,
        block_elems, flags, out, exp_cache, err, stream)


def ciera_update_cache(exp_cache, encoded, encoded_bytes, n_elems,
                       block_elems, workspace, workspace_bytes, stream,
                       flags=0):
    """The C call of the same name; `flags` (0 or FP16) comes last here."""
    return lib().ciera_update_cache(exp_cache, encoded, encoded_bytes,
                                    n_elems, block_elems, flags, workspace,
                                    workspace_bytes, stream)


def ciera_ans_code(encoded, n_elems, block_elems, out_bytes, workspace,
                   workspace_bytes, stream):
    return lib().ciera_ans_code(encoded, n_elems, block_elems, out_bytes,
                                workspace, workspace_bytes, stream)


def ciera_hash_blocks(w, n_elems, block_elems, hash_cache, stream):
    return lib().ciera_hash_blocks(w, n_elems, block_elems, hash_cache, stream)


def ciera_encode_hashed(w_new, hash_in, hash_out, n_elems, block_elems, out,
                        out_capacity, out_bytes, workspace, workspace_bytes,
                        stream):
    return lib().ciera_encode_hashed(w_new, hash_in, hash_out, n_elems,
                                     block_elems, out, out_capacity, out_bytes,
                                     workspace, workspace_bytes, stream)


def ciera_should_compress(n_elems, block_elems, q, world_size, alpha_s,
                          bus_bw_Bps, t_hash_s=0.0, t_cmp_s=0.0, t_decmp_s=0.0,
                          header_bytes=float(HEADER_BYTES), overlapped=True,
                          fp16=False):
    """Returns (decision 0/1, gain in seconds)."""
    st = ShardStats(n_elems, block_elems, FP16 if fp16 else 0, q)
    cm = CostModel(world_size, alpha_s, bus_bw_Bps, t_hash_s, t_cmp_s,
                   t_decmp_s, header_bytes, int(overlapped))
    g = ctypes.c_double(0.0)
    rc = lib().ciera_should_compress(ctypes.byref(st), ctypes.byref(cm),
                                     ctypes.byref(g))
    _check("ciera_should_compress", rc)
    return rc, g.value


def ciera_select(gains, mems, budget_bytes, flags=0):
    n = len(gains)
    G = (ctypes.c_double * n)(*gains)
    M = (ctypes.c_double * n)(*mems)
    S = (ctypes.c_uint8 * n)()
    rc = lib().ciera_select(G, M, n, budget_bytes, flags, S)
    _check("ciera_select", rc)
    return [bool(x) for x in S]


# ---- tensor-level marshalling ----

def _stream():
    return torch.cuda.current_stream().cuda_stream


def _ptr(t):
    return 0 if t is None else t.data_ptr()


class Workspace:
    """Device workspace sized for a shard size, shard count and B; with
    ans=True also for rANS coding and decoding (CIERA_WS_ANS)."""

    def __init__(self, n_elems, nshards, block_elems, device="cuda",
                 ans=False):
        self.nbytes = int(ciera_workspace_bytes(n_elems, nshards, block_elems,
                                                WS_ANS if ans else 0))
        if self.nbytes == 0:
            raise CieraError("ciera_workspace_bytes", EUNSUPPORTED)
        self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=device)
        _check("ciera_workspace_init",
               ciera_workspace_init(self.buf.data_ptr(), self.nbytes,
                                    _stream()))

    @property
    def ptr(self):
        return self.buf.data_ptr()

    def error(self, clear=True):
        return ciera_workspace_error(self.ptr, int(clear), _stream())


def encode_t(w_bits, cache, block_elems, ws, out, raw=False, out_bytes=None,
             fp16=False, update_cache=False):
    """Encode a 1-D int16 bit tensor into ``out`` (uint8, bound-sized); with
    update_cache the cache is brought forward in place."""
    n = w_bits.numel()
    flags = ((ENC_RAW if raw else 0) | (FP16 if fp16 else 0) |
             (ENC_UPDATE_CACHE if update_cache else 0))
    rc = ciera_encode(_ptr(w_bits), _ptr(cache), n, block_elems, flags,
                      _ptr(out), out.numel(), _ptr(out_bytes), ws.ptr,
                      ws.nbytes, _stream())
    return _check("ciera_encode", rc)


def hash_blocks_t(w_bits, block_elems, hash_cache):
    """HashCache (int64 tensor of 2 * ceil(n/B) words) of a 1-D bit tensor."""
    rc = ciera_hash_blocks(_ptr(w_bits), w_bits.numel(), block_elems,
                           _ptr(hash_cache), _stream())
    return _check("ciera_hash_blocks", rc)


def encode_hashed_t(w_bits, hash_in, hash_out, block_elems, ws, out,
                    out_bytes=None):
    rc = ciera_encode_hashed(_ptr(w_bits), _ptr(hash_in), _ptr(hash_out),
                             w_bits.numel(), block_elems, _ptr(out),
                             out.numel(), _ptr(out_bytes), ws.ptr, ws.nbytes,
                             _stream())
    return _check("ciera_encode_hashed", rc)


def ans_code_t(encoded, n_elems, block_elems, ws, out_bytes=None):
    """rANS-code the exception section of an encoded shard in place."""
    rc = ciera_ans_code(_ptr(encoded), n_elems, block_elems, _ptr(out_bytes),
                        ws.ptr, ws.nbytes, _stream())
    return _check("ciera_ans_code", rc)


def _nbytes(t, nbytes):
    return t.numel() * t.element_size() if nbytes is None else nbytes


def decode_gathered_t(gathered, offsets, shard_elems, block_elems, out, cache,
                      ws, fp16=False, nbytes=None):
    """Decode the shards of a gathered uint8 tensor; its length bounds every
    shard unless ``nbytes`` gives another."""
    rc = ciera_decode_gathered(_ptr(gathered), _nbytes(gathered, nbytes),
                               _ptr(offsets), offsets.numel(), shard_elems,
                               block_elems, _ptr(out), _ptr(cache), ws.ptr,
                               ws.nbytes, _stream(), FP16 if fp16 else 0)
    return _check("ciera_decode_gathered", rc)


def decode_gathered_noalloc_t(gathered, offsets, shard_elems, block_elems,
                              out, cache, err, fp16=False, nbytes=None):
    """decode_gathered_t without a workspace; ``err`` is a one-element int32
    device tensor that receives the call's device error bits."""
    rc = ciera_decode_gathered_noalloc(
        _ptr(gathered), _nbytes(gathered, nbytes), _ptr(offsets),
        offsets.numel(), shard_elems, block_elems, _ptr(out), _ptr(cache),
        _ptr(err), _stream(), FP16 if fp16 else 0)
    return _check("ciera_decode_gathered_noalloc", rc)


def update_cache_t(cache, encoded, n_elems, block_elems, ws, fp16=False,
                   nbytes=None):
    rc = ciera_update_cache(_ptr(cache), _ptr(encoded),
                            _nbytes(encoded, nbytes), n_elems, block_elems,
                            ws.ptr, ws.nbytes, _stream(), FP16 if fp16 else 0)
    return _check("ciera_update_cache", rc)
