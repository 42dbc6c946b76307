"""Helpers shared by the GPU tests: seeded inputs on the device, host copies
for the oracle, gathered-buffer layout. No codec arithmetic here."""
import numpy as np
import torch

from paper_2609_04609_amd import ciera, synth

DEV = "cuda"


def host_u16(t):
    return t.cpu().numpy().view(np.uint16)


def host_u8(t):
    return t.cpu().numpy().view(np.uint8)


def dev_u8(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.uint8)).to(DEV)


def dev_bits(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.uint16).view(np.int16)).to(DEV)


def pair(n, seed, c=0.01, std=0.02):
    """(W bits, W' bits) on the GPU: W ~ N(0, std), W' = W with a Bernoulli(c)
    set of exponents moved by +-1."""
    w = synth.normal_bf16_bits(n, std, seed, DEV)
    w2 = synth.forced_bernoulli_bits(w, c, seed + 1)
    return w, w2


def gpu_encode(w2, cache, B, ws=None, raw=False):
    n = w2.numel()
    if ws is None:
        ws = ciera.Workspace(n, 1, B)
    cap = int(ciera.ciera_encoded_bound(n, B))
    out = torch.full((cap,), 0xA5, dtype=torch.uint8, device=DEV)
    nbytes = torch.zeros(1, dtype=torch.int64, device=DEV)
    ciera.encode_t(w2, None if raw else cache, B, ws, out, raw=raw,
                   out_bytes=nbytes)
    torch.cuda.synchronize()
    total = int(nbytes.item())
    return out, total, ws


def gather(encs):
    """Place encoded shards (host uint8 arrays) back to back: the one-GPU
    stand-in for the Allgather output."""
    offs = np.cumsum([0] + [e.size for e in encs[:-1]]).astype(np.uint64)
    return np.concatenate(encs), offs


def check_fused_update(orc, w2, cache_h, B, expect, ws, fp16=False, msg=""):
    """Encode W' with the fused cache update (CIERA_ENC_UPDATE_CACHE) on a
    device copy of cache_h: the bytes must equal `expect` (the oracle's
    encoding) and the cache afterwards the oracle's update of cache_h from
    those bytes, the exponents of W'."""
    n = w2.numel()
    flags = ciera.FP16 if fp16 else 0
    cache = dev_u8(cache_h)
    cap = int(ciera.ciera_encoded_bound(n, B, flags))
    out = torch.full((cap,), 0xA5, dtype=torch.uint8, device=DEV)
    nbytes = torch.zeros(1, dtype=torch.int64, device=DEV)
    ciera.encode_t(w2, cache, B, ws, out, out_bytes=nbytes, fp16=fp16,
                   update_cache=True)
    torch.cuda.synchronize()
    total = int(nbytes.item())
    assert total == expect.size, msg
    np.testing.assert_array_equal(host_u8(out[:total]), expect, err_msg=msg)
    c_o = np.array(cache_h, dtype=np.uint8, copy=True)
    (orc.update_cache_f16 if fp16 else orc.update_cache)(c_o, expect, n)
    np.testing.assert_array_equal(host_u8(cache), c_o, err_msg=msg)

