"""fp16 shards on the GPU (the paper's second precision, Table 2) vs the CPU
oracle, byte for byte: encoded buffers (compressed and raw), gathered
decodes, the cache update, and a shard of the other value format refused.
All calls go through the C ABI."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

SIZES = [1, 7, 8, 9, 100, 511, 4097, 16385, 40000, 3 * 16384 + 17,
         32768 * 3 + 8, 262147]
BLOCKS = [16, 32, 64, 512, 1024, 4096]


@pytest.fixture(scope="module")
def gu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util
    from paper_2609_04609_amd import ciera
    ciera.lib()
    return gpu_util


def _pair(n, seed, c):
    from paper_2609_04609_amd import synth
    w = synth.normal_f16_bits(n, 0.02, seed)
    return w, synth.forced_bernoulli_f16_bits(w, c, seed + 1)


def _encode(gu, w2, cache, B, ws, raw=False):
    from paper_2609_04609_amd import ciera
    n = w2.numel()
    cap = int(ciera.ciera_encoded_bound(n, B, ciera.FP16))
    out = torch.full((cap,), 0xA5, dtype=torch.uint8, device="cuda")
    nbytes = torch.zeros(1, dtype=torch.int64, device="cuda")
    ciera.encode_t(w2, None if raw else cache, B, ws, out, raw=raw,
                   out_bytes=nbytes, fp16=True)
    torch.cuda.synchronize()
    total = int(nbytes.item())
    got = gu.host_u8(out)
    assert np.all(got[total:] == 0xA5)
    return got[:total]


@pytest.mark.parametrize("B", BLOCKS)
def test_encode_f16_matches_oracle(gu, orc, B):
    from paper_2609_04609_amd import ciera
    ws = ciera.Workspace(262147, 1, B)
    for i, n in enumerate(SIZES):
        w, w2 = _pair(n, 1000 * B + i, 0.002 * (1 + i % 4))
        cache_h = orc.split_f16(gu.host_u16(w))[0]
        got = _encode(gu, w2, gu.dev_u8(cache_h), B, ws)
        expect = orc.encode_f16(gu.host_u16(w2), cache_h, B)
        np.testing.assert_array_equal(got, expect, err_msg=f"n={n} B={B}")
        raw = _encode(gu, w2, None, B, ws, raw=True)
        np.testing.assert_array_equal(
            raw, orc.encode_f16(gu.host_u16(w2), None, B, raw=True))
        assert ws.error() == 0


def test_encode_f16_unaligned_and_every_exponent(gu, orc):
    """A shard starting one value into its buffer (element-wise loads), and a
    cache that disagrees everywhere (every block sent)."""
    from paper_2609_04609_amd import ciera
    B, n = 64, 70001
    ws = ciera.Workspace(n, 1, B)
    w, w2 = _pair(n + 1, 7, 0.01)
    w2u = w2[1:]
    assert w2u.data_ptr() % 16 != 0
    cache_h = orc.split_f16(gu.host_u16(w[1:]))[0]
    got = _encode(gu, w2u, gu.dev_u8(cache_h), B, ws)
    np.testing.assert_array_equal(got, orc.encode_f16(gu.host_u16(w2u),
                                                      cache_h, B))
    junk = (cache_h + 1) & 31
    got = _encode(gu, w2u, gu.dev_u8(junk), B, ws)
    expect = orc.encode_f16(gu.host_u16(w2u), junk, B)
    assert orc.header(expect)["E"] == n
    np.testing.assert_array_equal(got, expect)


@pytest.mark.parametrize("B", [16, 512, 4096])
@pytest.mark.parametrize("R,n", [(1, 1), (3, 16385), (4, 40000), (3, 81928),
                                 (5, 262147)])
def test_decode_gathered_f16_matches_oracle(gu, orc, B, R, n):
    _decode_f16_case(gu, orc, B, R, n)


def _decode_f16_case(gu, orc, B, R, n):
    from paper_2609_04609_amd import ciera
    ws_e = ciera.Workspace(n, 1, B)
    encs, caches, vals = [], [], []
    for j in range(R):
        w, w2 = _pair(n, 77 * B + 10 * R + j, 0.003)
        cache_h = orc.split_f16(gu.host_u16(w))[0]
        encs.append(_encode(gu, w2, gu.dev_u8(cache_h), B, ws_e,
                            raw=(j % 4 == 3)))
        caches.append(cache_h)
        vals.append(gu.host_u16(w2))
    g, offs = gu.gather(encs)
    cache0 = np.concatenate(caches)
    cache_o = cache0.copy()
    expect = orc.decode_gathered_f16(g, offs, n, cache_o)
    np.testing.assert_array_equal(expect, np.concatenate(vals))
    ws = ciera.Workspace(n, R, B)
    out = torch.full((R * n,), -1, dtype=torch.int16, device="cuda")
    cache = gu.dev_u8(cache0)
    offs_t = torch.from_numpy(offs.view(np.int64)).to("cuda")
    ciera.decode_gathered_t(gu.dev_u8(g), offs_t, n, B, out, cache, ws,
                            fp16=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u16(out), expect)
    np.testing.assert_array_equal(gu.host_u8(cache), cache_o)
    assert ws.error() == 0


def test_decode_f16_with_prefix_pass(gu, orc):
    """16 fp16 shards of 6,000,008 values at B = 16: large enough bitmaps
    that the decode scans the tile offsets in a pass of its own; equal to
    the oracle's decode of the same bytes and to W'."""
    _decode_f16_case(gu, orc, 16, 16, 6_000_008)


@pytest.mark.parametrize("B,n", [(16, 3 * 16384 + 17), (512, 3 * 16384 + 17),
                                 (4096, 3 * 16384 + 17),
                                 (16, 24_000_008)])  # the prefix pass
def test_update_cache_f16(gu, orc, B, n):
    from paper_2609_04609_amd import ciera
    ws = ciera.Workspace(n, 1, B)
    w, w2 = _pair(n, 9 + B, 0.004)
    cache_h = orc.split_f16(gu.host_u16(w))[0]
    enc = _encode(gu, w2, gu.dev_u8(cache_h), B, ws)
    c_o = cache_h.copy()
    orc.update_cache_f16(c_o, enc, n)
    cache = gu.dev_u8(cache_h)
    ciera.update_cache_t(cache, gu.dev_u8(enc), n, B, ws, fp16=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u8(cache), c_o)
    assert ws.error() == 0


def test_value_format_is_checked(gu, orc):
    """An fp16 shard given to the bf16 decode (and the other way round) is a
    format error; the shard is skipped and its output left alone."""
    from paper_2609_04609_amd import ciera
    B, n = 512, 40000
    ws = ciera.Workspace(n, 1, B)
    w, w2 = _pair(n, 3, 0.003)
    cache_h = orc.split_f16(gu.host_u16(w))[0]
    enc16 = _encode(gu, w2, gu.dev_u8(cache_h), B, ws)
    offs_t = torch.zeros(1, dtype=torch.int64, device="cuda")
    out = torch.full((n,), 5, dtype=torch.int16, device="cuda")
    ciera.decode_gathered_t(gu.dev_u8(enc16), offs_t, n, B, out,
                            gu.dev_u8(cache_h), ws)
    torch.cuda.synchronize()
    assert ws.error() == ciera.DEVERR_FORMAT
    assert torch.all(out == 5)
    wb, wb2 = gu.pair(n, 4)
    cb = orc.split(gu.host_u16(wb))[0]
    outb, total, _ = gu.gpu_encode(wb2, gu.dev_u8(cb), B)
    encb = gu.host_u8(outb)[:total]
    ciera.decode_gathered_t(gu.dev_u8(encb), offs_t, n, B, out,
                            gu.dev_u8(cb), ws, fp16=True)
    torch.cuda.synchronize()
    assert ws.error() == ciera.DEVERR_FORMAT
    assert torch.all(out == 5)


def test_encode_f16_with_cache_update(gu, orc):
    from paper_2609_04609_amd import ciera
    B, n = 512, 3 * 16384 + 17
    ws = ciera.Workspace(n, 1, B)
    w, w2 = _pair(n, 21, 0.004)
    cache_h = orc.split_f16(gu.host_u16(w))[0]
    expect = orc.encode_f16(gu.host_u16(w2), cache_h, B)
    c_o = cache_h.copy()
    orc.update_cache_f16(c_o, expect, n)
    cache = gu.dev_u8(cache_h)
    cap = int(ciera.ciera_encoded_bound(n, B, ciera.FP16))
    out = torch.full((cap,), 0xA5, dtype=torch.uint8, device="cuda")
    nbytes = torch.zeros(1, dtype=torch.int64, device="cuda")
    ciera.encode_t(w2, cache, B, ws, out, out_bytes=nbytes, fp16=True,
                   update_cache=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u8(out)[:int(nbytes.item())],
                                  expect)
    np.testing.assert_array_equal(gu.host_u8(cache), c_o)
