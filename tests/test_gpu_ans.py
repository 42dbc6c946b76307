"""rANS coding of the exception section on the GPU (Section 3.1: the changed
exponents travel ANS-coded) vs the CPU oracle, byte for byte: the recoded
shard (mode 2, or unchanged when coding does not pay), the decode of
gathered buffers mixing raw, compressed and coded shards, the cache update,
and the device error paths. All calls go through the C ABI."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

SIZES = [1, 100, 4097, 16385, 40000, 3 * 16384 + 17, 262147]
BLOCKS = [16, 64, 512, 4096]
RATES = [0.0, 0.001, 0.01, 0.05, 1.0]


@pytest.fixture(scope="module")
def gu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util
    from paper_2609_04609_amd import ciera
    ciera.lib()
    return gpu_util


def _gpu_coded(gu, w2, cache, B, ws):
    """GPU encode, then GPU rANS coding in place; returns (bytes, total)."""
    from paper_2609_04609_amd import ciera
    out, total0, _ = gu.gpu_encode(w2, cache, B, ws)
    nbytes = torch.full((1,), -1, dtype=torch.int64, device="cuda")
    ciera.ans_code_t(out, w2.numel(), B, ws, out_bytes=nbytes)
    torch.cuda.synchronize()
    total = int(nbytes.item())
    return gu.host_u8(out)[:total], total


@pytest.mark.parametrize("B", BLOCKS)
def test_ans_code_matches_oracle(gu, orc, B):
    from paper_2609_04609_amd import ciera
    ws = ciera.Workspace(262147, 1, B, ans=True)
    coded_seen = 0
    for i, n in enumerate(SIZES):
        for rate in RATES:
            w, w2 = gu.pair(n, 900 * B + 10 * i + int(rate * 100), c=rate)
            cache_h, _ = orc.split(gu.host_u16(w))
            got, total = _gpu_coded(gu, w2, gu.dev_u8(cache_h), B, ws)
            expect = orc.ans_code(orc.encode(gu.host_u16(w2), cache_h, B), n)
            assert total == expect.size, (n, B, rate)
            np.testing.assert_array_equal(got, expect,
                                          err_msg=f"n={n} B={B} c={rate}")
            coded_seen += orc.header(expect)["mode"] == 2
            assert ws.error() == 0
    assert coded_seen >= 5  # the coded path really ran


def _gather_mixed(gu, orc, n, B, R, seed):
    """R shards: some raw, some compressed, most rANS-coded (on the GPU)."""
    from paper_2609_04609_amd import ciera
    ws = ciera.Workspace(n, 1, B, ans=True)
    encs, caches, vals = [], [], []
    for j in range(R):
        w, w2 = gu.pair(n, seed + j, c=0.003 * (1 + j % 3))
        cache_h, _ = orc.split(gu.host_u16(w))
        if j % 5 == 1:
            out, total, _ = gu.gpu_encode(w2, None, B, ws, raw=True)
            enc = gu.host_u8(out)[:total]
        elif j % 5 == 2:
            out, total, _ = gu.gpu_encode(w2, gu.dev_u8(cache_h), B, ws)
            enc = gu.host_u8(out)[:total]
        else:
            enc, _ = _gpu_coded(gu, w2, gu.dev_u8(cache_h), B, ws)
        encs.append(enc)
        caches.append(cache_h)
        vals.append(gu.host_u16(w2))
    return encs, np.concatenate(caches), np.concatenate(vals)


@pytest.mark.parametrize("B", BLOCKS)
@pytest.mark.parametrize("R,n", [(1, 4097), (5, 40000), (6, 262147)])
def test_decode_mixed_gather_matches_oracle(gu, orc, B, R, n):
    from paper_2609_04609_amd import ciera
    encs, cache0, vals = _gather_mixed(gu, orc, n, B, R, 77 * B + R)
    if n >= 40000:  # smaller shards have too few exceptions to code
        assert any(orc.header(e)["mode"] == 2 for e in encs)
    g, offs = gu.gather(encs)
    cache_o = cache0.copy()
    expect = orc.decode_gathered(g, offs, n, cache_o)
    np.testing.assert_array_equal(expect, vals)
    ws = ciera.Workspace(n, R, B, ans=True)
    out = torch.full((R * n,), -1, dtype=torch.int16, device="cuda")
    cache = gu.dev_u8(cache0)
    offs_t = torch.from_numpy(offs.view(np.int64)).to("cuda")
    ciera.decode_gathered_t(gu.dev_u8(g), offs_t, n, B, out, cache, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u16(out), expect)
    np.testing.assert_array_equal(gu.host_u8(cache), cache_o)
    assert ws.error() == 0
    # idempotent
    ciera.decode_gathered_t(gu.dev_u8(g), offs_t, n, B, out, cache, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u16(out), expect)


@pytest.mark.parametrize("B", [16, 512, 4096])
def test_update_cache_on_coded_shards(gu, orc, B):
    from paper_2609_04609_amd import ciera
    n = 3 * 16384 + 17
    ws = ciera.Workspace(n, 1, B, ans=True)
    for seed in range(3):
        w, w2 = gu.pair(n, 300 + seed, c=0.004)
        cache_h, _ = orc.split(gu.host_u16(w))
        enc, _ = _gpu_coded(gu, w2, gu.dev_u8(cache_h), B, ws)
        assert orc.header(enc)["mode"] == 2
        c_o = cache_h.copy()
        orc.update_cache(c_o, enc, n)
        cache = gu.dev_u8(cache_h)
        ciera.update_cache_t(cache, gu.dev_u8(enc), n, B, ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(gu.host_u8(cache), c_o)
        assert ws.error() == 0


def test_ans_error_paths(gu, orc):
    """A coded shard met by a workspace without rANS room, and coded sections
    with a wrong frequency table, a flipped stream byte or a stream cut
    short: the device error word says so and every access stays in
    bounds."""
    from paper_2609_04609_amd import ciera
    B, n = 512, 70001
    ws = ciera.Workspace(n, 1, B, ans=True)
    w, w2 = gu.pair(n, 55, c=0.004)
    cache_h, _ = orc.split(gu.host_u16(w))
    enc, _ = _gpu_coded(gu, w2, gu.dev_u8(cache_h), B, ws)
    assert orc.header(enc)["mode"] == 2
    offs_t = torch.zeros(1, dtype=torch.int64, device="cuda")
    # no room: the shard is skipped, its output untouched
    ws_small = ciera.Workspace(n, 1, B)
    out = torch.full((n,), 7, dtype=torch.int16, device="cuda")
    ciera.decode_gathered_t(gu.dev_u8(enc), offs_t, n, B, out,
                            gu.dev_u8(cache_h), ws_small)
    torch.cuda.synchronize()
    assert ws_small.error() == ciera.DEVERR_NOSPACE
    assert torch.all(out == 7)
    # a buffer length 16 bytes short of the shard's total (the allocation is
    # the whole shard, so a missing check would still read mapped memory):
    # skipped by the rANS pass and the decode alike, output untouched
    cache_d = gu.dev_u8(cache_h)
    ciera.decode_gathered_t(gu.dev_u8(enc), offs_t, n, B, out, cache_d, ws,
                            nbytes=enc.size - 16)
    torch.cuda.synchronize()
    assert ws.error() == ciera.DEVERR_BOUNDS
    assert torch.all(out == 7)
    np.testing.assert_array_equal(gu.host_u8(cache_d), cache_h)
    a16 = lambda x: -(-x // 16) * 16
    sec = 64 + a16(n) + a16(-(-(-(-n // B)) // 8))
    # a frequency changed: the table no longer sums to 4096
    bad = enc.copy()
    bad[sec + 8 + 2 * 121] ^= 1
    ciera.decode_gathered_t(gu.dev_u8(bad), offs_t, n, B, out,
                            gu.dev_u8(cache_h), ws)
    torch.cuda.synchronize()
    assert ws.error() & ciera.DEVERR_FORMAT
    # a state of the first chunk flipped
    K = int(enc[sec:sec + 4].view(np.uint32)[0])
    bad = enc.copy()
    bad[sec + 520 + 4 * K + 4 * 7 + 1] ^= 0x40
    ciera.decode_gathered_t(gu.dev_u8(bad), offs_t, n, B, out,
                            gu.dev_u8(cache_h), ws)
    torch.cuda.synchronize()
    assert ws.error() & ciera.DEVERR_FORMAT
    # the first chunk's stream cut 4 bytes short: its decoder needs words
    # past the new end (taking padding or the next chunk's words instead)
    assert K >= 2
    bad = enc.copy()
    ends = bad[sec + 520:sec + 520 + 4 * K].view(np.uint32)
    ends[0] -= 4
    ciera.decode_gathered_t(gu.dev_u8(bad), offs_t, n, B, out,
                            gu.dev_u8(cache_h), ws)
    torch.cuda.synchronize()
    assert ws.error() & ciera.DEVERR_FORMAT
    # the good shard still decodes
    ciera.decode_gathered_t(gu.dev_u8(enc), offs_t, n, B, out,
                            gu.dev_u8(cache_h), ws)
    torch.cuda.synchronize()
    assert ws.error() == 0
    np.testing.assert_array_equal(gu.host_u16(out), gu.host_u16(w2))


def test_ans_code_is_deterministic_and_idempotent(gu, orc):
    from paper_2609_04609_amd import ciera
    B, n = 512, 262147
    ws = ciera.Workspace(n, 1, B, ans=True)
    w, w2 = gu.pair(n, 66, c=0.003)
    cache = gu.dev_u8(orc.split(gu.host_u16(w))[0])
    a, ta = _gpu_coded(gu, w2, cache, B, ws)
    b, tb = _gpu_coded(gu, w2, cache, B, ws)
    np.testing.assert_array_equal(a, b)
    # coding an already coded shard leaves it as it is
    buf = gu.dev_u8(np.concatenate([a, np.zeros(64, np.uint8)]))
    nbytes = torch.zeros(1, dtype=torch.int64, device="cuda")
    ciera.ans_code_t(buf, n, B, ws, out_bytes=nbytes)
    torch.cuda.synchronize()
    assert int(nbytes.item()) == ta
    np.testing.assert_array_equal(gu.host_u8(buf)[:ta], a)
