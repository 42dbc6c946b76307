"""Sender-side block hash on the GPU (Section 3.1, Hash128 / HashCache) vs the
CPU oracle, bit for bit: every block's two 64-bit hashes, and the encoded
bytes of the hashed encoder, which must also equal those of the exact-compare
encoder. All calls go through the C ABI."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

SIZES = [1, 7, 8, 9, 100, 511, 4097, 16383, 16384, 16385, 40000,
         3 * 16384 + 17, 32768 * 3 + 8, 262147]
BLOCKS = [16, 32, 64, 128, 512, 1024, 2048, 4096]


@pytest.fixture(scope="module")
def gu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util
    from paper_2609_04609_amd import ciera
    ciera.lib()
    return gpu_util


def _dev_u64(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.uint64).view(np.int64)
                            ).to("cuda")


def _host_u64(t):
    return t.cpu().numpy().view(np.uint64)


def _gpu_hash(w, B):
    from paper_2609_04609_amd import ciera
    nb = -(-w.numel() // B)
    h = torch.full((2 * nb + 2,), -1, dtype=torch.int64, device="cuda")
    ciera.hash_blocks_t(w, B, h)
    torch.cuda.synchronize()
    got = _host_u64(h)
    assert np.all(got[2 * nb:] == np.uint64(0xFFFFFFFFFFFFFFFF)), "wrote past"
    return got[:2 * nb]


def _gpu_encode_hashed(gu, w2, h_in, B, ws, in_place=False):
    from paper_2609_04609_amd import ciera
    n = w2.numel()
    cap = int(ciera.ciera_encoded_bound(n, B))
    out = torch.full((cap,), 0xA5, dtype=torch.uint8, device="cuda")
    nbytes = torch.zeros(1, dtype=torch.int64, device="cuda")
    hin = _dev_u64(h_in)
    hout = hin if in_place else torch.full_like(hin, -1)
    ciera.encode_hashed_t(w2, hin, hout, B, ws, out, out_bytes=nbytes)
    torch.cuda.synchronize()
    return gu.host_u8(out), int(nbytes.item()), _host_u64(hout)


@pytest.mark.parametrize("B", BLOCKS)
def test_hash_blocks_matches_oracle(gu, orc, B):
    for i, n in enumerate(SIZES):
        w, _ = gu.pair(n, 500 * B + i)
        got = _gpu_hash(w, B)
        np.testing.assert_array_equal(got, orc.hash_blocks(gu.host_u16(w), B),
                                      err_msg=f"n={n} B={B}")


@pytest.mark.parametrize("B", BLOCKS)
def test_encode_hashed_matches_oracle(gu, orc, B):
    from paper_2609_04609_amd import ciera
    ws = ciera.Workspace(262147, 1, B)
    for i, n in enumerate(SIZES):
        w, w2 = gu.pair(n, 700 * B + i, c=0.002 * (1 + i % 4))
        wh, w2h = gu.host_u16(w), gu.host_u16(w2)
        h_old = orc.hash_blocks(wh, B)
        expect, h_new = orc.encode_hashed(w2h, h_old, B)
        # the exact-compare wire, from the exponents of W
        cache_h, _ = orc.split(wh)
        np.testing.assert_array_equal(expect, orc.encode(w2h, cache_h, B))
        got, total, hout = _gpu_encode_hashed(gu, w2, h_old, B, ws,
                                              in_place=bool(i % 2))
        assert total == expect.size, (n, B)
        np.testing.assert_array_equal(got[:total], expect,
                                      err_msg=f"n={n} B={B}")
        assert np.all(got[total:] == 0xA5)
        np.testing.assert_array_equal(hout, h_new, err_msg=f"n={n} B={B}")
        assert ws.error() == 0


def test_hashed_edge_cases(gu, orc):
    """n = 0; an unaligned weight pointer (element-wise loads); a stored hash
    differing in one half only; every block changed."""
    from paper_2609_04609_amd import ciera
    B = 512
    ws = ciera.Workspace(1 << 18, 1, B)
    # n = 0: a header-only shard, no hash read or written
    w0 = torch.zeros(0, dtype=torch.int16, device="cuda")
    got, total, _ = _gpu_encode_hashed(gu, w0, np.zeros(0, np.uint64), B, ws)
    expect, _ = orc.encode_hashed(np.zeros(0, np.uint16), np.zeros(0, np.uint64), B)
    assert total == expect.size == 64
    np.testing.assert_array_equal(got[:total], expect)
    # unaligned: the shard starts one value into a buffer
    n = 70001
    w, w2 = gu.pair(n + 1, 91, c=0.003)
    w2u = w2[1:]
    assert w2u.data_ptr() % 16 != 0
    h_old = orc.hash_blocks(gu.host_u16(w[1:]), B)
    expect, h_new = orc.encode_hashed(gu.host_u16(w2u), h_old, B)
    got, total, hout = _gpu_encode_hashed(gu, w2u, h_old, B, ws)
    np.testing.assert_array_equal(got[:total], expect)
    np.testing.assert_array_equal(hout, h_new)
    np.testing.assert_array_equal(_gpu_hash(w2u, B), h_new)
    # one half of one stored hash altered: exactly that block is sent
    h_same = orc.hash_blocks(gu.host_u16(w2u), B)
    for half, blk in ((0, 3), (1, 100)):
        h2 = h_same.copy()
        h2[2 * blk + half] ^= np.uint64(1 << 63)
        expect, _ = orc.encode_hashed(gu.host_u16(w2u), h2, B)
        got, total, hout = _gpu_encode_hashed(gu, w2u, h2, B, ws)
        assert orc.header(expect)["changed_blocks"] == 1
        np.testing.assert_array_equal(got[:total], expect)
        np.testing.assert_array_equal(hout, h_same)
    # a HashCache matching nothing: every block is sent
    junk = np.arange(h_same.size, dtype=np.uint64)
    expect, _ = orc.encode_hashed(gu.host_u16(w2u), junk, B)
    got, total, _ = _gpu_encode_hashed(gu, w2u, junk, B, ws)
    assert orc.header(expect)["E"] == n
    np.testing.assert_array_equal(got[:total], expect)
    assert ws.error() == 0


@pytest.mark.parametrize("B", [512, 4096])
def test_hashed_chain_keeps_caches_in_step(gu, orc, B):
    """T steps of evolving weights: the sender keeps only its HashCache (in
    place), the receiver its exponent cache; every step decodes exactly."""
    from paper_2609_04609_amd import ciera, synth
    n = 3 * 16384 + 17
    ws = ciera.Workspace(n, 1, B)
    w, _ = gu.pair(n, 31)
    h = torch.zeros(2 * (-(-n // B)), dtype=torch.int64, device="cuda")
    ciera.hash_blocks_t(w, B, h)
    cache_rx = orc.split(gu.host_u16(w))[0]
    cur = w
    for step in range(4):
        nxt = synth.forced_bernoulli_bits(cur, 0.001 * (step + 1), 50 + step)
        cap = int(ciera.ciera_encoded_bound(n, B))
        out = torch.zeros(cap, dtype=torch.uint8, device="cuda")
        nbytes = torch.zeros(1, dtype=torch.int64, device="cuda")
        ciera.encode_hashed_t(nxt, h, h, B, ws, out, out_bytes=nbytes)
        torch.cuda.synchronize()
        enc = gu.host_u8(out)[:int(nbytes.item())]
        vals = orc.decode(enc, n, cache_rx)
        np.testing.assert_array_equal(vals, gu.host_u16(nxt))
        np.testing.assert_array_equal(_host_u64(h),
                                      orc.hash_blocks(gu.host_u16(nxt), B))
        cur = nxt


@pytest.mark.parametrize("B,n", [(512, 40_000_017), (64, 70_000_003)])
def test_encode_hashed_large_shards(gu, orc, B, n):
    """Shards large enough for the exception pass to take two tiles a wave
    or more, where the streaming pass walks its workgroups in runs per XCD:
    hashed and exact-compare encodes against the oracle."""
    from paper_2609_04609_amd import ciera
    w, w2 = gu.pair(n, 900 + B, c=0.001)
    wh, w2h = gu.host_u16(w), gu.host_u16(w2)
    h_old = orc.hash_blocks(wh, B)
    expect, h_new = orc.encode_hashed(w2h, h_old, B)
    cache_h, _ = orc.split(wh)
    np.testing.assert_array_equal(expect, orc.encode(w2h, cache_h, B))
    ws = ciera.Workspace(n, 1, B)
    got, total, hout = _gpu_encode_hashed(gu, w2, h_old, B, ws)
    assert total == expect.size
    np.testing.assert_array_equal(got[:total], expect)
    np.testing.assert_array_equal(hout, h_new)
    out, total, _ = gu.gpu_encode(w2, gu.dev_u8(cache_h), B, ws)
    assert total == expect.size
    np.testing.assert_array_equal(gu.host_u8(out[:total]), expect)
    assert ws.error() == 0
