"""GPU path vs the CPU oracle, byte for byte (tolerance 0: the codec is
integer bit manipulation). Encode is compared over the whole encoded buffer
(header, sections, padding); decode over the rebuilt values and the updated
caches. All calls go through the C ABI."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

# sizes that span several tiles and leave ragged tails (tile = 16384 values
# at B <= 2048, 32768 at B = 4096)
SIZES = [1, 7, 8, 9, 100, 511, 4097, 16383, 16384, 16385, 40000,
         3 * 16384 + 17, 32768 * 3 + 8, 262147]
BLOCKS = [1, 16, 32, 64, 128, 512, 2048, 4096]


@pytest.fixture(scope="module")
def gu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util
    from paper_2609_04609_amd import ciera
    ciera.lib()
    return gpu_util


@pytest.mark.parametrize("B", [16, 32, 64, 128, 256, 512, 1024, 2048, 4096])
def test_encode_rows_random_sizes(gu, orc, B):
    """The run-per-wave exception passes (over changed blocks for B <= 256,
    over changed rows for B >= 512) on seeded random sizes and change rates,
    bf16 and fp16, against the oracle byte for byte."""
    from paper_2609_04609_amd import ciera, synth
    rng = np.random.default_rng(B)
    sizes = [int(x) for x in rng.integers(1, 2_000_000, 6)]
    ws = ciera.Workspace(max(sizes), 1, B)
    for i, n in enumerate(sizes):
        c = float(rng.choice([0.0, 0.0005, 0.003, 0.05]))
        w, w2 = gu.pair(n, 9000 + B + i, c=c)
        cache_h = orc.split(gu.host_u16(w))[0]
        out, total, _ = gu.gpu_encode(w2, gu.dev_u8(cache_h), B, ws)
        expect = orc.encode(gu.host_u16(w2), cache_h, B)
        np.testing.assert_array_equal(gu.host_u8(out)[:total], expect,
                                      err_msg=f"n={n} c={c}")
        gu.check_fused_update(orc, w2, cache_h, B, expect, ws,
                              msg=f"fused n={n} c={c}")
        f = synth.normal_f16_bits(n, 0.02, 9100 + B + i, "cuda")
        f2 = synth.forced_bernoulli_f16_bits(f, c, 9200 + B + i)
        fc = orc.split_f16(gu.host_u16(f))[0]
        fb = torch.empty(int(ciera.ciera_encoded_bound(n, B, ciera.FP16)),
                         dtype=torch.uint8, device="cuda")
        nb = torch.zeros(1, dtype=torch.int64, device="cuda")
        ciera.encode_t(f2, gu.dev_u8(fc), B, ws, fb, out_bytes=nb, fp16=True)
        torch.cuda.synchronize()
        expect16 = orc.encode_f16(gu.host_u16(f2), fc, B)
        np.testing.assert_array_equal(
            gu.host_u8(fb)[:int(nb.item())], expect16, err_msg=f"fp16 n={n}")
        gu.check_fused_update(orc, f2, fc, B, expect16, ws, fp16=True,
                              msg=f"fused fp16 n={n}")
    assert ws.error() == 0


@pytest.mark.parametrize("B,waves", [(64, 16384), (512, 8192)])
@pytest.mark.parametrize("extra", [0, 1, 4097])
def test_encode_rows_run_boundary(gu, orc, B, waves, extra):
    """Shards around the size where the exception pass goes from one tile
    per wave to two (16,384 tiles of 4096 values at B < 512, 8192 at
    B >= 512, where runs of two tiles or more also take the deeper batch
    when the cache is brought forward): the last run may hold a single,
    partial tile. Plain and fused-update encodes match the oracle."""
    n = waves * 4096 + extra
    w, w2 = gu.pair(n, 9300 + n % 7, c=0.0005)
    cache_h = orc.split(gu.host_u16(w))[0]
    del w
    out, total, ws = gu.gpu_encode(w2, gu.dev_u8(cache_h), B)
    expect = orc.encode(gu.host_u16(w2), cache_h, B)
    assert total == expect.size
    np.testing.assert_array_equal(gu.host_u8(out)[:total], expect)
    del out
    gu.check_fused_update(orc, w2, cache_h, B, expect, ws, msg="fused")
    assert ws.error() == 0


def test_encode_rows_with_count_scan(gu, orc):
    """A 600,000,005-value shard at B = 512: the row-wise exception pass gives
    each wave a run of 18 tiles, and its workgroups' counting would re-read
    about 149 MB of bitmap, so the offsets come from pass 1's per-tile counts
    and the scan. bf16 and fp16 match the oracle byte for byte; a small call
    first must not leak its counts into the big one."""
    from paper_2609_04609_amd import ciera, synth
    n, B = 600_000_005, 512
    ws = ciera.Workspace(n, 1, B)
    w, w2 = gu.pair(n, 3131, c=0.0002)
    wh, w2h = gu.host_u16(w), gu.host_u16(w2)
    cache_h = orc.split(wh)[0]
    out, total, _ = gu.gpu_encode(w2[:70_000], gu.dev_u8(cache_h[:70_000]), B,
                                  ws)
    np.testing.assert_array_equal(gu.host_u8(out)[:total],
                                  orc.encode(w2h[:70_000], cache_h[:70_000], B))
    expect = orc.encode(w2h, cache_h, B)
    out, total, _ = gu.gpu_encode(w2, gu.dev_u8(cache_h), B, ws)
    assert total == expect.size
    np.testing.assert_array_equal(gu.host_u8(out)[:total], expect)
    del out
    gu.check_fused_update(orc, w2, cache_h, B, expect, ws, msg="fused")
    del w, w2, wh, w2h, cache_h, expect
    torch.cuda.empty_cache()
    f = synth.normal_f16_bits(n, 0.02, 3232, "cuda")
    f2 = synth.forced_bernoulli_f16_bits(f, 0.0002, 3233)
    fc = orc.split_f16(gu.host_u16(f))[0]
    fb = torch.empty(int(ciera.ciera_encoded_bound(n, B, ciera.FP16)),
                     dtype=torch.uint8, device="cuda")
    nb = torch.zeros(1, dtype=torch.int64, device="cuda")
    ciera.encode_t(f2, gu.dev_u8(fc), B, ws, fb, out_bytes=nb, fp16=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u8(fb)[:int(nb.item())],
                                  orc.encode_f16(gu.host_u16(f2), fc, B))
    assert ws.error() == 0


def test_encode_rows_several_chunks(gu, orc):
    """A 600,000,003-value shard at B = 4096: each wave of the row-wise
    exception pass takes three tiles, 192 rows of 512 values, so it walks its
    run in three chunks of 64 rows. Matches the oracle byte for byte."""
    n, B = 600_000_003, 4096
    w, w2 = gu.pair(n, 3434, c=0.00002)
    cache_h = orc.split(gu.host_u16(w))[0]
    del w
    out, total, ws = gu.gpu_encode(w2, gu.dev_u8(cache_h), B)
    expect = orc.encode(gu.host_u16(w2), cache_h, B)
    assert total == expect.size
    np.testing.assert_array_equal(gu.host_u8(out)[:total], expect)
    del out
    gu.check_fused_update(orc, w2, cache_h, B, expect, ws, msg="fused")
    assert ws.error() == 0


def test_encode_with_count_scan(gu, orc):
    """A 25,165,832-value shard at B = 16: counting the bitmap in front of
    every exception-pass workgroup would re-read about 151 MB, so pass 1
    writes per-tile counts and a scan gives the offsets. Exact compare,
    the block hash and fp16 all match the oracle byte for byte; the first
    call after a small one reuses the workspace."""
    from paper_2609_04609_amd import ciera, synth
    n, B = 25_165_832, 16
    ws = ciera.Workspace(n, 1, B)
    w, w2 = gu.pair(n, 2525, c=0.002)
    wh, w2h = gu.host_u16(w), gu.host_u16(w2)
    cache_h = orc.split(wh)[0]
    # a small call first: its counts and offsets must not leak into the next
    out, total, _ = gu.gpu_encode(w2[:5000], gu.dev_u8(cache_h[:5000]), B, ws)
    np.testing.assert_array_equal(gu.host_u8(out)[:total],
                                  orc.encode(w2h[:5000], cache_h[:5000], B))
    expect = orc.encode(w2h, cache_h, B)
    out, total, _ = gu.gpu_encode(w2, gu.dev_u8(cache_h), B, ws)
    assert total == expect.size
    np.testing.assert_array_equal(gu.host_u8(out)[:total], expect)
    gu.check_fused_update(orc, w2, cache_h, B, expect, ws, msg="fused")
    # the block-hash detector gives the same bytes
    nblk = -(-n // B)
    h_in = torch.empty(2 * nblk, dtype=torch.int64, device="cuda")
    h_out = torch.empty_like(h_in)
    ciera.hash_blocks_t(w, B, h_in)
    hb = torch.empty(int(ciera.ciera_encoded_bound(n, B)), dtype=torch.uint8,
                     device="cuda")
    nb = torch.zeros(1, dtype=torch.int64, device="cuda")
    ciera.encode_hashed_t(w2, h_in, h_out, B, ws, hb, out_bytes=nb)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u8(hb)[:int(nb.item())], expect)
    # fp16 at the same size
    f = synth.normal_f16_bits(n, 0.02, 2626, "cuda")
    f2 = synth.forced_bernoulli_f16_bits(f, 0.002, 2627)
    fc = orc.split_f16(gu.host_u16(f))[0]
    fb = torch.empty(int(ciera.ciera_encoded_bound(n, B, ciera.FP16)),
                     dtype=torch.uint8, device="cuda")
    ciera.encode_t(f2, gu.dev_u8(fc), B, ws, fb, out_bytes=nb, fp16=True)
    torch.cuda.synchronize()
    expect16 = orc.encode_f16(gu.host_u16(f2), fc, B)
    np.testing.assert_array_equal(gu.host_u8(fb)[:int(nb.item())], expect16)
    gu.check_fused_update(orc, f2, fc, B, expect16, ws, fp16=True,
                          msg="fused fp16")
    assert ws.error() == 0


@pytest.mark.parametrize("B", BLOCKS)
def test_encode_matches_oracle(gu, orc, B):
    ws = None
    for i, n in enumerate(SIZES):
        w, w2 = gu.pair(n, 100 * B + i, c=0.002 * (1 + i % 4))
        cache_h, _ = orc.split(gu.host_u16(w))
        cache = gu.dev_u8(cache_h)
        from paper_2609_04609_amd import ciera
        ws = ws if ws is not None and ws.nbytes >= ciera.ciera_workspace_bytes(
            n, 1, B, 0) else ciera.Workspace(max(n, 262147), 1, B)
        out, total, ws = gu.gpu_encode(w2, cache, B, ws)
        expect = orc.encode(gu.host_u16(w2), cache_h, B)
        got = gu.host_u8(out)
        assert total == expect.size, (n, B)
        np.testing.assert_array_equal(got[:total], expect, err_msg=f"n={n} B={B}")
        # nothing written past the encoded size
        assert np.all(got[total:] == 0xA5)
        gu.check_fused_update(orc, w2, cache_h, B, expect, ws,
                              msg=f"fused n={n} B={B}")
        assert ws.error() == 0


def test_encode_edge_cases(gu, orc):
    from paper_2609_04609_amd import ciera
    B = 512
    ws = ciera.Workspace(1 << 20, 1, B)
    rng = np.random.default_rng(5)
    n = 70001
    w, _ = gu.pair(n, 77)
    wh = gu.host_u16(w)
    e_h, _ = orc.split(wh)
    cases = {
        "no_change": e_h.copy(),
        "all_change": (e_h + 1).astype(np.uint8),
        "random_cache": rng.integers(0, 256, n, dtype=np.uint8),
    }
    for name, cache_h in cases.items():
        out, total, _ = gu.gpu_encode(w, gu.dev_u8(cache_h), B, ws)
        expect = orc.encode(wh, cache_h, B)
        np.testing.assert_array_equal(gu.host_u8(out)[:total], expect,
                                      err_msg=name)
    # n = 0: header only
    out, total, _ = gu.gpu_encode(torch.zeros(0, dtype=torch.int16,
                                              device="cuda"),
                                  torch.zeros(0, dtype=torch.uint8,
                                              device="cuda"), B, ws)
    expect = orc.encode(np.zeros(0, np.uint16), np.zeros(0, np.uint8), B)
    np.testing.assert_array_equal(gu.host_u8(out)[:total], expect)
    # raw form
    for n in [0, 1, 9, 16385]:
        w, _ = gu.pair(n, 90 + n)
        out, total, _ = gu.gpu_encode(w, None, B, ws, raw=True)
        expect = orc.encode(gu.host_u16(w), None, B, raw=True)
        np.testing.assert_array_equal(gu.host_u8(out)[:total], expect)
    assert ws.error() == 0


@pytest.mark.parametrize("B", [1, 64, 512, 4096])
def test_encode_unaligned_pointers(gu, orc, B):
    """Inputs that are not 16-byte aligned take the element-wise path."""
    from paper_2609_04609_amd import ciera
    n = 50001
    w_all, w2_all = gu.pair(n + 1, 31)
    w, w2 = w_all[1:], w2_all[1:]            # 2-byte offset
    cache_all = gu.dev_u8(np.concatenate(
        [[0], orc.split(gu.host_u16(w))[0]]))
    cache = cache_all[1:]                    # 1-byte offset
    ws = ciera.Workspace(n, 1, B)
    out, total, _ = gu.gpu_encode(w2, cache, B, ws)
    expect = orc.encode(gu.host_u16(w2), gu.host_u8(cache), B)
    np.testing.assert_array_equal(gu.host_u8(out)[:total], expect)


@pytest.mark.parametrize("B", [1, 512, 4096])
def test_encode_repeats_and_reuses_workspace(gu, orc, B):
    """The workspace is reused call after call, with shard sizes that grow
    and shrink between calls; the bytes never change."""
    from paper_2609_04609_amd import ciera
    n = 300000
    w, w2 = gu.pair(n, 41, c=0.001)
    cache_h, _ = orc.split(gu.host_u16(w))
    cache = gu.dev_u8(cache_h)
    expect = orc.encode(gu.host_u16(w2), cache_h, B)
    small = 777
    expect_small = orc.encode(gu.host_u16(w2[:small]), cache_h[:small], B)
    ws = ciera.Workspace(n, 1, B)
    for i in range(20):
        out, total, _ = gu.gpu_encode(w2, cache, B, ws)
        np.testing.assert_array_equal(gu.host_u8(out)[:total], expect)
        if i % 5 == 4:
            out, total, _ = gu.gpu_encode(w2[:small], cache[:small], B, ws)
            np.testing.assert_array_equal(gu.host_u8(out)[:total],
                                          expect_small)
    assert ws.error() == 0


def _decode_case(gu, orc, R, n_s, B, raw_mask, seed):
    """Encode R shards with the oracle, gather them, decode on the GPU."""
    from paper_2609_04609_amd import synth
    encs, caches, values = [], [], []
    for j in range(R):
        w = synth.normal_bf16_bits(n_s, 0.02, seed + j).numpy().view(np.uint16)
        w2 = synth.forced_bernoulli_bits(
            torch.from_numpy(w.view(np.int16)), 0.003, seed + 100 + j
        ).numpy().view(np.uint16)
        c, _ = orc.split(w)
        encs.append(orc.encode(w2, None if raw_mask[j] else c, B,
                               raw=bool(raw_mask[j])))
        caches.append(c)
        values.append(w2)
    gathered, offs = gu.gather(encs)
    cache0 = np.concatenate(caches)
    return gathered, offs, cache0, np.concatenate(values)


@pytest.mark.parametrize("B", [1, 16, 64, 512, 4096])
@pytest.mark.parametrize("R,n_s", [(1, 1), (3, 16385), (4, 40000),
                                   (5, 7777), (16, 16384), (2, 100003),
                                   # 310 decode tiles of 16384 values, the
                                   # last of each shard ragged: runs of 32
                                   # tiles per XCD over the first 256, the
                                   # rest in order
                                   (5, 1_000_003)])
def test_decode_gathered_matches_oracle(gu, orc, B, R, n_s):
    from paper_2609_04609_amd import ciera
    raw_mask = [(j % 3) == 2 for j in range(R)]
    gathered, offs, cache0, values = _decode_case(gu, orc, R, n_s, B,
                                                  raw_mask, 1000 * B + R)
    cache_o = cache0.copy()
    expect = orc.decode_gathered(gathered, offs, n_s, cache_o)
    np.testing.assert_array_equal(expect, values)  # oracle round trip
    g = gu.dev_u8(gathered)
    o = torch.from_numpy(offs.view(np.int64)).to("cuda")
    out = torch.empty(R * n_s, dtype=torch.int16, device="cuda")
    cache = gu.dev_u8(cache0)
    ws = ciera.Workspace(n_s, R, B)
    ciera.decode_gathered_t(g, o, n_s, B, out, cache, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u16(out), expect)
    np.testing.assert_array_equal(gu.host_u8(cache), cache_o)
    # idempotent
    ciera.decode_gathered_t(g, o, n_s, B, out, cache, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u16(out), expect)
    np.testing.assert_array_equal(gu.host_u8(cache), cache_o)
    assert ws.error() == 0


@pytest.mark.parametrize("n_s", [6_000_008, 6_000_003])
def test_decode_with_prefix_pass(gu, orc, n_s):
    """16 shards of about 6M values at B = 16: counting each tile's offset in
    the tile would re-read about 138 MB of bitmap per call, so the decode
    scans every shard's tile counts in a pass of its own first. One raw shard
    in the middle; n % 8 == 0 takes the vector path, the other size the
    element-wise one. Values and caches equal the oracle's; the cache update
    of one 24M-value shard takes the same pass."""
    from paper_2609_04609_amd import ciera
    R, B = 16, 16
    raw_mask = [j == 7 for j in range(R)]
    gathered, offs, cache0, values = _decode_case(gu, orc, R, n_s, B,
                                                  raw_mask, 31337 + n_s % 8)
    cache_o = cache0.copy()
    expect = orc.decode_gathered(gathered, offs, n_s, cache_o)
    np.testing.assert_array_equal(expect, values)
    out = torch.empty(R * n_s, dtype=torch.int16, device="cuda")
    cache = gu.dev_u8(cache0)
    ws = ciera.Workspace(n_s, R, B)
    ciera.decode_gathered_t(gu.dev_u8(gathered),
                            torch.from_numpy(offs.view(np.int64)).to("cuda"),
                            n_s, B, out, cache, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u16(out), expect)
    np.testing.assert_array_equal(gu.host_u8(cache), cache_o)
    assert ws.error() == 0
    # the prefix pass too skips a shard that runs past the given length
    out.fill_(7)
    cache = gu.dev_u8(cache0)
    ciera.decode_gathered_t(gu.dev_u8(gathered),
                            torch.from_numpy(offs.view(np.int64)).to("cuda"),
                            n_s, B, out, cache, ws,
                            nbytes=gathered.size - 16)
    torch.cuda.synchronize()
    assert ws.error() == ciera.DEVERR_BOUNDS
    last = (R - 1) * n_s
    np.testing.assert_array_equal(gu.host_u16(out[:last]), expect[:last])
    assert bool(torch.all(out[last:] == 7))
    np.testing.assert_array_equal(gu.host_u8(cache[last:]), cache0[last:])
    del gathered, cache0, values, out, cache
    n1 = 4 * n_s
    g1, o1, c1, _ = _decode_case(gu, orc, 1, n1, B, [False], 99 + n_s % 8)
    c1_o = c1.copy()
    orc.update_cache(c1_o, g1, n1)
    c1_d = gu.dev_u8(c1)
    ws1 = ciera.Workspace(n1, 1, B)
    ciera.update_cache_t(c1_d, gu.dev_u8(g1), n1, B, ws1)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u8(c1_d), c1_o)
    assert ws1.error() == 0


@pytest.mark.parametrize("B,fp16", [(64, False), (512, True), (1, False)])
def test_decode_caches_past_1gib(gu, orc, B, fp16):
    """17 shards of 67,108,864 values: 1.14 GB of caches, past the size
    where the merge writes its cache patches with non-temporal stores. Every
    shard is encoded by the oracle and its decoded values and updated cache
    are compared with the oracle's, shard by shard on the host."""
    import concurrent.futures as cf
    import os
    from paper_2609_04609_amd import ciera, synth
    R, n = 17, 1 << 26
    enc_o = orc.encode_f16 if fp16 else orc.encode
    split = orc.split_f16 if fp16 else orc.split
    dec_o = orc.decode_f16 if fp16 else orc.decode

    def shard(j):
        if fp16:
            w = synth.normal_f16_bits(n, 0.02, 4100 + j, "cuda")
            w2 = synth.forced_bernoulli_f16_bits(w, 0.001, 4200 + j)
        else:
            w, w2 = gu.pair(n, 4100 + 2 * j, c=0.001)
        return gu.host_u16(w), gu.host_u16(w2)

    def encode(j):
        wh, w2h = shard(j)
        c = split(wh)[0]
        return enc_o(w2h, c, B), c, w2h

    workers = max(1, min(8, os.cpu_count() or 1))
    with cf.ThreadPoolExecutor(workers) as ex:
        parts = list(ex.map(encode, range(R)))
    encs = [p[0] for p in parts]
    gathered, offs = gu.gather(encs)
    cache = torch.empty(R * n, dtype=torch.uint8, device="cuda")
    for j, (_, c, _) in enumerate(parts):
        cache[j * n:(j + 1) * n].copy_(torch.from_numpy(c))
    out = torch.empty(R * n, dtype=torch.int16, device="cuda")
    ws = ciera.Workspace(n, R, B)
    ciera.decode_gathered_t(gu.dev_u8(gathered),
                            torch.from_numpy(offs.view(np.int64)).cuda(), n,
                            B, out, cache, ws, fp16=fp16)
    torch.cuda.synchronize()
    assert ws.error() == 0
    del gathered

    def check(j):
        enc, c, w2h = parts[j]
        c_o = c.copy()
        out_o = dec_o(enc, n, c_o)
        sl = slice(j * n, (j + 1) * n)
        if not np.array_equal(out_o, w2h):
            return f"shard {j}: oracle round trip"
        if not np.array_equal(gu.host_u16(out[sl]), out_o):
            return f"shard {j}: values"
        if not np.array_equal(gu.host_u8(cache[sl]), c_o):
            return f"shard {j}: cache"
        return None

    with cf.ThreadPoolExecutor(workers) as ex:
        errs = [e for e in ex.map(check, range(R)) if e]
    assert not errs, errs


@pytest.mark.parametrize("B", [1, 16, 512, 4096])
def test_update_cache_matches_oracle(gu, orc, B):
    from paper_2609_04609_amd import ciera
    for n, raw in [(1, False), (16385, False), (100003, False), (5000, True)]:
        gathered, offs, cache0, values = _decode_case(gu, orc, 1, n, B,
                                                      [raw], 7 * n + B)
        cache_o = cache0.copy()
        orc.update_cache(cache_o, gathered, n)
        cache = gu.dev_u8(cache0)
        ws = ciera.Workspace(n, 1, B)
        ciera.update_cache_t(cache, gu.dev_u8(gathered), n, B, ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(gu.host_u8(cache), cache_o)
        assert ws.error() == 0


@pytest.mark.parametrize("B", [1, 64])
def test_decode_unaligned_and_bad_shards(gu, orc, B):
    from paper_2609_04609_amd import ciera
    R, n_s = 3, 5003                 # n_s % 8 != 0: element-wise stores
    gathered, offs, cache0, values = _decode_case(gu, orc, R, n_s, B,
                                                  [False] * R, 555)
    cache_o = cache0.copy()
    expect = orc.decode_gathered(gathered, offs, n_s, cache_o)
    g = gu.dev_u8(gathered)
    o = torch.from_numpy(offs.view(np.int64)).to("cuda")
    out = torch.empty(R * n_s, dtype=torch.int16, device="cuda")
    cache = gu.dev_u8(cache0)
    ws = ciera.Workspace(n_s, R, B)
    ciera.decode_gathered_t(g, o, n_s, B, out, cache, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u16(out), expect)
    np.testing.assert_array_equal(gu.host_u8(cache), cache_o)
    # corrupt shard 1's magic: device reports FORMAT, shard 1 left untouched
    bad = gathered.copy()
    bad[int(offs[1])] ^= 0xFF
    out2 = torch.full((R * n_s,), 7, dtype=torch.int16, device="cuda")
    cache2 = gu.dev_u8(cache0)
    ciera.decode_gathered_t(gu.dev_u8(bad), o, n_s, B, out2, cache2, ws)
    torch.cuda.synchronize()
    assert ws.error() & ciera.DEVERR_FORMAT
    got = gu.host_u16(out2)
    np.testing.assert_array_equal(got[:n_s], expect[:n_s])
    assert np.all(got[n_s:2 * n_s] == 7)
    np.testing.assert_array_equal(gu.host_u8(cache2)[n_s:2 * n_s],
                                  cache0[n_s:2 * n_s])
    # a shard offset that is not 16-byte aligned
    o_bad = o.clone()
    o_bad[2] += 8
    ciera.decode_gathered_t(g, o_bad, n_s, B, out2, cache2, ws)
    torch.cuda.synchronize()
    assert ws.error() & ciera.DEVERR_ALIGN
    # a compressed shard decoded with the wrong block size
    ciera.decode_gathered_t(g, o, n_s, 128 if B != 128 else 64, out2, cache2,
                            ws)
    torch.cuda.synchronize()
    assert ws.error() & ciera.DEVERR_FORMAT


@pytest.mark.parametrize("B", [1, 64, 512])
def test_decode_respects_buffer_length(gu, orc, B):
    """The decoding calls read nothing past the length the caller gives.
    A valid copy of shard 2 sits in the allocation just past that length, so
    a missing check would read mapped memory and decode it: the test sees
    that as an untouched shard that changed. Each case: shard 2 is skipped
    with CIERA_DEVERR_BOUNDS (its values and cache untouched) and the other
    shards decode as the oracle does."""
    from paper_2609_04609_amd import ciera
    R, n_s = 3, 5003
    gathered, offs, cache0, values = _decode_case(gu, orc, R, n_s, B,
                                                  [False, True, False], 777)
    cache_o = cache0.copy()
    expect = orc.decode_gathered(gathered, offs, n_s, cache_o)
    L = gathered.size  # a multiple of 16
    enc2 = gathered[int(offs[2]):]
    big = gu.dev_u8(np.concatenate([gathered, enc2]))
    ws = ciera.Workspace(n_s, R, B)
    moved = offs.copy()
    moved[2] = L  # the copy past the buffer's end
    cases = [
        ("offset at the end", moved, L),
        ("header inside, total outside", moved, L + 64),
        ("total runs 16 bytes past", offs, L - 16),
    ]
    for name, o_h, nbytes in cases:
        o = torch.from_numpy(o_h.view(np.int64)).to("cuda")
        out = torch.full((R * n_s,), 7, dtype=torch.int16, device="cuda")
        cache = gu.dev_u8(cache0)
        ciera.decode_gathered_t(big, o, n_s, B, out, cache, ws, nbytes=nbytes)
        torch.cuda.synchronize()
        assert ws.error() == ciera.DEVERR_BOUNDS, name
        got, gc = gu.host_u16(out), gu.host_u8(cache)
        np.testing.assert_array_equal(got[:2 * n_s], expect[:2 * n_s],
                                      err_msg=name)
        np.testing.assert_array_equal(gc[:2 * n_s], cache_o[:2 * n_s],
                                      err_msg=name)
        assert np.all(got[2 * n_s:] == 7), name
        np.testing.assert_array_equal(gc[2 * n_s:], cache0[2 * n_s:],
                                      err_msg=name)
    # the exact length: everything decodes, no error
    o = torch.from_numpy(moved.view(np.int64)).to("cuda")
    out = torch.empty(R * n_s, dtype=torch.int16, device="cuda")
    cache = gu.dev_u8(cache0)
    ciera.decode_gathered_t(big, o, n_s, B, out, cache, ws,
                            nbytes=L + enc2.size)
    torch.cuda.synchronize()
    assert ws.error() == 0
    np.testing.assert_array_equal(gu.host_u16(out), expect)
    np.testing.assert_array_equal(gu.host_u8(cache), cache_o)
    # the stand-alone cache update with a short length leaves the cache alone
    one = gu.dev_u8(enc2)
    c2 = cache0[2 * n_s:]
    for nbytes in (enc2.size - 16, 63, 0):
        cache = gu.dev_u8(c2)
        ciera.update_cache_t(cache, one, n_s, B, ws, nbytes=nbytes)
        torch.cuda.synchronize()
        assert ws.error() == ciera.DEVERR_BOUNDS, nbytes
        np.testing.assert_array_equal(gu.host_u8(cache), c2)
    cache = gu.dev_u8(c2)
    ciera.update_cache_t(cache, one, n_s, B, ws)
    torch.cuda.synchronize()
    assert ws.error() == 0
    np.testing.assert_array_equal(gu.host_u8(cache), cache_o[2 * n_s:])


@pytest.mark.parametrize("B", [1, 512])
def test_round_trip_chain_on_gpu(gu, orc, B):
    """T iterations of encode -> gather -> decode entirely on the GPU: every
    shard decodes to its exact values, the sender caches (brought forward by
    ciera_update_cache) equal the receiver caches, and the oracle agrees on
    every encoded byte."""
    from paper_2609_04609_amd import ciera, synth
    R, n, T = 4, 33333, 4
    ws_e = ciera.Workspace(n, 1, B)
    ws_d = ciera.Workspace(n, R, B)
    ws = [synth.normal_bf16_bits(n, 0.02, 300 + j, "cuda") for j in range(R)]
    send_cache = [torch.zeros(n, dtype=torch.uint8, device="cuda")
                  for _ in range(R)]
    recv_cache = torch.zeros(R * n, dtype=torch.uint8, device="cuda")
    out = torch.empty(R * n, dtype=torch.int16, device="cuda")
    for t in range(T):
        encs = []
        for j in range(R):
            enc, total, _ = gu.gpu_encode(ws[j], send_cache[j], B, ws_e,
                                          raw=(t == 0))
            expect = orc.encode(gu.host_u16(ws[j]),
                                None if t == 0 else gu.host_u8(send_cache[j]),
                                B, raw=(t == 0))
            np.testing.assert_array_equal(gu.host_u8(enc)[:total], expect)
            ciera.update_cache_t(send_cache[j], enc, n, B, ws_e)
            encs.append(gu.host_u8(enc)[:total])
        gathered, offs = gu.gather(encs)
        ciera.decode_gathered_t(gu.dev_u8(gathered),
                                torch.from_numpy(offs.view(np.int64)).cuda(),
                                n, B, out, recv_cache, ws_d)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(gu.host_u16(out),
                                      np.concatenate([gu.host_u16(x)
                                                      for x in ws]))
        np.testing.assert_array_equal(gu.host_u8(recv_cache),
                                      np.concatenate([gu.host_u8(c)
                                                      for c in send_cache]))
        ws = [synth.forced_bernoulli_bits(x, 0.002, 7000 + 10 * t + j)
              for j, x in enumerate(ws)]
    assert ws_e.error() == 0 and ws_d.error() == 0


@pytest.mark.parametrize("B", [1, 16, 32, 64, 128, 256, 512, 1024, 2048,
                               4096])
def test_encode_with_cache_update(gu, orc, B):
    """CIERA_ENC_UPDATE_CACHE: the same bytes as the pure encode, and the
    cache afterwards equals the oracle's update of it from those bytes (the
    exponents of W'); also with a cache pointer off the 8-byte grid."""
    from paper_2609_04609_amd import ciera
    ws = ciera.Workspace(262147, 1, B)
    for i, n in enumerate([1, 9, 4097, 16385, 3 * 16384 + 17, 262147]):
        w, w2 = gu.pair(n, 600 * B + i, c=0.003)
        cache_h, _ = orc.split(gu.host_u16(w))
        expect = orc.encode(gu.host_u16(w2), cache_h, B)
        c_o = cache_h.copy()
        orc.update_cache(c_o, expect, n)
        for shift in (0, 3):
            buf = torch.zeros(n + 8, dtype=torch.uint8, device="cuda")
            cache = buf[shift:shift + n]
            cache.copy_(gu.dev_u8(cache_h))
            cap = int(ciera.ciera_encoded_bound(n, B))
            out = torch.full((cap,), 0xA5, dtype=torch.uint8, device="cuda")
            nbytes = torch.zeros(1, dtype=torch.int64, device="cuda")
            ciera.encode_t(w2, cache, B, ws, out, out_bytes=nbytes,
                           update_cache=True)
            torch.cuda.synchronize()
            total = int(nbytes.item())
            np.testing.assert_array_equal(gu.host_u8(out)[:total], expect,
                                          err_msg=f"n={n} B={B}")
            np.testing.assert_array_equal(gu.host_u8(cache), c_o,
                                          err_msg=f"n={n} B={B} s={shift}")
            assert ws.error() == 0
