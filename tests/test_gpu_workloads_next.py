"""Full-size parity for the block hash, the rANS-coded exception section and
the fp16 shards, on the OLMoE layer the benchmark times (16 shards of
25,165,824 values, c = 0.1%, B = 512) and on one 88,080,384-value
DeepSeek-style shard, through the same C-ABI calls. The oracle redoes every
shard byte for byte."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

DEV = "cuda"
B = 512


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_04609_amd import ciera
    ciera.lib()
    return ciera


def _h16(t):
    return t.cpu().numpy().view(np.uint16)


def _h8(t):
    return t.cpu().numpy().view(np.uint8)


def _h64(t):
    return t.cpu().numpy().view(np.uint64)


@pytest.fixture(scope="module")
def layer(lib):
    from paper_2609_04609_amd import synth
    wl = synth.WORKLOADS["olmoe_layer_c0.1"]
    pairs = [synth.shard_pair(wl, j, DEV) for j in range(wl.shards)]
    return wl.shards, wl.shard_elems, pairs


def test_hashed_encode_full_layer(lib, orc, layer):
    R, n, pairs = layer
    ws = lib.Workspace(n, 1, B)
    cap = int(lib.ciera_encoded_bound(n, B))
    out = torch.empty(cap, dtype=torch.uint8, device=DEV)
    ref = torch.empty_like(out)
    nb = torch.zeros(1, dtype=torch.int64, device=DEV)
    nblk = -(-n // B)
    for j, (w, w2) in enumerate(pairs):
        h_in = torch.empty(2 * nblk, dtype=torch.int64, device=DEV)
        h_out = torch.empty_like(h_in)
        lib.hash_blocks_t(w, B, h_in)
        lib.encode_hashed_t(w2, h_in, h_out, B, ws, out, out_bytes=nb)
        torch.cuda.synchronize()
        total = int(nb.item())
        got = _h8(out)[:total]
        wh, w2h = _h16(w), _h16(w2)
        h_old = orc.hash_blocks(wh, B)
        np.testing.assert_array_equal(_h64(h_in), h_old)
        expect, h_new = orc.encode_hashed(w2h, h_old, B)
        np.testing.assert_array_equal(got, expect, err_msg=f"shard {j}")
        np.testing.assert_array_equal(_h64(h_out), h_new)
        # the same bytes as the exact-compare encoder on the GPU
        cache = torch.from_numpy(orc.split(wh)[0]).to(DEV)
        lib.encode_t(w2, cache, B, ws, ref, out_bytes=nb)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(_h8(ref)[:int(nb.item())], got)
    assert ws.error() == 0


def test_ans_full_layer(lib, orc, layer):
    """Every shard encoded and rANS-coded on the GPU equals the oracle's; the
    gathered decode of the coded layer equals the oracle's and W'."""
    R, n, pairs = layer
    ws1 = lib.Workspace(n, 1, B, ans=True)
    cap = int(lib.ciera_encoded_bound(n, B))
    buf = torch.empty(cap, dtype=torch.uint8, device=DEV)
    nb = torch.zeros(1, dtype=torch.int64, device=DEV)
    encs, caches = [], []
    for j, (w, w2) in enumerate(pairs):
        cache_h = orc.split(_h16(w))[0]
        lib.encode_t(w2, torch.from_numpy(cache_h).to(DEV), B, ws1, buf)
        lib.ans_code_t(buf, n, B, ws1, out_bytes=nb)
        torch.cuda.synchronize()
        got = _h8(buf)[:int(nb.item())]
        expect = orc.ans_code(orc.encode(_h16(w2), cache_h, B), n)
        assert orc.header(expect)["mode"] == 2
        np.testing.assert_array_equal(got, expect, err_msg=f"shard {j}")
        encs.append(got)
        caches.append(cache_h)
    offs = np.cumsum([0] + [e.size for e in encs[:-1]]).astype(np.uint64)
    g = np.concatenate(encs)
    del encs
    cache0 = np.concatenate(caches)
    wsR = lib.Workspace(n, R, B, ans=True)
    out = torch.empty(R * n, dtype=torch.int16, device=DEV)
    cache = torch.from_numpy(cache0).to(DEV)
    lib.decode_gathered_t(torch.from_numpy(g).to(DEV),
                          torch.from_numpy(offs.view(np.int64)).to(DEV), n, B,
                          out, cache, wsR)
    torch.cuda.synchronize()
    cache_o = cache0.copy()
    out_o = orc.decode_gathered(g, offs, n, cache_o)
    np.testing.assert_array_equal(_h16(out), out_o)
    np.testing.assert_array_equal(_h8(cache), cache_o)
    np.testing.assert_array_equal(out_o,
                                  np.concatenate([_h16(w2) for _, w2 in pairs]))
    assert wsR.error() == 0 and ws1.error() == 0


def test_fp16_full_layer(lib, orc, layer):
    """The same geometry in fp16: every shard's encoding and the gathered
    decode equal the oracle's."""
    from paper_2609_04609_amd import synth
    R, n, _ = layer
    ws1 = lib.Workspace(n, 1, B)
    cap = int(lib.ciera_encoded_bound(n, B, lib.FP16))
    buf = torch.empty(cap, dtype=torch.uint8, device=DEV)
    nb = torch.zeros(1, dtype=torch.int64, device=DEV)
    encs, caches, vals = [], [], []
    for j in range(R):
        w = synth.normal_f16_bits(n, 0.02, synth.seed_for("f16layer", j, 0),
                                  DEV)
        w2 = synth.forced_bernoulli_f16_bits(w, 0.001,
                                             synth.seed_for("f16layer", j, 1))
        cache_h = orc.split_f16(_h16(w))[0]
        lib.encode_t(w2, torch.from_numpy(cache_h).to(DEV), B, ws1, buf,
                     out_bytes=nb, fp16=True)
        torch.cuda.synchronize()
        got = _h8(buf)[:int(nb.item())]
        np.testing.assert_array_equal(
            got, orc.encode_f16(_h16(w2), cache_h, B), err_msg=f"shard {j}")
        encs.append(got)
        caches.append(cache_h)
        vals.append(_h16(w2))
    offs = np.cumsum([0] + [e.size for e in encs[:-1]]).astype(np.uint64)
    g = np.concatenate(encs)
    cache0 = np.concatenate(caches)
    wsR = lib.Workspace(n, R, B)
    out = torch.empty(R * n, dtype=torch.int16, device=DEV)
    cache = torch.from_numpy(cache0).to(DEV)
    lib.decode_gathered_t(torch.from_numpy(g).to(DEV),
                          torch.from_numpy(offs.view(np.int64)).to(DEV), n, B,
                          out, cache, wsR, fp16=True)
    torch.cuda.synchronize()
    cache_o = cache0.copy()
    out_o = orc.decode_gathered_f16(g, offs, n, cache_o)
    np.testing.assert_array_equal(_h16(out), out_o)
    np.testing.assert_array_equal(_h8(cache), cache_o)
    np.testing.assert_array_equal(out_o, np.concatenate(vals))
    assert wsR.error() == 0


def test_ans_deepseek_shard(lib, orc):
    """One 88,080,384-value DeepSeek-style shard (clustered 0.5% change):
    encoding, rANS coding and the coded decode equal the oracle's."""
    from paper_2609_04609_amd import synth
    wl = synth.WORKLOADS["dsv3_layer"]
    n = wl.shard_elems
    w, w2 = synth.shard_pair(wl, 0, DEV)
    cache_h = orc.split(_h16(w))[0]
    ws = lib.Workspace(n, 1, B, ans=True)
    buf = torch.empty(int(lib.ciera_encoded_bound(n, B)), dtype=torch.uint8,
                      device=DEV)
    nb = torch.zeros(1, dtype=torch.int64, device=DEV)
    lib.encode_t(w2, torch.from_numpy(cache_h).to(DEV), B, ws, buf)
    lib.ans_code_t(buf, n, B, ws, out_bytes=nb)
    torch.cuda.synchronize()
    got = _h8(buf)[:int(nb.item())]
    expect = orc.ans_code(orc.encode(_h16(w2), cache_h, B), n)
    assert orc.header(expect)["mode"] == 2
    np.testing.assert_array_equal(got, expect)
    out = torch.empty(n, dtype=torch.int16, device=DEV)
    cache = torch.from_numpy(cache_h).to(DEV)
    lib.decode_gathered_t(torch.from_numpy(got).to(DEV),
                          torch.zeros(1, dtype=torch.int64, device=DEV), n, B,
                          out, cache, ws)
    torch.cuda.synchronize()
    assert torch.equal(out, w2)
    np.testing.assert_array_equal(_h8(cache), orc.split(_h16(w2))[0])
    assert ws.error() == 0
