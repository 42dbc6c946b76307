"""Every bit pattern through the HIP kernels (the losslessness claim of the
abstract and the bitwise-exact reconstruction of Section 4.6): all 65,536
bf16 patterns against each of the 256 cached exponents (16,777,216 pairs,
every old/new exponent pair, so +-0, subnormals, +-Inf and every NaN payload
meet every cache byte), and all 65,536 fp16 patterns against each of the 32
cached 5-bit exponents. For each block size the encode (pure and with the
fused cache update), the gathered decode of several shards and the
stand-alone cache update are compared with the oracle byte for byte, on the
full length and on a ragged one.

Three orders of the pairs: segments of one old exponent (pattern order
within), the unchanged pairs first (so that whole blocks are reused), and a
seeded random permutation."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util
    from paper_2609_04609_amd import ciera
    ciera.lib()
    return gpu_util


def _pairs(ebits, order):
    """(new patterns u16, cached exponents u8) over every pattern and every
    old exponent of an `ebits`-bit exponent field."""
    ne = 1 << ebits
    shift = 15 - ebits  # exponent field bits 14..shift
    pat = np.tile(np.arange(65536, dtype=np.uint32), ne)
    old = np.repeat(np.arange(ne, dtype=np.uint32), 65536)
    if order == "unchanged_first":
        same = ((pat >> shift) & (ne - 1)) == old
        idx = np.concatenate([np.flatnonzero(same), np.flatnonzero(~same)])
        pat, old = pat[idx], old[idx]
    elif order == "shuffled":
        idx = np.random.default_rng(0x5BEC1A1).permutation(pat.size)
        pat, old = pat[idx], old[idx]
    return pat.astype(np.uint16), old.astype(np.uint8)


def _run(gu, orc, w2h, cache_h, B, R, fp16):
    """Encode every one of R shards on the GPU (pure and fused), decode the
    oracle's gathered encodings on the GPU, update shard 0's cache alone."""
    from paper_2609_04609_amd import ciera
    n = w2h.size // R
    enc_o = orc.encode_f16 if fp16 else orc.encode
    dec_o = orc.decode_gathered_f16 if fp16 else orc.decode_gathered
    upd_o = orc.update_cache_f16 if fp16 else orc.update_cache
    flags = ciera.FP16 if fp16 else 0
    ws = ciera.Workspace(n, R, B)
    cap = int(ciera.ciera_encoded_bound(n, B, flags))
    out = torch.empty(cap, dtype=torch.uint8, device="cuda")
    nbytes = torch.zeros(1, dtype=torch.int64, device="cuda")
    encs = []
    for j in range(R):
        w2s, cs = w2h[j * n:(j + 1) * n], cache_h[j * n:(j + 1) * n]
        expect = enc_o(w2s, cs, B)
        w2d = gu.dev_bits(w2s)
        out.fill_(0xA5)
        ciera.encode_t(w2d, gu.dev_u8(cs), B, ws, out, out_bytes=nbytes,
                       fp16=fp16)
        torch.cuda.synchronize()
        total = int(nbytes.item())
        got = gu.host_u8(out)
        assert total == expect.size, (B, j)
        np.testing.assert_array_equal(got[:total], expect,
                                      err_msg=f"B={B} shard {j}")
        assert np.all(got[total:] == 0xA5)
        gu.check_fused_update(orc, w2d, cs, B, expect, ws, fp16=fp16,
                              msg=f"fused B={B} shard {j}")
        encs.append(expect)
    gathered, offs = gu.gather(encs)
    cache_o = cache_h[:R * n].copy()
    expect_v = dec_o(gathered, offs, n, cache_o)
    np.testing.assert_array_equal(expect_v, w2h[:R * n])
    out_v = torch.full((R * n,), 0x5A5A, dtype=torch.int16, device="cuda")
    cache = gu.dev_u8(cache_h[:R * n])
    ciera.decode_gathered_t(gu.dev_u8(gathered),
                            torch.from_numpy(offs.view(np.int64)).cuda(), n,
                            B, out_v, cache, ws, fp16=fp16)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u16(out_v), expect_v,
                                  err_msg=f"decode B={B}")
    np.testing.assert_array_equal(gu.host_u8(cache), cache_o,
                                  err_msg=f"decode cache B={B}")
    c0 = cache_h[:n].copy()
    upd_o(c0, encs[0], n)
    cache = gu.dev_u8(cache_h[:n])
    ciera.update_cache_t(cache, gu.dev_u8(encs[0]), n, B, ws, fp16=fp16)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gu.host_u8(cache), c0,
                                  err_msg=f"update B={B}")
    assert ws.error() == 0


@pytest.mark.parametrize("order", ["segments", "unchanged_first",
                                   "shuffled"])
@pytest.mark.parametrize("B", [1, 16, 512, 4096])
def test_every_bf16_pattern_and_old_exponent(gu, orc, B, order):
    """16,777,216 (pattern, old exponent) pairs as 4 shards of 4,194,304,
    then the first 16,777,211 as one ragged shard."""
    w2h, cache_h = _pairs(8, order)
    _run(gu, orc, w2h, cache_h, B, 4, False)
    _run(gu, orc, w2h[:-5], cache_h[:-5], B, 1, False)


@pytest.mark.parametrize("order", ["segments", "unchanged_first",
                                   "shuffled"])
@pytest.mark.parametrize("B", [16, 512])
def test_every_fp16_pattern_and_old_exponent(gu, orc, B, order):
    """2,097,152 (pattern, old 5-bit exponent) pairs as 2 shards, then the
    first 2,097,141 as one ragged shard."""
    w2h, cache_h = _pairs(5, order)
    _run(gu, orc, w2h, cache_h, B, 2, True)
    _run(gu, orc, w2h[:-11], cache_h[:-11], B, 1, True)


def test_special_values_round_trip_chain(gu, orc):
    """The special values as the weights of a few iterations: +-0, the
    smallest and largest subnormals, +-Inf, quiet and signalling NaNs with
    several payloads, the largest finite values, mixed with ordinary weights.
    Each iteration's W' comes back bit for bit from the GPU decode, and the
    sender's fused cache update keeps pace with the receivers'."""
    from paper_2609_04609_amd import ciera
    special = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x007F, 0x807F,
                        0x7F80, 0xFF80, 0x7FC0, 0xFFC0, 0x7F81, 0xFF81,
                        0x7FFF, 0xFFFF, 0x7FA5, 0x7F7F, 0xFF7F, 0x0080,
                        0x8080], dtype=np.uint16)
    rng = np.random.default_rng(77)
    n, B, R = 40_003, 64, 2
    ws_e = ciera.Workspace(n, 1, B)
    ws_d = ciera.Workspace(n, R, B)
    base = rng.integers(0x3C00, 0x3D00, size=R * n).astype(np.uint16)
    w = base.copy()
    send = [gu.dev_u8(orc.split(w[j * n:(j + 1) * n])[0]) for j in range(R)]
    recv = gu.dev_u8(orc.split(w)[0])
    out = torch.empty(R * n, dtype=torch.int16, device="cuda")
    for t in range(4):
        w2 = w.copy()
        pos = rng.choice(R * n, size=2000, replace=False)
        w2[pos] = special[rng.integers(0, special.size, size=pos.size)]
        encs = []
        for j in range(R):
            sh = w2[j * n:(j + 1) * n]
            expect = orc.encode(sh, gu.host_u8(send[j]), B)
            cap = int(ciera.ciera_encoded_bound(n, B))
            buf = torch.empty(cap, dtype=torch.uint8, device="cuda")
            nb = torch.zeros(1, dtype=torch.int64, device="cuda")
            ciera.encode_t(gu.dev_bits(sh), send[j], B, ws_e, buf,
                           out_bytes=nb, update_cache=True)
            torch.cuda.synchronize()
            got = gu.host_u8(buf)[:int(nb.item())]
            np.testing.assert_array_equal(got, expect, err_msg=f"t={t}")
            encs.append(expect)
        gathered, offs = gu.gather(encs)
        ciera.decode_gathered_t(gu.dev_u8(gathered),
                                torch.from_numpy(offs.view(np.int64)).cuda(),
                                n, B, out, recv, ws_d)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(gu.host_u16(out), w2, err_msg=f"t={t}")
        np.testing.assert_array_equal(
            gu.host_u8(recv), np.concatenate([gu.host_u8(c) for c in send]))
        w = w2
    assert ws_e.error() == 0 and ws_d.error() == 0
