"""CPU-side checks of the library boundary: it loads, exports every symbol
include/ciera.h declares, its host-only calls (sizes, the Section 3.2
selection rule) agree with closed forms and the oracle, and host-side
argument checks reject bad calls before anything is enqueued. No GPU."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def cl():
    from paper_2609_04609_amd import ciera
    if not os.path.exists(ciera.LIB_PATH):
        from paper_2609_04609_amd import build
        build.build()
    ciera.lib()
    return ciera


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "ciera.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ciera_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(cl):
    names = _declared_functions()
    assert len(names) >= 9
    handle = ctypes.CDLL(cl.LIB_PATH)
    for name in names:
        assert hasattr(handle, name), name
    assert set(names) == set(cl.EXPORTED)


def test_sizes_closed_form(cl, orc):
    for n in [0, 1, 15, 16, 17, 4096, 4097, 25165824, 88080384]:
        for B in [1, 16, 64, 512, 4096]:
            S_b = -(-n // B)
            bm = -(-S_b // 8)
            a16 = lambda x: -(-x // 16) * 16
            expect = max(64 + a16(n) + a16(bm) + a16(n), 64 + a16(2 * n))
            assert cl.ciera_encoded_bound(n, B) == expect
            assert orc.encoded_bound(n, B) == expect
    # fp16: sign+mantissa n + 3 ceil(n/8), exceptions 5 ceil(n/8) at most
    for n in [0, 1, 15, 16, 17, 4096, 4097, 25165824]:
        for B in [16, 512, 4096]:
            bm = -(-(-(-n // B)) // 8)
            a16 = lambda x: -(-x // 16) * 16
            c = 64 + a16(n + 3 * (-(-n // 8))) + a16(bm) + a16(5 * (-(-n // 8)))
            assert cl.ciera_encoded_bound(n, B, cl.FP16) == \
                max(c, 64 + a16(2 * n)) == orc.encoded_bound_f16(n, B)
    for B in [0, 2, 3, 8, 24, 8192]:
        assert cl.ciera_encoded_bound(100, B) == 0
        assert cl.ciera_workspace_bytes(100, 1, B) == 0
    # room for rANS coding and decoding: at least the coder's word slots
    # (2 bytes per exception byte) and one list of n bytes per shard
    for n in [1, 4096, 4097, 25165824]:
        base = cl.ciera_workspace_bytes(n, 16, 512)
        ans = cl.ciera_workspace_bytes(n, 16, 512, cl.WS_ANS)
        assert ans >= base + max(2 * n, 16 * n) and ans % 256 == 0
        # no rANS at B = 1: the flag adds nothing there
        assert cl.ciera_workspace_bytes(n, 16, 1, cl.WS_ANS) == \
            cl.ciera_workspace_bytes(n, 16, 1)
    assert cl.ciera_workspace_bytes(100, 1, 512, 2) == 0  # unknown flag
    # every B: the control block, one count per 4096-value encode tile plus
    # the total, and for each shard one offset per 16384-value decode tile
    # plus the total (segments 16-byte aligned)
    for n in [1, 16384, 16385, 88080384]:
        for R in [1, 16, 128]:
            for B in [1, 16, 512, 4096]:
                t_enc = max(1, -(-n // (4096 if B <= 512 else 8 * B)))
                t_dec = -(-n // 16384)
                stride = -(-(t_dec + 1) // 4) * 4
                need = max(256 + 4 * (t_enc + 1), 256 + 4 * R * stride)
                assert cl.ciera_workspace_bytes(n, R, B) >= need, (n, R, B)


def test_host_argument_checks(cl):
    """Rejected before any HIP call: these never touch a device."""
    L = cl.lib()
    ws_bytes = cl.ciera_workspace_bytes(1000, 1, 512)
    fake = 0x10000  # never dereferenced: every call below fails its checks
    # unsupported block size
    assert cl.ciera_encode(fake, fake, 1000, 100, 0, fake, 1 << 20, 0, fake,
                           ws_bytes, 0) == cl.EUNSUPPORTED
    # null output / input / cache
    assert cl.ciera_encode(fake, fake, 1000, 512, 0, 0, 1 << 20, 0, fake,
                           ws_bytes, 0) == cl.EINVAL
    assert cl.ciera_encode(0, fake, 1000, 512, 0, fake, 1 << 20, 0, fake,
                           ws_bytes, 0) == cl.EINVAL
    assert cl.ciera_encode(fake, 0, 1000, 512, 0, fake, 1 << 20, 0, fake,
                           ws_bytes, 0) == cl.EINVAL
    # unknown flag, unaligned output, too-large shard
    assert cl.ciera_encode(fake, fake, 1000, 512, 0x80000000, fake, 1 << 20,
                           0, fake, ws_bytes, 0) == cl.EINVAL
    # the fused cache update needs a cache and no raw form
    assert cl.ciera_encode(fake, fake, 1000, 512,
                           cl.ENC_RAW | cl.ENC_UPDATE_CACHE, fake, 1 << 20, 0,
                           fake, ws_bytes, 0) == cl.EINVAL
    assert cl.ciera_encode(fake, 0, 1000, 512, cl.ENC_UPDATE_CACHE, fake,
                           1 << 20, 0, fake, ws_bytes, 0) == cl.EINVAL
    # fp16 needs B >= 16 (encode, decode, cache update, bound)
    assert cl.ciera_encode(fake, fake, 1000, 1, cl.FP16, fake, 1 << 20, 0,
                           fake, ws_bytes, 0) == cl.EUNSUPPORTED
    MB = 1 << 20  # buffer length of the decoding calls
    assert cl.ciera_decode_gathered(fake, MB, fake, 4, 1000, 1, fake, fake,
                                    fake, ws_bytes, 0,
                                    cl.FP16) == cl.EUNSUPPORTED
    assert cl.ciera_update_cache(fake, fake, MB, 1000, 1, fake, ws_bytes, 0,
                                 cl.FP16) == cl.EUNSUPPORTED
    assert cl.ciera_decode_gathered(fake, MB, fake, 4, 1000, 512, fake, fake,
                                    fake, ws_bytes, 0, 0x80000000) == cl.EINVAL
    assert cl.ciera_encoded_bound(1000, 1, cl.FP16) == 0
    assert cl.ciera_encoded_bound(1000, 512, 0x80000000) == 0
    assert cl.ciera_encode(fake, fake, 1000, 512, 0, fake + 8, 1 << 20, 0,
                           fake, ws_bytes, 0) == cl.EINVAL
    assert cl.ciera_encode(fake, fake, 1 << 32, 512, 0, fake, 1 << 40, 0,
                           fake, ws_bytes, 0) == cl.EINVAL
    # output smaller than the bound, workspace too small
    bound = cl.ciera_encoded_bound(1000, 512)
    assert cl.ciera_encode(fake, fake, 1000, 512, 0, fake, bound - 1, 0, fake,
                           ws_bytes, 0) == cl.ENOSPC
    assert cl.ciera_encode(fake, fake, 1000, 512, 0, fake, bound, 0, fake,
                           256, 0) == cl.ENOSPC
    # decode: zero shards, null offsets, unaligned gathered buffer
    assert cl.ciera_decode_gathered(fake, MB, fake, 0, 1000, 512, fake, fake,
                                    fake, ws_bytes, 0) == cl.EINVAL
    assert cl.ciera_decode_gathered(fake, MB, 0, 4, 1000, 512, fake, fake,
                                    fake, ws_bytes, 0) == cl.EINVAL
    assert cl.ciera_decode_gathered(fake + 4, MB, fake, 4, 1000, 512, fake,
                                    fake, fake, ws_bytes, 0) == cl.EINVAL
    assert cl.ciera_decode_gathered(fake, MB, fake, 4, 1000, 3, fake, fake,
                                    fake, ws_bytes, 0) == cl.EUNSUPPORTED
    assert cl.ciera_update_cache(0, fake, MB, 1000, 512, fake, ws_bytes,
                                 0) == cl.EINVAL
    # the decode without a workspace: a null or misaligned error word, and
    # tile offsets that would not fit its 4 MiB scratch (16 bytes per 4
    # decode tiles of 16384 values, counting one more tile per shard) are
    # refused before any HIP call
    nd = cl.ciera_decode_gathered_noalloc
    assert nd(fake, MB, fake, 4, 1000, 512, fake, fake, 0, 0) == cl.EINVAL
    assert nd(fake, MB, fake, 4, 1000, 512, fake, fake, fake + 2,
              0) == cl.EINVAL
    assert nd(fake, MB, fake, 4, 1000, 3, fake, fake, fake,
              0) == cl.EUNSUPPORTED
    assert nd(fake, MB, fake, 0, 1000, 512, fake, fake, fake,
              0) == cl.EINVAL
    # 256 shards of 4095 tiles fill the scratch exactly; one value more per
    # shard needs a 4096th tile and 4 more words per shard
    assert 256 * 4096 * 4 == 4 << 20
    assert nd(fake, MB, fake, 256, 4095 * 16384 + 1, 512, fake, fake, fake,
              0) == cl.ENOSPC
    assert nd(fake, MB, fake, 16, (1 << 32) - 1, 1, fake, fake, fake,
              0) == cl.ENOSPC
    assert cl.ciera_workspace_init(0, 1024, 0) == cl.EINVAL
    # block hash: B = 1 and unsupported B, null / misaligned hash arrays
    assert cl.ciera_hash_blocks(fake, 1000, 1, fake, 0) == cl.EUNSUPPORTED
    assert cl.ciera_hash_blocks(fake, 1000, 100, fake, 0) == cl.EUNSUPPORTED
    assert cl.ciera_hash_blocks(fake, 1000, 512, 0, 0) == cl.EINVAL
    assert cl.ciera_hash_blocks(fake, 1000, 512, fake + 4, 0) == cl.EINVAL
    assert cl.ciera_hash_blocks(0, 0, 512, 0, 0) == cl.OK  # nothing to do
    assert cl.ciera_encode_hashed(fake, fake, fake, 1000, 1, fake, bound, 0,
                                  fake, ws_bytes, 0) == cl.EUNSUPPORTED
    assert cl.ciera_encode_hashed(fake, 0, fake, 1000, 512, fake, bound, 0,
                                  fake, ws_bytes, 0) == cl.EINVAL
    assert cl.ciera_encode_hashed(fake, fake, fake + 4, 1000, 512, fake,
                                  bound, 0, fake, ws_bytes, 0) == cl.EINVAL
    assert cl.ciera_encode_hashed(fake, fake, fake, 1000, 512, fake,
                                  bound - 1, 0, fake, ws_bytes, 0) == cl.ENOSPC
    assert cl.ciera_encode_hashed(fake, fake, fake, 1000, 512, fake, bound, 0,
                                  fake, 256, 0) == cl.ENOSPC
    # rANS coding: B = 1, null, misaligned, workspace without the rANS room
    ws_ans = cl.ciera_workspace_bytes(1000, 1, 512, cl.WS_ANS)
    assert cl.ciera_ans_code(fake, 1000, 1, 0, fake, ws_ans, 0) == \
        cl.EUNSUPPORTED
    assert cl.ciera_ans_code(0, 1000, 512, 0, fake, ws_ans, 0) == cl.EINVAL
    assert cl.ciera_ans_code(fake + 8, 1000, 512, 0, fake, ws_ans, 0) == \
        cl.EINVAL
    assert cl.ciera_ans_code(fake, 1000, 512, 0, fake, ws_bytes, 0) == \
        cl.ENOSPC
    assert L is not None


# ---------------------------------------------- Section 3.2 selection -----

XGMI = dict(alpha_s=10e-6, bus_bw_Bps=8e9)


def test_gain_hand_computed(cl, orc):
    """n = 1e6, B = 512, q = 0.2, R = 16, alpha = 10 us, bw = 8 GB/s,
    T_decmp = 1 ms, overlapped, 64-byte header. By hand:
      Comm(S)  = 1e-5 + 15 * 2e6 / 8e9            = 0.00376 s
      S_b = ceil(1e6/512) = 1954, S_bm = ceil(1954/8) = 245
      payload  = 1e6 + 245 + 0.2e6 + 64           = 1,200,309 B
      Comm(P)  = 1e-5 + 15 * 1,200,309 / 8e9      = 0.002260579375 s
      g        = 0.00376 - 0.002260579375 - 0.001 = 0.000499420625 s"""
    dec, g = cl.ciera_should_compress(1_000_000, 512, 0.2, 16, 10e-6, 8e9,
                                      t_decmp_s=1e-3)
    assert dec == 1
    assert math.isclose(g, 0.000499420625, rel_tol=1e-12)
    go = orc.gain(1_000_000, 512, 0.2, 16, 10e-6, 8e9, t_decmp_s=1e-3)
    assert math.isclose(go, 0.000499420625, rel_tol=1e-12)
    # not overlapped: T_hash + T_cmp join the critical path
    dec, g2 = cl.ciera_should_compress(1_000_000, 512, 0.2, 16, 10e-6, 8e9,
                                       t_hash_s=2e-4, t_cmp_s=4e-4,
                                       t_decmp_s=1e-3, overlapped=False)
    assert dec == 0 and math.isclose(g2, 0.000499420625 - 6e-4,
                                     rel_tol=1e-9)


def test_gain_fp16_hand_computed(cl, orc):
    """The same shard in fp16 (CIERA_FP16): its sections are S_{s+m} =
    n + 3 ceil(n/8) and S_e = 5 ceil(n/8) bytes. By hand, n = 1e6 (125,000
    octets), B = 512, q = 0.2, R = 16, alpha = 10 us, bw = 8 GB/s,
    T_decmp = 1 ms, overlapped, 64-byte header:
      payload  = 1,375,000 + 245 + 0.2 * 625,000 + 64 = 1,500,309 B
      Comm(P)  = 1e-5 + 15 * 1,500,309 / 8e9          = 0.002823079375 s
      g        = 0.00376 - 0.002823079375 - 0.001     = -0.000063079375 s
    The bf16 shard of the same size gains (above); the fp16 one does not."""
    dec, g = cl.ciera_should_compress(1_000_000, 512, 0.2, 16, 10e-6, 8e9,
                                      t_decmp_s=1e-3, fp16=True)
    assert dec == 0
    assert math.isclose(g, -0.000063079375, rel_tol=1e-12)
    go = orc.gain(1_000_000, 512, 0.2, 16, 10e-6, 8e9, t_decmp_s=1e-3,
                  fp16=True)
    assert math.isclose(go, -0.000063079375, rel_tol=1e-12)
    # a ragged n: ceil(n/8) octets; library and oracle agree over q
    for q in np.linspace(0, 1, 11):
        a = cl.ciera_should_compress(1_000_003, 64, float(q), 8, 5e-6, 50e9,
                                     t_decmp_s=2e-5, fp16=True)[1]
        b = orc.gain(1_000_003, 64, float(q), 8, 5e-6, 50e9, t_decmp_s=2e-5,
                     fp16=True)
        assert math.isclose(a, b, rel_tol=1e-12, abs_tol=1e-15)
    # unknown flags are refused
    st = cl.ShardStats(1000, 512, 0x80, 0.1)
    cm = cl.CostModel(16, 1e-5, 8e9, 0.0, 0.0, 0.0, 64.0, 1)
    assert cl.lib().ciera_should_compress(st, cm, None) == cl.EINVAL


def test_gain_qualitative(cl, orc):
    n, B, R = 25_165_824, 512, 16
    qs = np.linspace(0, 1, 41)
    gains = [cl.ciera_should_compress(n, B, float(q), R, **XGMI,
                                      t_decmp_s=3e-4)[1] for q in qs]
    assert all(a > b for a, b in zip(gains, gains[1:]))  # falls with q
    # every exponent changed: the payload exceeds the raw shard
    assert cl.ciera_should_compress(n, B, 1.0, R, **XGMI)[0] == 0
    # g = 0 is not a gain
    assert cl.ciera_should_compress(0, B, 0.0, R, **XGMI)[0] == 0
    # a tiny tensor (layer-norm shard) cannot repay a 5 us decode
    assert cl.ciera_should_compress(128, B, 0.2, R, **XGMI,
                                    t_decmp_s=5e-6)[0] == 0
    # a fast link and high q: the paper's Scout case selects nothing
    assert cl.ciera_should_compress(4_194_304 // 16, B, 0.96, R,
                                    alpha_s=5e-6, bus_bw_Bps=150e9,
                                    t_decmp_s=5e-6)[0] == 0
    # a low-q expert shard over a slow inter-node link is compressed
    assert cl.ciera_should_compress(n, B, 0.22, R, alpha_s=10e-6,
                                    bus_bw_Bps=8e9, t_decmp_s=3e-4)[0] == 1
    # the library and the oracle agree everywhere
    for q in qs:
        a = cl.ciera_should_compress(n, B, float(q), R, **XGMI,
                                     t_decmp_s=3e-4)[1]
        b = orc.gain(n, B, float(q), R, **XGMI, t_decmp_s=3e-4)
        assert math.isclose(a, b, rel_tol=1e-12, abs_tol=1e-18)


def test_select_ranking_hand_case(cl, orc):
    """g/M ranking under a budget (Section 3.2): shards 0..4 with
    g = [3, 1, -1, 4, 2] ms, M = [3, 2, 1, 2, 1] MB -> ratios
    [1, 0.5, -, 2, 2]; order 3, 4 (tie: lower index first), 0, 1.
    Budget 6 MB: take 3 (2), 4 (3), 0 (6), skip 1 (would be 8)."""
    g = [3e-3, 1e-3, -1e-3, 4e-3, 2e-3]
    m = [3e6, 2e6, 1e6, 2e6, 1e6]
    assert cl.ciera_select(g, m, 6e6) == [True, False, False, True, True]
    assert list(orc.select(g, m, 6e6)) == [True, False, False, True, True]
    # skip-and-continue vs stop at the first misfit
    g2 = [5e-3, 4e-3, 1e-3]
    m2 = [1e6, 4e6, 1e6]        # ratios 5, 1, 1
    assert cl.ciera_select(g2, m2, 2e6) == [True, False, True]
    assert cl.ciera_select(g2, m2, 2e6, cl.SELECT_STOP_AT_MISFIT) == [
        True, False, False]
    assert list(orc.select(g2, m2, 2e6, True)) == [True, False, False]
    # a zero gain is no gain, even where the budget has room for it
    g3, m3 = [2e-3, 0.0, -0.0], [1e6, 1e6, 1e6]
    assert cl.ciera_select(g3, m3, 5e6) == [True, False, False]
    assert list(orc.select(g3, m3, 5e6)) == [True, False, False]
    rng = np.random.default_rng(9)
    for _ in range(50):
        k = int(rng.integers(1, 30))
        gg = rng.normal(size=k).tolist()
        mm = rng.uniform(0.1, 5, size=k).tolist()
        b = float(rng.uniform(0, 20))
        assert cl.ciera_select(gg, mm, b) == list(orc.select(gg, mm, b))
