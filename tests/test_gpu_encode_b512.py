"""The encode at B = 512 (the paper's default block size) on shards of
2^20 values and more, against the oracle, byte for byte, with and without
the fused cache update: the row-wise exception pass with one tile per wave
and with runs of several tiles (the deeper batch from the updated cache),
ragged last tiles and blocks, a last block changed and unchanged, no change
at all and every block changed, the DeepSeek-style clustered changes, and
calls of different sizes in a row on one workspace."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

B = 512


@pytest.fixture(scope="module")
def gu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util
    from paper_2609_04609_amd import ciera
    ciera.lib()
    return gpu_util


def _check(gu, orc, w2, cache_h, ws=None, msg=""):
    """Plain encode and fused-update encode of W' against cache_h."""
    out, total, ws = gu.gpu_encode(w2, gu.dev_u8(cache_h), B, ws)
    expect = orc.encode(gu.host_u16(w2), cache_h, B)
    assert total == expect.size, msg
    got = gu.host_u8(out)
    np.testing.assert_array_equal(got[:total], expect, err_msg=msg)
    # nothing past the encoded size is written (the buffer was 0xA5)
    assert np.all(got[total:] == 0xA5), msg
    del out
    gu.check_fused_update(orc, w2, cache_h, B, expect, ws, msg="fused " + msg)
    assert ws.error() == 0, msg
    return ws


@pytest.mark.parametrize("n", [1 << 20, (1 << 20) + 1, 25_165_824,
                               25_165_824 + 4097 + 511, 40_000_013,
                               88_080_384])
def test_b512_matches_oracle(gu, orc, n):
    w, w2 = gu.pair(n, 7100 + n % 97, c=0.001)
    cache_h = orc.split(gu.host_u16(w))[0]
    del w
    _check(gu, orc, w2, cache_h, msg=f"n={n}")


@pytest.mark.parametrize("n", [(1 << 21) + 300, (1 << 21) + 512])
@pytest.mark.parametrize("last_changed", [True, False])
def test_b512_last_block(gu, orc, n, last_changed):
    """The last block (partial or whole) changed or not: E takes the last
    block's length, and its exceptions stop at n."""
    w, w2 = gu.pair(n, 7300 + n % 13, c=0.0)  # W' == W: no change at all
    wh = gu.host_u16(w).copy()
    w2h = wh.copy()
    # a change in the first block and, or not, in the last value
    w2h[5] ^= 1 << 7
    if last_changed:
        w2h[n - 1] ^= 1 << 7
    else:
        w2h[n - 600] ^= 1 << 7  # the block before the last
    cache_h = orc.split(wh)[0]
    _check(gu, orc, gu.dev_bits(w2h), cache_h,
           msg=f"n={n} last_changed={last_changed}")


@pytest.mark.parametrize("c", [0.0, 0.3])
def test_b512_no_change_and_all_changed(gu, orc, c):
    n = 3 * (1 << 20) + 77
    w, w2 = gu.pair(n, 7400, c=c)
    cache_h = orc.split(gu.host_u16(w))[0]
    expect = orc.encode(gu.host_u16(w2), cache_h, B)
    E = int(expect[32:40].view(np.uint64)[0])
    assert (E == 0) if c == 0.0 else (E == n)
    _check(gu, orc, w2, cache_h, msg=f"c={c}")


def test_b512_clustered_changes(gu, orc):
    """The DeepSeek-style pattern on one 88,080,384-value shard: 90% of the
    changes in 10% of the 4096-value blocks."""
    from paper_2609_04609_amd import synth
    wl = synth.WORKLOADS["dsv3_layer"]
    w, w2 = synth.shard_pair(wl, 3, "cuda")
    cache_h = orc.split(gu.host_u16(w))[0]
    del w
    _check(gu, orc, w2, cache_h, msg="dsv3 shard 3")


def test_b512_calls_in_a_row(gu, orc):
    """A large call, a small one and a large one again on one workspace: the
    second large call's tiles sit where the first one's status words are."""
    from paper_2609_04609_amd import ciera
    big, small = 30_000_011, (1 << 20) + 4096
    ws = ciera.Workspace(big, 1, B)
    for k, n in enumerate([big, small, big, small]):
        w, w2 = gu.pair(n, 7500 + k, c=0.002 * (k + 1))
        cache_h = orc.split(gu.host_u16(w))[0]
        del w
        _check(gu, orc, w2, cache_h, ws, msg=f"call {k} n={n}")
