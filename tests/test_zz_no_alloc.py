"""ciera_decode_gathered_noalloc (the gathered decode that allocates nothing:
its tile offsets live in the library's device scratch array) against
ciera_decode_gathered with a workspace, through the C ABI, bit for bit: two
calls in a row on the same scratch, the second with a smaller input, for the
paths that use the scratch (B = 1 per-tile counts, added up in the merge or
scanned first on large layers; B >= 16 with the prefix pass) and one that
does not; then the error word of a call with a bad shard,
and of the clean call after it."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_04609_amd import ciera
    ciera.lib()
    return ciera


def _gathered(orc, R, n, B, seed):
    """R shards encoded by the oracle against the exponents of W, gathered
    back to back; one raw shard when R > 2."""
    from paper_2609_04609_amd import synth
    encs, caches = [], []
    for j in range(R):
        w = synth.normal_bf16_bits(n, 0.02, seed + j)
        w2 = synth.forced_bernoulli_bits(w, 0.003, seed + 500 + j)
        wh = w.numpy().view(np.uint16)
        w2h = w2.numpy().view(np.uint16)
        c = orc.split(wh)[0]
        raw = R > 2 and j == 1
        encs.append(orc.encode(w2h, None if raw else c, B, raw=raw))
        caches.append(c)
    offs = np.cumsum([0] + [e.size for e in encs[:-1]]).astype(np.uint64)
    return (torch.from_numpy(np.concatenate(encs)).cuda(),
            torch.from_numpy(offs.view(np.int64)).cuda(),
            torch.from_numpy(np.concatenate(caches)).cuda())


def _both(lib, g, o, n, B, cache0):
    """The workspace decode and the no-alloc decode of the same buffer from
    the same caches: (out, cache, error word) of each."""
    R = o.numel()
    ws = lib.Workspace(n, R, B)
    out_w = torch.full((R * n,), 3, dtype=torch.int16, device="cuda")
    cache_w = cache0.clone()
    lib.decode_gathered_t(g, o, n, B, out_w, cache_w, ws)
    out_n = torch.full((R * n,), 5, dtype=torch.int16, device="cuda")
    cache_n = cache0.clone()
    err = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    lib.decode_gathered_noalloc_t(g, o, n, B, out_n, cache_n, err)
    torch.cuda.synchronize()
    return (out_w, cache_w, ws.error()), (out_n, cache_n, int(err.item()))


@pytest.mark.parametrize("B,first,second", [
    (1, (4, 1_000_003), (2, 70_001)),          # per-tile counts summed
    (1, (3, 90_000_007), (2, 70_001)),         # counts scanned, then summed
    (16, (16, 6_000_008), (3, 100_000)),       # prefix pass, then without
    (512, (3, 300_007), (2, 16_385)),          # counts in the tile
])
def test_noalloc_decode_matches_workspace_decode(lib, orc, B, first, second):
    for k, (R, n) in enumerate((first, second)):
        g, o, cache0 = _gathered(orc, R, n, B, 1000 * B + 10 * k)
        (ow, cw, ew), (on, cn, en) = _both(lib, g, o, n, B, cache0)
        assert ew == 0 and en == 0, (B, R, n)
        assert torch.equal(on, ow), (B, R, n)
        assert torch.equal(cn, cw), (B, R, n)


def test_noalloc_decode_error_word(lib, orc):
    """A corrupted header: both decodes skip that shard and report
    CIERA_DEVERR_FORMAT; the next clean call's word is 0 again."""
    B, R, n = 64, 3, 40_001
    g, o, cache0 = _gathered(orc, R, n, B, 77)
    bad = g.clone()
    bad[int(o[2])] ^= 0xFF
    (ow, cw, ew), (on, cn, en) = _both(lib, bad, o, n, B, cache0)
    assert ew == lib.DEVERR_FORMAT and en == lib.DEVERR_FORMAT
    assert torch.equal(on[:2 * n], ow[:2 * n])
    assert bool(torch.all(on[2 * n:] == 5))
    assert torch.equal(cn, cw)
    (ow, cw, ew), (on, cn, en) = _both(lib, g, o, n, B, cache0)
    assert ew == 0 and en == 0
    assert torch.equal(on, ow) and torch.equal(cn, cw)
