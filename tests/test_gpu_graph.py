"""The codec step captured in a HIP graph (torch.cuda.CUDAGraph over the
library's launches) and replayed: the sender's encode with the fused cache
update, the copy of its bytes into rank 0's slot of the gathered buffer, and
the gathered decode (with a workspace, and the allocation-free entry point).
Between replays eager work restores the inputs and poisons the outputs; every
replay must give the oracle's bytes, values and caches, as the eager calls
do. The calls launch kernels only (no memset nodes, no allocation, no host
synchronisation), which is what makes them capturable."""
import numpy as np
import pytest
import torch

from tests.gpu_util import dev_bits, dev_u8, host_u16, host_u8
from paper_2609_04609_amd import ciera, synth

pytestmark = pytest.mark.gpu

N = 1_000_003  # ragged: 245 encode tiles, 62 decode tiles per shard
R = 4
REPLAYS = 4


def _inputs(orc, B, seed):
    w2s, e0 = [], []
    for j in range(R):
        w = synth.normal_bf16_bits(N, 0.02, seed + 2 * j, "cpu")
        w2 = synth.forced_bernoulli_bits(w, 0.005, seed + 2 * j + 1)
        wh, w2h = host_u16(w), host_u16(w2)
        w2s.append(w2h)
        e0.append(orc.split(wh)[0])
    encs = [orc.encode(w2s[j], e0[j], B) for j in range(R)]
    offs = np.cumsum([0] + [e.size for e in encs[:-1]]).astype(np.uint64)
    gathered = np.concatenate(encs)
    cache_o = np.concatenate(e0)
    out_o = orc.decode_gathered(gathered, offs, N, cache_o)
    return w2s, e0, encs, offs, gathered, out_o, cache_o


@pytest.mark.parametrize("B", [1, 512])
def test_captured_step_replays_match_oracle(orc, B):
    w2s, e0, encs, offs, gathered, out_o, cache_o = _inputs(orc, B, 7100 + B)
    L = encs[0].size
    send_o = orc.split(w2s[0])[0]  # the sender's cache after its step
    win = dev_bits(w2s[0])
    send0 = dev_u8(e0[0])
    recv0 = dev_u8(np.concatenate(e0))
    g = dev_u8(gathered)
    off = torch.from_numpy(offs.view(np.int64)).cuda()
    send = send0.clone()
    cache = recv0.clone()
    out = torch.empty(R * N, dtype=torch.int16, device="cuda")
    ws_enc = ciera.Workspace(N, 1, B)
    ws_dec = ciera.Workspace(N, R, B)
    cap = int(ciera.ciera_encoded_bound(N, B))
    enc = torch.empty(cap, dtype=torch.uint8, device="cuda")
    nb = torch.zeros(1, dtype=torch.int64, device="cuda")

    def step():
        ciera.encode_t(win, send, B, ws_enc, enc, out_bytes=nb,
                       update_cache=True)
        g[:L].copy_(enc[:L])
        ciera.decode_gathered_t(g, off, N, B, out, cache, ws_dec)

    def reset():
        send.copy_(send0)
        cache.copy_(recv0)
        g[:L].fill_(0xFF)
        enc.fill_(0xA5)
        out.fill_(0)
        nb.zero_()

    def check(what):
        torch.cuda.synchronize()
        assert int(nb.item()) == L, what
        np.testing.assert_array_equal(host_u8(enc[:L]), encs[0], err_msg=what)
        np.testing.assert_array_equal(host_u8(send), send_o, err_msg=what)
        np.testing.assert_array_equal(host_u16(out), out_o, err_msg=what)
        np.testing.assert_array_equal(host_u8(cache), cache_o, err_msg=what)
        assert ws_dec.error() == 0 and ws_enc.error() == 0, what

    # eager first (on a side stream, as torch wants before a capture)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        reset()
        step()
    torch.cuda.current_stream().wait_stream(side)
    check("eager")

    graph = torch.cuda.CUDAGraph()
    reset()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        step()
    for r in range(REPLAYS):
        reset()
        graph.replay()
        check(f"replay {r}")
        # eager calls between the replays, on the same buffers
        reset()
        step()
        check(f"eager after replay {r}")


@pytest.mark.parametrize("B", [1, 512])
def test_captured_noalloc_decode_replays_match_oracle(orc, B):
    """The allocation-free decode under capture: its scratch address is
    taken on the first call (eager, before the capture)."""
    _, e0, _, offs, gathered, out_o, cache_o = _inputs(orc, B, 7300 + B)
    g = dev_u8(gathered)
    off = torch.from_numpy(offs.view(np.int64)).cuda()
    recv0 = dev_u8(np.concatenate(e0))
    cache = recv0.clone()
    out = torch.zeros(R * N, dtype=torch.int16, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")

    def check(what):
        torch.cuda.synchronize()
        assert int(err.item()) == 0, what
        np.testing.assert_array_equal(host_u16(out), out_o, err_msg=what)
        np.testing.assert_array_equal(host_u8(cache), cache_o, err_msg=what)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        ciera.decode_gathered_noalloc_t(g, off, N, B, out, cache, err)
    torch.cuda.current_stream().wait_stream(side)
    check("eager")

    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        ciera.decode_gathered_noalloc_t(g, off, N, B, out, cache, err)
    for r in range(REPLAYS):
        cache.copy_(recv0)
        out.fill_(0)
        err.fill_(-1)
        graph.replay()
        check(f"replay {r}")
