"""The overlapped schedule (Section 3.3 on one GPU: sender, link, receiver
and compute streams joined by events). Every layer's receiver decodes the
gathered buffer whose rank-0 slot its own sender stream has just overwritten
with 0xFF and then encoded into, so the event waits carry the data: the
oracle redoes that slot's encoding and the decode of every layer's whole
buffer, step after step, in both schedules."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def setup():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import bench
    from paper_2609_04609_amd import synth
    wl = synth.WORKLOADS["olmoe_expert"]  # 16 shards of 131,072 values
    return bench.Setup(wl, 512, torch.device("cuda:0"))


def _h8(t):
    return t.cpu().numpy().view(np.uint8)


def _h16(t):
    return t.cpu().numpy().view(np.uint16)


def _check_with_oracle(orc, P, before):
    """Layer by layer: rank 0's slot equals the oracle's encoding of the
    step's input against the sender cache the step started from, and the
    decoded values and caches equal the oracle's decode of the layer's
    gathered buffer against the receiver caches the step started from."""
    n, B = P.n, P.B
    side = P.parity ^ 1
    w_in = _h16(P.S.W2[:n] if side == 0 else P.S.W[:n])
    for i in range(P.L):
        send0, recv0 = before[i]
        g, off = P.last_gathered(i)
        gh = _h8(g)
        exp0 = orc.encode(w_in, send0, B)
        np.testing.assert_array_equal(gh[:exp0.size], exp0,
                                      err_msg=f"layer {i} slot 0")
        cache_o = recv0.copy()
        out_o = orc.decode_gathered(gh, off.cpu().numpy().view(np.uint64), n,
                                    cache_o)
        np.testing.assert_array_equal(_h16(P.outs[i]), out_o,
                                      err_msg=f"layer {i} values")
        np.testing.assert_array_equal(_h8(P.caches[i]), cache_o,
                                      err_msg=f"layer {i} caches")
        np.testing.assert_array_equal(_h8(P.send[i]), cache_o[:n])


def _state(P):
    return [(_h8(P.send[i]).copy(), _h8(P.caches[i]).copy())
            for i in range(P.L)]


def test_overlapped_schedule_carries_the_data(setup, orc):
    from paper_2609_04609_amd.pipeline import OverlapPipeline
    P = OverlapPipeline(setup, 3, 1e12, tokens=64)
    for overlapped in (False, False, True, True, True, True):
        before = _state(P)
        P.step(overlapped)
        assert P.check(), f"overlapped={overlapped}"
        _check_with_oracle(orc, P, before)
    y_ovl = [y.clone() for y in P.y]
    P.step(False)
    P.step(False)  # the same side as the last overlapped step
    for a, b in zip(P.y, y_ovl):
        torch.testing.assert_close(a.float(), b.float(), rtol=1e-2,
                                   atol=1e-2)
    # timing the pieces of layer 0 leaves it where the others are
    comp = P.component_us(reps=2)
    assert set(comp) == {"encode", "link", "decode", "compute"}
    before = _state(P)
    P.step(True)
    assert P.check()
    _check_with_oracle(orc, P, before)
