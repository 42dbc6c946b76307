"""The overlapped schedule (Section 3.3 on one GPU: sender, link, receiver
and compute streams joined by events) gives every layer exactly the values
and caches of the one-stream schedule, step after step."""
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


def test_overlapped_equals_sequential(setup):
    from paper_2609_04609_amd.pipeline import OverlapPipeline
    P = OverlapPipeline(setup, 3, 1e12, tokens=64)
    P.step(False)
    assert P.check()
    y_seq = [y.clone() for y in P.y]
    P.step(False)  # back to the start side
    assert P.check()
    for k in range(4):
        P.step(True)
        assert P.check(), f"overlapped step {k}"
        if k == 0:
            for a, b in zip(P.y, y_seq):
                torch.testing.assert_close(a.float(), b.float(), rtol=1e-2,
                                           atol=1e-2)
    # timing the pieces of layer 0 leaves it where the others are
    comp = P.component_us(reps=2)
    assert set(comp) == {"encode", "link", "decode", "compute"}
    assert P.check()
