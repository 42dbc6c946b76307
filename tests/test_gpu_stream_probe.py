"""The benchmark's stream probes (libciera_probe.so): their outputs are the
plain byte maps they state, so that the bytes they move are the ones the
benchmark counts. Not codec parity; the codec is tested elsewhere."""
import ctypes
import os

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROBE = os.path.join(ROOT, "paper_2609_04609_amd", "libciera_probe.so")


def test_probe_library_exports_its_two_calls():
    if not os.path.exists(PROBE):
        from paper_2609_04609_amd import build
        build.build_probe()
    lib = ctypes.CDLL(PROBE)
    for name in ("ciera_probe_encode_shaped", "ciera_probe_decode_shaped"):
        assert hasattr(lib, name), name


@pytest.mark.gpu
@pytest.mark.parametrize("n", [8, 4096, 16384 * 3 + 8, 1 << 20,
                               16384 * 300 + 8,  # 301 tiles: runs and tail
                               16384 * 700 + 8])  # 701 workgroups (encode)
def test_probes_compute_their_byte_maps(n):
    import torch
    import bench
    lib = bench.probe_lib()
    rng = np.random.default_rng(n)
    w = rng.integers(0, 1 << 16, n, dtype=np.uint16)
    c = rng.integers(0, 256, n, dtype=np.uint8)
    sm = rng.integers(0, 256, n, dtype=np.uint8)
    dw = torch.from_numpy(w.view(np.int16)).cuda()
    dc = torch.from_numpy(c).cuda()
    dsm = torch.from_numpy(sm).cuda()
    o8 = torch.empty(n, dtype=torch.uint8, device="cuda")
    o16 = torch.empty(n, dtype=torch.int16, device="cuda")
    h = torch.cuda.current_stream().cuda_stream
    for runs in (0, 1):  # workgroups in order, and in runs of 32 per XCD
        o8.fill_(0)
        assert lib.ciera_probe_encode_shaped(dw.data_ptr(), dc.data_ptr(),
                                             o8.data_ptr(), n, runs, h) == 0
        torch.cuda.synchronize()
        np.testing.assert_array_equal(o8.cpu().numpy(),
                                      ((w >> 8).astype(np.uint8) ^ c))
    assert lib.ciera_probe_decode_shaped(dsm.data_ptr(), dc.data_ptr(),
                                         o16.data_ptr(), n, h) == 0
    torch.cuda.synchronize()
    np.testing.assert_array_equal(
        o16.cpu().numpy().view(np.uint16),
        (c.astype(np.uint16) << 8) | sm.astype(np.uint16))
    # a length that is not a multiple of 8 is refused before any launch
    assert lib.ciera_probe_encode_shaped(dw.data_ptr(), dc.data_ptr(),
                                         o8.data_ptr(), n - 1, 0, h) != 0
