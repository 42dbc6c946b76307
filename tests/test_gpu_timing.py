"""ciera_time_next_call: the next library call's kernels stamp the caller's
events (the first kernel the start, the last one the end), the request
ends with that call, and a call that fails clears it. The stamped span of
an encode must lie inside the span of events recorded around the same call
on the same stream."""
import ctypes

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000


class _Hip:
    def __init__(self):
        self.h = ctypes.CDLL("libamdhip64.so.7")  # the runtime torch loaded
        self.h.hipEventCreateWithFlags.argtypes = [
            ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.h.hipEventElapsedTime.argtypes = [
            ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.h.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def event(self, flags=HIP_EVENT_DISABLE_SYSTEM_FENCE):
        e = ctypes.c_void_p()
        assert self.h.hipEventCreateWithFlags(ctypes.byref(e), flags) == 0
        return e

    def elapsed_ms(self, a, b):
        """(status, ms) of hipEventElapsedTime(a, b)."""
        ms = ctypes.c_float()
        rc = self.h.hipEventElapsedTime(ctypes.byref(ms), a, b)
        return rc, ms.value


@pytest.fixture(scope="module")
def env():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_04609_amd import ciera
    ciera.lib()
    return ciera, _Hip()


def _encode_inputs(n, B):
    from paper_2609_04609_amd import ciera, synth
    w = synth.normal_bf16_bits(n, 0.02, 901, "cuda")
    w2 = synth.forced_bernoulli_bits(w, 0.01, 902)
    cache = ((w.to(torch.int32) >> 7) & 0xFF).to(torch.uint8)
    ws = ciera.Workspace(n, 1, B)
    out = torch.empty(int(ciera.ciera_encoded_bound(n, B)), dtype=torch.uint8,
                      device="cuda")
    return w2, cache, ws, out


@pytest.mark.parametrize("B", [1, 512])
def test_stamped_span_inside_marker_span(env, B):
    ciera, hip = env
    n = 1 << 24
    w2, cache, ws, out = _encode_inputs(n, B)
    stream = torch.cuda.current_stream()
    for _ in range(3):
        ciera.encode_t(w2, cache, B, ws, out)
    m0, m1 = hip.event(), hip.event()
    k0, k1 = hip.event(), hip.event()
    assert hip.h.hipEventRecord(m0, stream.cuda_stream) == 0
    ciera.ciera_time_next_call(k0, k1)
    ciera.encode_t(w2, cache, B, ws, out)
    assert hip.h.hipEventRecord(m1, stream.cuda_stream) == 0
    torch.cuda.synchronize()
    rc_k, t_k = hip.elapsed_ms(k0, k1)
    rc_m, t_m = hip.elapsed_ms(m0, m1)
    assert rc_k == 0 and rc_m == 0
    # 33.5 MB of W' and 16.8 MB of cache take microseconds, not nothing
    assert 0.002 < t_k <= t_m + 0.002, (t_k, t_m)
    for e in (m0, m1, k0, k1):
        hip.h.hipEventDestroy(e)


def test_request_covers_one_call(env):
    """A second call without a new request leaves the events as the first
    call stamped them; a failing call ends the request too."""
    ciera, hip = env
    n, B = 1 << 22, 512
    w2, cache, ws, out = _encode_inputs(n, B)
    k0, k1 = hip.event(), hip.event()
    ciera.ciera_time_next_call(k0, k1)
    ciera.encode_t(w2, cache, B, ws, out)
    torch.cuda.synchronize()
    rc, t1 = hip.elapsed_ms(k0, k1)
    assert rc == 0 and t1 > 0
    for _ in range(2):
        ciera.encode_t(w2, cache, B, ws, out)
    torch.cuda.synchronize()
    rc, t2 = hip.elapsed_ms(k0, k1)
    assert rc == 0 and t2 == t1
    # a request followed by a refused call (B = 3): nothing is stamped, and
    # the next good call does not take the request over
    f0, f1 = hip.event(), hip.event()
    ciera.ciera_time_next_call(f0, f1)
    rc = ciera.lib().ciera_encode(w2.data_ptr(), cache.data_ptr(), n, 3, 0,
                                  out.data_ptr(), out.numel(), None,
                                  ws.ptr, ws.nbytes,
                                  torch.cuda.current_stream().cuda_stream)
    assert rc == ciera.EUNSUPPORTED
    ciera.encode_t(w2, cache, B, ws, out)
    torch.cuda.synchronize()
    rc, _ = hip.elapsed_ms(f0, f1)
    assert rc != 0
    for e in (k0, k1, f0, f1):
        hip.h.hipEventDestroy(e)


def test_pending_hip_error_is_not_reported(env):
    """A HIP error that the caller's own earlier call left pending (here the
    elapsed time of two events never recorded) does not come back as the
    library's CIERA_EHIP."""
    ciera, hip = env
    a, b = hip.event(), hip.event()
    assert hip.elapsed_ms(a, b)[0] != 0
    ws = ciera.Workspace(1 << 16, 1, 512)  # ciera_workspace_init
    assert ws.error() == 0
    for e in (a, b):
        hip.h.hipEventDestroy(e)


def test_stamped_decode_is_exact(env, orc):
    """A stamped call computes what an unstamped one does."""
    ciera, hip = env
    from paper_2609_04609_amd import synth
    R, n, B = 4, 1 << 20, 512
    encs, caches, ws2 = [], [], []
    for j in range(R):
        w = synth.normal_bf16_bits(n, 0.02, 950 + j)
        w2 = synth.forced_bernoulli_bits(w, 0.003, 960 + j)
        c = orc.split(w.numpy().view(np.uint16))[0]
        encs.append(orc.encode(w2.numpy().view(np.uint16), c, B))
        caches.append(c)
        ws2.append(w2.numpy().view(np.uint16))
    offs = np.cumsum([0] + [e.size for e in encs[:-1]]).astype(np.uint64)
    g = torch.from_numpy(np.concatenate(encs)).cuda()
    o = torch.from_numpy(offs.view(np.int64)).cuda()
    cache = torch.from_numpy(np.concatenate(caches)).cuda()
    out = torch.empty(R * n, dtype=torch.int16, device="cuda")
    ws = ciera.Workspace(n, R, B)
    k0, k1 = hip.event(), hip.event()
    ciera.ciera_time_next_call(k0, k1)
    ciera.decode_gathered_t(g, o, n, B, out, cache, ws)
    torch.cuda.synchronize()
    assert ws.error() == 0
    assert hip.elapsed_ms(k0, k1)[0] == 0
    np.testing.assert_array_equal(out.cpu().numpy().view(np.uint16),
                                  np.concatenate(ws2))
    for e in (k0, k1):
        hip.h.hipEventDestroy(e)
