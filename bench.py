"""Benchmark of the CIERA codec hot path on one MI355X.

One step is one iteration of the codec for one tensor group, as rank 0 of R
ranks sees it:
  1. the Section 3.2 compress-or-not decision for the group (host);
  2. ciera_encode of rank 0's shard against its exponent cache, bringing
     that cache forward in the same pass (CIERA_ENC_UPDATE_CACHE);
  3. ciera_decode_gathered over all R encoded shards placed back to back in
     one HBM buffer (the one-GPU stand-in for the Allgather output), which
     patches the R receiver caches and rebuilds every bf16 value.
Steps alternate between the update W -> W' and its reverse W' -> W, so every
step changes the same set of exponents against caches that really hold the
previous iteration's exponents, and the work per step is constant.

The headline workload is the DeepSeek-V3-style MoE layer (256 experts, 128
shards of 88,080,384 values, 0.5% clustered exponent changes, B = 512), the
largest configuration that fits one GPU. Beside it: the OLMoE layer (16
shards of 25,165,824 values) at B = 512 and at B = 1, its fp16, block-hash,
rANS and overlap variants, the small configurations and one layer of the
mixed model step.

Inputs are resident in HBM before timing starts. Phase times come from HIP
timing events recorded on the stream the kernels run on, right before and
after each library call, created without the system-scope fence a default
event makes (its L2 write-back idles the stream for microseconds). The CPU
oracle is timed on the host cores as a reported baseline, on the same bytes,
streamed shard by shard.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--block B]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, 8 TB/s
COPY_CAL_BYTES = 1 << 30
# the kernels and their launch configuration (grids, tile orders, passes)
KERNEL_SRC = [os.path.join(ROOT, "paper_2609_04609_amd", "csrc", f)
              for f in ("ciera_kernels.hip", "ciera_internal.h",
                        "ciera_api.cpp")]
# HBM bytes per call measured with rocprofv3 FETCH_SIZE + WRITE_SIZE (each
# scaled by what the counters read for a 1 GiB copy) for the sources whose
# concatenation has this sha256; see profiles/hbm_traffic_*.md. Reported only
# while those sources are unchanged.
_SRC_SHA = "af9052628ae3d84f8ef73c869c5cab68544f0451f31ad7e535ecdd7522c7e00d"
MEASURED_TRAFFIC = {
    # ciera_decode_gathered (tile_prefix_kernel + decode_kernel) and the
    # fused-update ciera_encode (encode_pass_kernel + encode_exc_rows_kernel)
    ("dsv3_layer", 512, "bf16"): {"sha": _SRC_SHA, "decode": 48928094659,
                                  "encode": 423501392},
    ("olmoe_layer_c0.1", 512, "bf16"): {"sha": _SRC_SHA,
                                        "decode": 1778761534,
                                        "encode": 123671142},
}


def measured_traffic(name, B, dtype="bf16"):
    """{"decode": bytes, "encode": bytes} of the current kernel source, or
    None when no counter run covers it."""
    rec = MEASURED_TRAFFIC.get((name, B, dtype))
    if rec is None:
        return None
    return rec if source_digest() == rec["sha"] else None


def source_digest():
    """sha256 of the kernel and launch sources, concatenated in order."""
    import hashlib
    h = hashlib.sha256()
    for path in KERNEL_SRC:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


METRIC = ("encode & N-shard decode GB/s (bf16 weights), % HBM peak, "
          "wire-bytes ratio")


class TimingEvent:
    """A HIP event for timing only, created with hipEventDisableSystemFence:
    recording it makes no system-scope release, so it neither writes back
    nor invalidates the L2 between the kernels it brackets (a default event
    does both, which costs the stream about 5 us per event on MI355X and
    moves the write-back of one kernel's dirty lines into the gap). The
    timestamps are read after a device synchronisation. With fenced=True it
    is a default (fenced) timing event instead, for comparison."""
    _hip = None
    fenced = False

    def __init__(self):
        import ctypes
        if TimingEvent._hip is None:
            lib = ctypes.CDLL("libamdhip64.so.7")  # the runtime torch loaded
            lib.hipEventCreateWithFlags.argtypes = [
                ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventElapsedTime.argtypes = [
                ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                ctypes.c_void_p]
            lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
            TimingEvent._hip = lib
        self._h = ctypes.c_void_p()
        flags = 0 if TimingEvent.fenced else 0x20000000
        if TimingEvent._hip.hipEventCreateWithFlags(ctypes.byref(self._h),
                                                    flags) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, stream):
        if self._hip.hipEventRecord(self._h, stream.cuda_stream) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, end):
        """Milliseconds from this event to `end` (both recorded and done)."""
        import ctypes
        ms = ctypes.c_float()
        if self._hip.hipEventElapsedTime(ctypes.byref(ms), self._h,
                                         end._h) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def __del__(self):
        if getattr(self, "_h", None) and self._hip is not None:
            self._hip.hipEventDestroy(self._h)


class Span:
    """The time one library call takes on its stream: timing events recorded
    right before and right after it."""

    def __init__(self):
        self.a, self.b = TimingEvent(), TimingEvent()

    def arm(self, stream):
        self.a.record(stream)

    def close(self, stream):
        self.b.record(stream)

    def us(self):
        return self.a.elapsed_time(self.b) * 1e3


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def describe(wl, B):
    if wl.name.startswith("olmoe_layer"):
        shape = ("OLMoE-1B-7B MoE layer: 64 experts x (gate 2048x1024, up "
                 "2048x1024, down 1024x2048) bf16")
        change = f"forced uniform exponent change c={wl.rate * 100:g}%"
    elif wl.name == "dsv3_layer":
        shape = ("DeepSeek-V3-style MoE layer: 256 experts x (gate 7168x2048, "
                 "up 7168x2048, down 2048x7168) bf16")
        change = ("0.5% exponent change, clustered: 10% of 4096-value blocks "
                  "hold 90% of the changes")
    else:
        shape, change = wl.name, wl.update
    return (f"{shape} = {wl.total_elems:,} values, R={wl.shards} shards of "
            f"{wl.shard_elems:,}, {change}, B={B}")


class Setup:
    """All device buffers of one workload, built before any timing. With
    raw=True every gather sends raw shards (tensors the selection rule
    leaves uncompressed)."""

    def __init__(self, wl, B, dev):
        import torch
        from paper_2609_04609_amd import synth
        R, n = wl.shards, wl.shard_elems
        t0 = time.time()
        W = torch.empty(R * n, dtype=torch.int16, device=dev)
        W2 = torch.empty(R * n, dtype=torch.int16, device=dev)
        for j in range(R):
            w, w2 = synth.shard_pair(wl, j, dev)
            W[j * n:(j + 1) * n].copy_(w)
            W2[j * n:(j + 1) * n].copy_(w2)
            del w, w2
        torch.cuda.synchronize()
        log(f"generated {2 * R * n * 2 / 1e9:.2f} GB of bf16 shards "
            f"in {time.time() - t0:.1f}s")
        self._build(wl, W, W2, R, n, B, dev, False, t0)

    @classmethod
    def from_tensors(cls, W, W2, R, n, B, dev, raw=False):
        S = cls.__new__(cls)
        S._build(None, W, W2, R, n, B, dev, raw, time.time())
        return S

    def _build(self, wl, W, W2, R, n, B, dev, raw, t0):
        import torch
        from paper_2609_04609_amd import ciera
        self.wl, self.B, self.dev, self.raw = wl, B, dev, raw
        self.R, self.n, self.W, self.W2 = R, n, W, W2
        self.ws_enc = ciera.Workspace(n, 1, B, dev)
        self.ws_dec = ciera.Workspace(n, R, B, dev)
        self.cap = int(ciera.ciera_encoded_bound(n, B))
        self.tmp = torch.empty(self.cap, dtype=torch.uint8, device=dev)
        self.nbytes = torch.zeros(1, dtype=torch.int64, device=dev)
        self.out = torch.empty(R * n, dtype=torch.int16, device=dev)
        self.cache = torch.empty(R * n, dtype=torch.uint8, device=dev)
        # the first gather after warm-up is raw: it seeds every receiver
        # cache (shard by shard, so no raw copy of the layer is held)
        for j in range(R):
            ciera.encode_t(self.W[j * n:(j + 1) * n], None, B, self.ws_enc,
                           self.tmp, raw=True, out_bytes=self.nbytes)
            ciera.update_cache_t(self.cache[j * n:(j + 1) * n], self.tmp, n,
                                 B, self.ws_enc)
        # A: W -> W' against exp(W);  B: W' -> W against exp(W')
        self.gA, self.offA, self.totA = self._gather(self.W2, self.cache,
                                                     raw=raw)
        ciera.decode_gathered_t(self.gA, self.offA, n, B, self.out,
                                self.cache, self.ws_dec)
        self.gB, self.offB, self.totB = self._gather(self.W, self.cache,
                                                     raw=raw)
        ciera.decode_gathered_t(self.gB, self.offB, n, B, self.out,
                                self.cache, self.ws_dec)
        torch.cuda.synchronize()
        if not (torch.equal(self.out, self.W) and self.ws_dec.error() == 0):
            raise RuntimeError("setup round trip is not exact")
        # rank 0's sender cache holds exp(W) now, like the receivers'
        self.send_cache = self.cache[:n].clone()
        hA = self.gA[:64].cpu().numpy()
        self.changed_blocks = int(hA[24:32].view(np.uint64)[0])
        self.E0 = int(hA[32:40].view(np.uint64)[0])
        log(f"encoded 2 x {R} shards; setup {time.time() - t0:.1f}s")

    def _gather(self, src, cache, raw=False):
        """Encode every rank's shard on the GPU and place them back to back:
        one pass for the sizes, then each shard straight into its place (the
        encoding is deterministic)."""
        import torch
        from paper_2609_04609_amd import ciera
        R, n, B = self.R, self.n, self.B
        totals = []
        for j in range(R):
            ciera.encode_t(src[j * n:(j + 1) * n],
                           None if raw else cache[j * n:(j + 1) * n], B,
                           self.ws_enc, self.tmp, raw=raw,
                           out_bytes=self.nbytes)
            totals.append(int(self.nbytes.item()))
        offs = np.cumsum([0] + totals[:-1]).astype(np.uint64)
        # room for a bound-sized write at the last offset
        g = torch.empty(int(sum(totals)) + self.cap, dtype=torch.uint8,
                        device=self.dev)
        for j in range(R):
            ciera.encode_t(src[j * n:(j + 1) * n],
                           None if raw else cache[j * n:(j + 1) * n], B,
                           self.ws_enc, g[int(offs[j]):], raw=raw,
                           out_bytes=self.nbytes)
            if int(self.nbytes.item()) != totals[j]:
                raise RuntimeError("encode is not deterministic")
        off_t = torch.from_numpy(offs.view(np.int64)).to(self.dev)
        return g, off_t, totals


def codec_step(S, s, stream, se=None, sd=None):
    """Step s of the codec on a Setup: rank 0's encode (bringing its cache
    forward; raw groups encode raw), then the gathered decode. Even steps go
    W -> W', odd steps back. se and sd (Spans) time the two calls."""
    from paper_2609_04609_amd import ciera
    n, B = S.n, S.B
    even = (s % 2) == 0
    w_in = S.W2[:n] if even else S.W[:n]
    g, off = (S.gA, S.offA) if even else (S.gB, S.offB)
    if se is not None:
        se.arm(stream)
    if S.raw:
        ciera.encode_t(w_in, None, B, S.ws_enc, S.tmp, raw=True)
    else:
        ciera.encode_t(w_in, S.send_cache, B, S.ws_enc, S.tmp,
                       update_cache=True)
    if se is not None:
        se.close(stream)
        sd.arm(stream)
    ciera.decode_gathered_t(g, off, n, B, S.out, S.cache, S.ws_dec)
    if sd is not None:
        sd.close(stream)


def check_last_step(S, last):
    """The encoded bytes, decoded values and caches after step `last`, bit
    for bit, and no device error; raises otherwise."""
    import torch
    n = S.n
    last_even = last % 2 == 0
    expect = S.W2 if last_even else S.W
    ok = bool(torch.equal(S.out, expect))
    if not S.raw:
        g, t = (S.gA, S.totA[0]) if last_even else (S.gB, S.totB[0])
        ok = ok and bool(torch.equal(S.cache[:n], S.send_cache)) and \
            bool(torch.equal(S.tmp[:t], g[:t]))
    errs = S.ws_enc.error() | S.ws_dec.error()
    if not ok or errs:
        raise RuntimeError(f"codec steps are not exact (err={errs})")


def timed_steps(S, warmup, steps, stream, decide=None, start=0):
    """The codec step on a Setup (rank 0's encode, bringing its cache
    forward, then the gathered decode; raw groups encode raw), alternating
    W -> W' and back: step s goes W -> W' when s is even, so a sequence of
    calls continues with start = the steps already run. `decide(s)` runs on
    the host before step s (the Section 3.2 decision). Each call is timed
    by a Span. Returns per-step encode and decode times (us) and the wall
    time per step (s). The last step's encoded bytes, decoded values and
    caches are checked bit for bit."""
    import torch

    def one(s, se, sd):
        if decide is not None:
            decide(s)
        codec_step(S, s, stream, se, sd)

    for s in range(warmup):
        one(start + s, None, None)
    spans = [(Span(), Span()) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        one(start + warmup + s, *spans[s])
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    check_last_step(S, start + warmup + steps - 1)
    enc = [se.us() for se, _ in spans]
    dec = [sd.us() for _, sd in spans]
    return enc, dec, wall


def codec_steps(S, warmup, steps, stream):
    """Mean encode and decode times and the wall time per step (s)."""
    enc, dec, wall = timed_steps(S, warmup, steps, stream)
    return float(np.mean(enc)) / 1e6, float(np.mean(dec)) / 1e6, wall


def graph_steps(S, reps, start):
    """The codec step from a HIP graph: steps start and start + 1 (one each
    way, so that replays continue the alternation) captured once, then
    replayed `reps` times between two events on the current stream; the
    library's calls launch kernels only, so they capture as they are.
    Returns us per step; the state after the last replay is checked bit for
    bit."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # one eager pair on a side stream first
        codec_step(S, start, side)
        codec_step(S, start + 1, side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        cap = torch.cuda.current_stream()
        codec_step(S, start, cap)
        codec_step(S, start + 1, cap)
    graph.replay()  # the first replay uploads the graph
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(reps):
        graph.replay()
    b.record()
    torch.cuda.synchronize()
    check_last_step(S, start + 1)
    us = a.elapsed_time(b) * 1e3 / (2 * reps)
    del graph
    return us


def time_small_configs(B, dev, steps, stream):
    """The tiny tensor and the single OLMoE expert (natural update, and 1%
    of exponents forced), R shards each: the codec step as for the layer,
    called from Python, and the same step replayed from a HIP graph
    (us_per_step_graph). These sizes measure launch latency more than
    bandwidth."""
    from paper_2609_04609_amd import synth
    out = {}
    for name in ("tiny", "olmoe_expert", "olmoe_expert_forced"):
        wl = synth.WORKLOADS[name]
        S = Setup(wl, B, dev)
        t_enc, t_dec, wall = codec_steps(S, 10, steps, stream)
        us_graph = graph_steps(S, max(steps, 10), 10 + steps)
        n, R = S.n, S.R
        out[name] = {"workload": describe(wl, B),
                     "us_per_step": round(wall * 1e6, 2),
                     "encode_us": round(t_enc * 1e6, 2),
                     "decode_us": round(t_dec * 1e6, 2),
                     "bf16_gbps": round((2 * n + 2 * R * n) / wall / 1e9, 1),
                     "us_per_step_graph": round(us_graph, 2),
                     "bf16_gbps_graph": round((2 * n + 2 * R * n) /
                                              (us_graph * 1e-6) / 1e9, 1),
                     "wire_ratio": round(sum(S.totA) / (2.0 * R * n), 5)}
        del S
    return out


def time_mixed_layer(B, dev, steps, stream, warmup_regime=False):
    """One layer of the mixed model step (attention q/k/v/o, router, two
    layer norms and the 64-expert group, 16 shards each) at the steady
    per-type change rates, or in the warm-up regime (30% of every tensor's
    exponents change). The Section 3.2 rule decides per tensor on an
    xGMI-class link (alpha 10 us, 150 GB/s per peer) from the block change
    rate of this step's data, with a modelled decode time; the selected
    tensors form one compressed group and the rest one raw group, and the
    layer's codec step is both groups' steps, called from Python and also
    replayed from HIP graphs. All 16 layers of the model have this shape
    and these rates."""
    import torch
    from paper_2609_04609_amd import ciera, synth
    R = synth.MIXED_SHARDS
    shards, dec, ns = {}, {}, {}
    for name, numel, kind in synth.MIXED_TENSORS:
        n = numel // R
        W = torch.empty(R * n, dtype=torch.int16, device=dev)
        W2 = torch.empty_like(W)
        for j in range(R):
            w = synth.normal_bf16_bits(
                n, 0.02, synth.seed_for("mixed", 0, name, j), dev)
            W[j * n:(j + 1) * n] = w
            W2[j * n:(j + 1) * n] = synth.forced_bernoulli_bits(
                w, synth.WARMUP_RATE if warmup_regime else
                synth.STEADY_RATE[kind],
                synth.seed_for("mixed", 0, name, "u", j))
        e1 = (W.view(R, n).to(torch.int32) >> 7) & 0xFF
        e2 = (W2.view(R, n).to(torch.int32) >> 7) & 0xFF
        nb = -(-n // B)
        d = torch.nn.functional.pad((e1 != e2).to(torch.int8),
                                    (0, nb * B - n))
        q = float(d.view(R, nb, B).amax(dim=2).float().mean())
        t_dec_model = 5e-6 + R * (4 * n + q * n) / 5.5e12
        dec[name], _ = ciera.ciera_should_compress(
            n, B, q, R, 10e-6, 150e9, t_decmp_s=t_dec_model)
        shards[name] = (W, W2, n)
        ns[name] = n
        del e1, e2, d
    res = {"workload": ("mixed model step, one of 16 identical layers: "
                        "q/k/v/o 2048x2048, router 2048x64, 2 layer norms "
                        "of 2048, 64 experts x 3 matrices; R=16, " +
                        ("warm-up regime, 30% of exponents change"
                         if warmup_regime else "steady per-type rates")),
           "compressed": sorted(k for k, v in dec.items() if v),
           "raw": sorted(k for k, v in dec.items() if not v)}
    total_us, total_graph_us, vals = 0.0, 0.0, 0
    for raw in (False, True):
        names = [nm for nm, _, _ in synth.MIXED_TENSORS
                 if bool(dec[nm]) != raw]
        if not names:
            continue
        n_flat = sum(ns[nm] for nm in names)
        Wf = torch.empty(R * n_flat, dtype=torch.int16, device=dev)
        W2f = torch.empty_like(Wf)
        for j in range(R):
            off = j * n_flat
            for nm in names:
                W, W2, n = shards[nm]
                Wf[off:off + n] = W[j * n:(j + 1) * n]
                W2f[off:off + n] = W2[j * n:(j + 1) * n]
                off += n
        S = Setup.from_tensors(Wf, W2f, R, n_flat, B, dev, raw=raw)
        t_enc, t_dec, wall = codec_steps(S, 5, steps, stream)
        us_graph = graph_steps(S, max(steps, 10), 5 + steps)
        key = "raw_group" if raw else "compressed_group"
        res[key] = {"values_per_shard": n_flat,
                    "us_per_step": round(wall * 1e6, 2),
                    "encode_us": round(t_enc * 1e6, 2),
                    "decode_us": round(t_dec * 1e6, 2),
                    "us_per_step_graph": round(us_graph, 2),
                    "wire_ratio": round(sum(S.totA) / (2.0 * R * n_flat), 5)}
        total_us += wall * 1e6
        total_graph_us += us_graph
        vals += R * n_flat
        del S, Wf, W2f
    res["us_per_layer"] = round(total_us, 2)
    res["bf16_gbps"] = round(2 * vals / (total_us * 1e-6) / 1e9, 1)
    # the same two group steps, each replayed from a HIP graph
    res["us_per_layer_graph"] = round(total_graph_us, 2)
    return res


def time_update_cache(S, steps, stream):
    """ciera_update_cache on its own: rank 0's shard applied to a copy of its
    cache (idempotent, so the calls repeat), HIP events."""
    import torch
    from paper_2609_04609_amd import ciera
    n, B = S.n, S.B
    c = S.send_cache.clone()
    enc = S.gA[:int(S.totA[0])]
    for _ in range(3):
        ciera.update_cache_t(c, enc, n, B, S.ws_enc)
    spans = [Span() for _ in range(steps)]
    for sp in spans:
        sp.arm(stream)
        ciera.update_cache_t(c, enc, n, B, S.ws_enc)
        sp.close(stream)
    torch.cuda.synchronize()
    return float(np.mean([sp.us() for sp in spans])) / 1e6


def algorithmic_bytes(n, R, B, E_list, changed_list):
    """Bytes each kernel must move at minimum (B >= 16).
    encode: read 2n (W') + n (cache); write n (sign|mantissa) + bm + E + 64
            (the fused cache update adds one byte per changed exponent).
    decode: per shard read 64 + n (sign|mantissa) + bm + (n - E) cache + E
            exceptions; write 2n (values) + E (cache patch).
    update_cache: read 64 + bm + E, write E."""
    blocks = -(-n // B)
    bm = -(-blocks // 8)
    E0 = E_list[0]
    enc = 2 * n + n + n + bm + E0 + 64
    dec = sum(64 + n + bm + (n - E) + E + 2 * n + E for E in E_list)
    upd = 64 + bm + 2 * E0
    return enc, dec, upd


def time_encode_hashed(S, steps, stream, cache_is_w2):
    """The sender's pass with the HashCache detector of Algorithm 1 in place
    of the exponent cache, on the same shards as the timed step (W' against
    the hashes of W, and back). Checked byte for byte against the exact
    encoder on the sender cache as the timed loop left it (the exponents of
    W' when cache_is_w2, else of W), then event-timed on the kernels' stream."""
    import torch
    from paper_2609_04609_amd import ciera
    n, B = S.n, S.B
    nb = -(-n // B)
    hW = torch.empty(2 * nb, dtype=torch.int64, device=S.dev)
    hW2 = torch.empty_like(hW)
    hout = torch.empty_like(hW)
    ciera.hash_blocks_t(S.W[:n], B, hW)
    ciera.hash_blocks_t(S.W2[:n], B, hW2)
    ref = torch.empty_like(S.tmp)
    out = torch.empty_like(S.tmp)
    # the input that differs from what the cache holds, and its hashes
    w_in, h_in, h_new = ((S.W[:n], hW2, hW) if cache_is_w2
                         else (S.W2[:n], hW, hW2))
    ciera.encode_t(w_in, S.send_cache, B, S.ws_enc, ref, out_bytes=S.nbytes)
    torch.cuda.synchronize()
    t_ref = int(S.nbytes.item())
    ciera.encode_hashed_t(w_in, h_in, hout, B, S.ws_enc, out,
                          out_bytes=S.nbytes)
    torch.cuda.synchronize()
    if int(S.nbytes.item()) != t_ref or not torch.equal(out[:t_ref],
                                                        ref[:t_ref]):
        raise RuntimeError("hashed and exact encodes differ")
    if not torch.equal(hout, h_new):
        raise RuntimeError("HashCache update is wrong")
    pairs = [(S.W2[:n], hW), (S.W[:n], hW2)]
    for i in range(4):
        ciera.encode_hashed_t(pairs[i % 2][0], pairs[i % 2][1], hout, B,
                              S.ws_enc, out)
    spans = [Span() for _ in range(steps)]
    for i in range(steps):
        spans[i].arm(stream)
        ciera.encode_hashed_t(pairs[i % 2][0], pairs[i % 2][1], hout, B,
                              S.ws_enc, out)
        spans[i].close(stream)
    torch.cuda.synchronize()
    t = np.mean([sp.us() for sp in spans]) / 1e6
    bm = -(-nb // 8)
    alg = 2 * n + 16 * nb + n + bm + S.E0 + 64 + 16 * nb
    return {"us": round(t * 1e6, 2), "bf16_gbps": round(2 * n / t / 1e9, 1),
            "hbm_gbps": round(alg / t / 1e9, 1),
            "hbm_frac": round(alg / t / 1e9 / HBM_PEAK_GBPS, 4),
            "alg_bytes": alg,
            "note": "HashCache detector (16 B per block) in place of the "
                    "exponent cache; same wire bytes as the exact encode"}


def time_ans(S, steps, stream, cache_is_w2):
    """The exception sections rANS-coded (Section 3.1's ANS step): coding of
    rank 0's freshly encoded shard (events around ciera_ans_code), and the
    decode of gathered buffers in which every shard is coded, alternating
    W -> W' and back like the timed step. Checked bit for bit."""
    import torch
    from paper_2609_04609_amd import ciera
    n, B, R = S.n, S.B, S.R
    ws1 = ciera.Workspace(n, 1, B, S.dev, ans=True)
    wsR = ciera.Workspace(n, R, B, S.dev, ans=True)

    def coded_gather(g, off, tots):
        parts, totals = [], []
        buf = torch.empty(S.cap, dtype=torch.uint8, device=S.dev)
        offs = off.cpu().numpy().astype(np.int64)
        for j in range(R):
            buf[:tots[j]].copy_(g[offs[j]:offs[j] + tots[j]])
            ciera.ans_code_t(buf, n, B, ws1, out_bytes=S.nbytes)
            t = int(S.nbytes.item())
            totals.append(t)
            parts.append(buf[:t].clone())
        o = np.cumsum([0] + totals[:-1]).astype(np.int64)
        gg = torch.cat(parts)
        return gg, torch.from_numpy(o).to(S.dev), totals

    gA, oA, tA = coded_gather(S.gA, S.offA, S.totA)
    gB, oB, tB = coded_gather(S.gB, S.offB, S.totB)
    h = gA[:64].cpu().numpy()
    mode0 = int(h[6:8].view(np.uint16)[0])
    bm = -(-(-(-n // B)) // 8)
    C0 = int(h[40:48].view(np.uint64)[0]) - n - bm if mode0 == 2 else None
    # coding time: encode (fresh mode-0 bytes) then code, events between
    w_in = S.W[:n] if cache_is_w2 else S.W2[:n]
    out = torch.empty_like(S.tmp)
    spans = [Span() for _ in range(steps)]
    for i in range(steps + 3):
        sp = spans[i - 3] if i >= 3 else None
        ciera.encode_t(w_in, S.send_cache, B, S.ws_enc, out)
        if sp: sp.arm(stream)
        ciera.ans_code_t(out, n, B, ws1)
        if sp: sp.close(stream)
    torch.cuda.synchronize()
    t_code = np.mean([sp.us() for sp in spans]) / 1e6
    # decode of the coded buffers, starting on the side the caches are at
    pairs = [(gB, oB, S.W), (gA, oA, S.W2)] if cache_is_w2 else \
        [(gA, oA, S.W2), (gB, oB, S.W)]
    dspans = [Span() for _ in range(steps)]
    for i in range(steps):
        g, o, _ = pairs[i % 2]
        dspans[i].arm(stream)
        ciera.decode_gathered_t(g, o, n, B, S.out, S.cache, wsR)
        dspans[i].close(stream)
    torch.cuda.synchronize()
    expect = pairs[(steps - 1) % 2][2]
    if not torch.equal(S.out, expect) or wsR.error() != 0:
        raise RuntimeError("rANS-coded decode is not exact")
    # put the caches back on the side the rest of the bench expects
    if steps % 2 == 1:
        g, o, _ = pairs[1]
        ciera.decode_gathered_t(g, o, n, B, S.out, S.cache, wsR)
        torch.cuda.synchronize()
    t_dec = np.mean([sp.us() for sp in dspans]) / 1e6
    E0 = S.E0
    q_eff = (C0 if C0 is not None else E0) / n
    dec, gain = ciera.ciera_should_compress(n, B, q_eff, R, 10e-6, 8e9,
                                            t_decmp_s=t_dec)
    return {"wire_ratio": round(sum(tA) / (2.0 * R * n), 5),
            "exceptions_local": E0,
            "coded_exceptions_local": C0,
            "code_us": round(t_code * 1e6, 2),
            "decode_us": round(t_dec * 1e6, 2),
            "decode_bf16_gbps": round(2 * R * n / t_dec / 1e9, 1),
            "should_compress": {"decision": int(dec), "gain_s": gain,
                                "q_effective": round(q_eff, 5)},
            "note": "exception sections rANS-coded (mode 2); decode = "
                    "ans_decode_kernel + decode_kernel"}


def time_f16(wl, B, dev, steps, stream):
    """The same layer geometry in fp16 (the paper's second precision, Table
    2): N(0, std) weights rounded to fp16, the workload's forced exponent
    change rate, R encoded shards gathered in HBM; encode of rank 0's shard
    bringing its cache forward, and decode of all R, alternating W -> W' and
    back, checked exact."""
    import torch
    from paper_2609_04609_amd import ciera, synth
    R, n = wl.shards, wl.shard_elems
    c = wl.rate if wl.rate else 0.001
    W = torch.empty(R * n, dtype=torch.int16, device=dev)
    W2 = torch.empty_like(W)
    for j in range(R):
        w = synth.normal_f16_bits(n, wl.std, synth.seed_for(wl.name + "f16",
                                                               j, 0), dev)
        W[j * n:(j + 1) * n].copy_(w)
        W2[j * n:(j + 1) * n].copy_(
            synth.forced_bernoulli_f16_bits(w, c, synth.seed_for(
                wl.name + "f16", j, 1)))
    cap = int(ciera.ciera_encoded_bound(n, B, ciera.FP16))
    ws_e = ciera.Workspace(n, 1, B, dev)
    ws_d = ciera.Workspace(n, R, B, dev)
    tmp = torch.empty(cap, dtype=torch.uint8, device=dev)
    nb = torch.zeros(1, dtype=torch.int64, device=dev)
    out = torch.empty_like(W)
    cache = torch.empty(R * n, dtype=torch.uint8, device=dev)

    def gather(src, raw):
        parts, tots = [], []
        for j in range(R):
            ciera.encode_t(src[j * n:(j + 1) * n],
                           None if raw else cache[j * n:(j + 1) * n], B, ws_e,
                           tmp, raw=raw, out_bytes=nb, fp16=True)
            t = int(nb.item())
            tots.append(t)
            parts.append(tmp[:t].clone())
        offs = np.cumsum([0] + tots[:-1]).astype(np.int64)
        return torch.cat(parts), torch.from_numpy(offs).to(dev), tots

    g0, o0, _ = gather(W, True)
    ciera.decode_gathered_t(g0, o0, n, B, out, cache, ws_d, fp16=True)
    del g0
    gA, oA, tA = gather(W2, False)
    ciera.decode_gathered_t(gA, oA, n, B, out, cache, ws_d, fp16=True)
    gB, oB, _ = gather(W, False)
    ciera.decode_gathered_t(gB, oB, n, B, out, cache, ws_d, fp16=True)
    torch.cuda.synchronize()
    send = cache[:n].clone()  # exp(W)
    hA = gA[:64].cpu().numpy()
    E0 = int(hA[32:40].view(np.uint64)[0])
    pairs = [(W2, gA, oA), (W, gB, oB)]
    spans = [(Span(), Span()) for _ in range(steps)]
    for i in range(steps + 2):
        w_in, g, o = pairs[i % 2]
        se, sd = spans[i - 2] if i >= 2 else (None, None)
        if se: se.arm(stream)
        ciera.encode_t(w_in[:n], send, B, ws_e, tmp, fp16=True,
                       update_cache=True)
        if se: se.close(stream)
        if sd: sd.arm(stream)
        ciera.decode_gathered_t(g, o, n, B, out, cache, ws_d, fp16=True)
        if sd: sd.close(stream)
    torch.cuda.synchronize()
    last = (steps + 1) % 2
    if not torch.equal(out, pairs[last][0]) or ws_d.error() or ws_e.error():
        raise RuntimeError("fp16 steps are not exact")
    t_enc = np.mean([se.us() for se, _ in spans]) / 1e6
    t_dec = np.mean([sd.us() for _, sd in spans]) / 1e6
    nbk = -(-n // B)
    bm = -(-nbk // 8)
    S_sm = n + 3 * (-(-n // 8))
    exc = lambda E: 5 * (-(-E // 8))
    E_list = []
    for j in range(R):
        h = gA[int(oA[j]):int(oA[j]) + 64].cpu().numpy()
        E_list.append(int(h[32:40].view(np.uint64)[0]))
    # the fused cache update writes one byte per changed exponent
    alg_enc = 2 * n + n + S_sm + bm + exc(E0) + 64 + E0
    alg_dec = sum(64 + S_sm + bm + (n - E) + exc(E) + 2 * n + E
                  for E in E_list)
    return {"workload": f"{wl.name} geometry in fp16, forced c={c * 100:g}%",
            "wire_ratio": round(sum(tA) / (2.0 * R * n), 5),
            "encode_us": round(t_enc * 1e6, 2),
            "encode_hbm_frac": round(alg_enc / t_enc / 1e9 / HBM_PEAK_GBPS, 4),
            "decode_us": round(t_dec * 1e6, 2),
            "decode_bf16_gbps": round(2 * R * n / t_dec / 1e9, 1),
            "decode_hbm_gbps": round(alg_dec / t_dec / 1e9, 1),
            "decode_hbm_frac": round(alg_dec / t_dec / 1e9 / HBM_PEAK_GBPS, 4),
            "decode_alg_bytes": alg_dec,
            "decode_traffic": (measured_traffic(wl.name, B, "fp16") or
                               {}).get("decode"),
            "exceptions_local": E0}


XGMI_GATHER_BPS = 7 * 153e9  # one MI355X's 7 xGMI links, direct gather


def time_overlap(S, layers, steps, cache_is_w2):
    """Section 3.3 on one GPU: L layer groups, sequential vs overlapped
    (sender, link, receiver and compute streams joined by events); the
    Allgather is a spin kernel lasting its alpha-beta time on the xGMI
    links. Every layer's output is checked bit for bit."""
    from paper_2609_04609_amd.pipeline import OverlapPipeline
    P = OverlapPipeline(S, layers, XGMI_GATHER_BPS,
                        caches_hold_w2=cache_is_w2)
    comp = P.component_us()
    res = {}
    for mode in (False, True):
        P.step(mode)  # warm-up
        P.step(mode)
        ts = [P.step(mode) for _ in range(2 * steps)]
        if not P.check():
            raise RuntimeError("overlap schedule output is not exact")
        res["overlapped" if mode else "sequential"] = float(np.median(ts))
    link = float(np.mean(P.link_us))
    floor = layers * link + comp["decode"] + comp["compute"]
    out = {"layers": layers,
           "link": (f"alpha 10 us + (R-1) x / {XGMI_GATHER_BPS / 1e9:.0f} "
                    "GB/s (7 xGMI links of 153 GB/s, direct gather)"),
           "sequential_us": round(res["sequential"], 1),
           "overlapped_us": round(res["overlapped"], 1),
           "speedup": round(res["sequential"] / res["overlapped"], 3),
           "per_layer_us": comp,
           "link_bound_us": round(floor, 1),
           "note": "link_bound_us = L x link + one decode + one compute: "
                   "the overlapped schedule's floor"}
    del P
    return out


def cpu_baseline(S, budget_s=20.0):
    """The oracle on the host cores, on the same bytes as the GPU step,
    streamed shard by shard (each shard's inputs copied from the device and
    its receiver cache split from W just before use): the encode of rank 0's
    shard on one thread; the decode of gathered shards on one thread, shard
    after shard, for about a third of the budget; and the decode of every
    one of the R shards with one shard per thread on up to 16 cores (a
    host's share of cores per GPU), in rounds of one shard per thread. The step
    rate is encode + that all-core decode of all R shards."""
    import concurrent.futures as cf
    from oracle import oracle
    oracle.build(force=False)
    n, R, B = S.n, S.R, S.B
    offs = S.offA.cpu().numpy().view(np.uint64)
    tot = S.totA

    def shard_inputs(j):
        w = S.W[j * n:(j + 1) * n].cpu().numpy().view(np.uint16)
        enc = S.gA[int(offs[j]):int(offs[j]) + tot[j]].cpu().numpy()
        return oracle.split(w)[0], enc

    cache0, enc0 = shard_inputs(0)
    w2 = S.W2[:n].cpu().numpy().view(np.uint16)
    t0 = time.perf_counter()
    enc = oracle.encode(w2, cache0, B)
    t_enc = time.perf_counter() - t0
    if not np.array_equal(enc, enc0):
        raise RuntimeError("oracle and GPU encodings of shard 0 differ")
    del enc
    # one thread, shard after shard
    t_1, k1 = 0.0, 0
    while k1 == 0 or (t_1 < budget_s / 3 and k1 < R):
        c, e = (cache0.copy(), enc0) if k1 == 0 else shard_inputs(k1)
        t0 = time.perf_counter()
        out = oracle.decode(e, n, c)
        t_1 += time.perf_counter() - t0
        if k1 == 0 and not np.array_equal(out, w2):
            raise RuntimeError("oracle decode of shard 0 is not exact")
        k1 += 1
    del out, w2
    threads = max(1, min(16, os.cpu_count() or 1, R))
    t_all, k_all = 0.0, 0
    with cf.ThreadPoolExecutor(threads) as ex:
        while k_all < R and (k_all == 0 or t_all < budget_s):
            js = list(range(k_all, min(R, k_all + threads)))
            inputs = list(ex.map(shard_inputs, js))
            t0 = time.perf_counter()
            list(ex.map(lambda ce: oracle.decode(ce[1], n, ce[0]), inputs))
            t_all += time.perf_counter() - t0
            k_all += len(js)
            del inputs
    t_step = t_enc + t_all * R / k_all
    return {"value": round((2 * n + 2 * R * n) / t_step / 1e9, 4),
            "unit": "GB/s", "cores": threads, "kind": "oracle",
            "encode_1thread_gbps": round(2 * n / t_enc / 1e9, 4),
            "decode_1thread_gbps": round(2 * n * k1 / t_1 / 1e9, 4),
            "decode_allcores_gbps": round(2 * n * k_all / t_all / 1e9, 4),
            "sample": (f"encode of rank 0's shard ({n:,} values, 1 thread, "
                       f"{t_enc:.2f} s); decode of {k1} shard(s) on 1 thread "
                       f"({t_1:.1f} s); decode of {k_all} of {R} shards, one "
                       f"per thread on {threads} threads ({t_all:.1f} s)"
                       + ("" if k_all == R else
                          f", scaled to all {R}") +
                       "; shards streamed from the GPU set-up one at a "
                       "time")}


def copy_ceiling(dev, stream, nbytes=2 << 30, reps=10):
    """A plain device copy of nbytes (torch copy_ of uint8 tensors), event
    timed: read + write bytes per second (GB/s)."""
    import torch
    src = torch.ones(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    evs = [(TimingEvent(),
            TimingEvent()) for _ in range(reps)]
    for a, b in evs:
        a.record(stream)
        dst.copy_(src)
        b.record(stream)
    torch.cuda.synchronize()
    t = float(np.median([a.elapsed_time(b) for a, b in evs])) / 1e3
    del src, dst
    torch.cuda.empty_cache()
    return 2 * nbytes / t / 1e9


def spread(v):
    return [round(float(x), 2) for x in np.percentile(v, [10, 50, 90])]


_PROBE = None


def probe_lib():
    """libciera_probe.so (built beside libciera.so by build()): the encode-
    and decode-shaped stream probes."""
    global _PROBE
    if _PROBE is None:
        import ctypes
        path = os.path.join(ROOT, "paper_2609_04609_amd", "libciera_probe.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: run build() first")
        lib = ctypes.CDLL(path)
        for f in (lib.ciera_probe_encode_shaped, lib.ciera_probe_decode_shaped):
            f.restype = ctypes.c_int
        lib.ciera_probe_encode_shaped.argtypes = (
            [ctypes.c_void_p] * 3 + [ctypes.c_uint64, ctypes.c_int,
                                     ctypes.c_void_p])
        lib.ciera_probe_decode_shaped.argtypes = (
            [ctypes.c_void_p] * 3 + [ctypes.c_uint64, ctypes.c_void_p])
        _PROBE = lib
    return _PROBE


def encode_xcd_runs(n, B):
    """Whether the encode's streaming pass walks its workgroups in runs of 32
    per XCD at this shard size and block size: the library's own rule (the
    exception pass gives each wave two tiles or more, B >= 16), restated so
    that the encode-shaped probe takes the same order."""
    if B < 16:
        return False
    l = B.bit_length() - 1
    tile = 4096 if l <= 9 else 8 << l
    tiles = max(1, -(-n // tile))
    waves = 8192 if l >= 9 else 16384
    return -(-tiles // waves) >= 2


def time_stream_ceiling(S, steps, stream, start):
    """The codec step's access patterns with none of its arithmetic, timed in
    the codec's own slots: `steps` more codec steps (continuing the W <-> W'
    alternation from step `start`), each with the decode-shaped probe right
    after its encode and the encode-shaped probe right after its decode.
    encode-shaped: read 2n + n bytes, write n (the streaming pass's pattern);
    decode-shaped: read R n + R n bytes, write 2 R n (the merge's)."""
    import torch
    from paper_2609_04609_amd import ciera
    n, B, R = S.n, S.B, S.R
    lib = probe_lib()
    h = torch.cuda.current_stream().cuda_stream
    scratch = torch.empty(n, dtype=torch.uint8, device=S.dev)
    runs = int(encode_xcd_runs(n, B))
    sm = S.gA[:R * n] if S.gA.numel() >= R * n else None
    pe, pd = [], []
    for i in range(steps + 2):
        s = start + i
        even = s % 2 == 0
        w_in = S.W2[:n] if even else S.W[:n]
        g, off = (S.gA, S.offA) if even else (S.gB, S.offB)
        ciera.encode_t(w_in, S.send_cache, B, S.ws_enc, S.tmp,
                       update_cache=True)
        sd = Span()
        if sm is not None:
            sd.arm(stream)
            rc = lib.ciera_probe_decode_shaped(sm.data_ptr(), S.cache.data_ptr(),
                                               S.out.data_ptr(), R * n, h)
            sd.close(stream)
            if rc:
                raise RuntimeError("decode-shaped probe failed")
        ciera.decode_gathered_t(g, off, n, B, S.out, S.cache, S.ws_dec)
        se = Span()
        se.arm(stream)
        rc = lib.ciera_probe_encode_shaped(w_in.data_ptr(),
                                           S.send_cache.data_ptr(),
                                           scratch.data_ptr(), n, runs, h)
        se.close(stream)
        if rc:
            raise RuntimeError("encode-shaped probe failed")
        if i >= 2:
            pe.append(se)
            if sm is not None:
                pd.append(sd)
    torch.cuda.synchronize()
    last_even = (start + steps + 1) % 2 == 0
    if not torch.equal(S.out, S.W2 if last_even else S.W):
        raise RuntimeError("codec steps around the probes are not exact")
    t_e = float(np.mean([x.us() for x in pe])) / 1e6
    out = {"encode_shaped_us": round(t_e * 1e6, 2),
           "encode_shaped_gbps": round(4 * n / t_e / 1e9, 1)}
    if pd:
        t_d = float(np.mean([x.us() for x in pd])) / 1e6
        out["decode_shaped_us"] = round(t_d * 1e6, 2)
        out["decode_shaped_gbps"] = round(4 * R * n / t_d / 1e9, 1)
    return out


def measure_layer(S, args, stream, decide_link_bps=8e9):
    """The timed codec steps of one Setup and their figures: per-phase times,
    algorithmic bytes and HBM fractions (decode and encode rooflines), the
    stand-alone cache update, the wire ratio and the Section 3.2 decision
    taken every step on an inter-node link (the paper's ~8 GB/s bus, alpha
    10 us) with the decode time measured in warm-up."""
    import torch
    from paper_2609_04609_amd import ciera
    wl, B, R, n = S.wl, S.B, S.R, S.n
    q = S.changed_blocks / max(1, -(-n // B))
    decision = {"t_decmp_s": 0.0}

    def decide(s):
        decision["dec"], decision["gain"] = ciera.ciera_should_compress(
            n, B, q, R, 10e-6, decide_link_bps,
            t_decmp_s=decision["t_decmp_s"])

    if args.warmup:
        _, dec_w, _ = timed_steps(S, 0, args.warmup, stream, decide)
        decision["t_decmp_s"] = float(np.mean(dec_w)) / 1e6
    enc_us, dec_us, wall = timed_steps(S, 0, args.steps, stream, decide,
                                       start=args.warmup)
    t_enc = float(np.mean(enc_us)) / 1e6
    t_dec = float(np.mean(dec_us)) / 1e6
    # an even number of steps (with the two warm-up ones) leaves the caches
    # on the side the timed steps left them
    ceil = time_stream_ceiling(S, 2 * max(1, args.steps // 4), stream,
                               args.warmup + args.steps)
    t_upd = time_update_cache(S, args.steps, stream)
    # exponents that changed in rank 0's shard: the fused cache update's bytes
    d0 = ((S.W[:n].to(torch.int32) ^ S.W2[:n].to(torch.int32)) >> 7) & 0xFF
    changed_vals = int((d0 != 0).sum().item())
    del d0
    E_A = []
    for j in range(R):
        h = S.gA[int(S.offA[j]):int(S.offA[j]) + 64].cpu().numpy()
        E_A.append(int(h[32:40].view(np.uint64)[0]))
    b_enc, b_dec, b_upd = algorithmic_bytes(n, R, B, E_A, None)
    b_enc += changed_vals
    tr = measured_traffic(wl.name, B)
    dec_gbps = b_dec / t_dec / 1e9
    enc_gbps = b_enc / t_enc / 1e9
    return {
        "workload": describe(wl, B),
        "ms_per_step": round(wall * 1e3, 4),
        "bf16_gbps": round((2 * n + 2 * R * n) / wall / 1e9, 2),
        "encode": {"us": round(t_enc * 1e6, 2),
                   "us_p10_p50_p90": spread(enc_us),
                   "bf16_gbps": round(2 * n / t_enc / 1e9, 1),
                   "hbm_gbps": round(enc_gbps, 1),
                   "hbm_frac": round(enc_gbps / HBM_PEAK_GBPS, 4),
                   "alg_bytes": b_enc},
        "decode": {"us": round(t_dec * 1e6, 2),
                   "us_p10_p50_p90": spread(dec_us),
                   "bf16_gbps": round(2 * R * n / t_dec / 1e9, 1),
                   "hbm_gbps": round(dec_gbps, 1),
                   "hbm_frac": round(dec_gbps / HBM_PEAK_GBPS, 4),
                   "alg_bytes": b_dec},
        "update_cache": {"us": round(t_upd * 1e6, 2),
                         "hbm_gbps": round(b_upd / t_upd / 1e9, 1),
                         "alg_bytes": b_upd},
        "roofline": {"bound": "hbm",
                     "kernel": ("tile_prefix_kernel + decode_kernel "
                                "(ciera_decode_gathered)" if B > 1 else
                                "count_tile_bits + scan_counts + "
                                "decode_elems_kernel (ciera_decode_gathered)"),
                     "achieved": round(dec_gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(dec_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": tr["decode"] if tr else None},
        "roofline_encode": {"bound": "hbm",
                            "kernel": ("encode_pass_kernel + exception pass "
                                       "(ciera_encode with the fused cache "
                                       "update)"),
                            "achieved": round(enc_gbps, 1),
                            "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                            "frac": round(enc_gbps / HBM_PEAK_GBPS, 4),
                            "traffic": tr["encode"] if tr else None},
        "stream_ceiling": {
            **ceil,
            "encode_frac_of_stream": round(
                enc_gbps / ceil["encode_shaped_gbps"], 4),
            **({"decode_frac_of_stream": round(
                dec_gbps / ceil["decode_shaped_gbps"], 4)}
               if "decode_shaped_gbps" in ceil else {}),
            "note": ("stream probes with the codec's access patterns and no "
                     "codec arithmetic, timed in its slots of the step: "
                     "encode-shaped after the decode (4n bytes), "
                     "decode-shaped after the encode (4Rn bytes); the "
                     "fractions compare algorithmic GB/s")},
        "wire_ratio": round(sum(S.totA) / (2.0 * R * n), 5),
        "q_blocks": round(q, 5),
        "exceptions_local": E_A[0],
        "should_compress": {"decision": int(decision["dec"]),
                            "gain_s": decision["gain"],
                            "link": "alpha 10us, 8 GB/s per rank pair"},
        "verified": ("every step's encode bytes equal rank 0's gathered "
                     "slot; the last decoded layer equals W' (or W) bit for "
                     "bit and the sender cache equals the receivers'"),
        "_cache_is_w2": (args.warmup + args.steps - 1) % 2 == 0,
    }


def run(args):
    import torch
    from paper_2609_04609_amd import ciera, synth

    if not os.path.exists(ciera.LIB_PATH):
        from paper_2609_04609_amd import build
        build.build()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    wl = synth.WORKLOADS[args.workload]
    B = args.block
    S = Setup(wl, B, dev)
    R, n = S.R, S.n
    rec = measure_layer(S, args, stream)
    rec.pop("_cache_is_w2")
    copy_gbps = copy_ceiling(dev, stream)
    ms = rec["ms_per_step"]
    res = {
        "metric": METRIC,
        "value": rec["bf16_gbps"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": rec["workload"], "name": wl.name,
                   "shards": R, "shard_elems": n, "block_elems": B},
        "roofline": rec["roofline"],
        "roofline_encode": rec["roofline_encode"],
        "encode": rec["encode"],
        "decode": rec["decode"],
        "update_cache": rec["update_cache"],
        "wire_ratio": rec["wire_ratio"],
        "q_blocks": rec["q_blocks"],
        "exceptions_local": rec["exceptions_local"],
        "should_compress": rec["should_compress"],
        "copy_ceiling": {
            "gbps": round(copy_gbps, 1),
            "frac_of_peak": round(copy_gbps / HBM_PEAK_GBPS, 4),
            "decode_frac_of_copy": round(
                rec["decode"]["hbm_gbps"] / copy_gbps, 4),
            "encode_frac_of_copy": round(
                rec["encode"]["hbm_gbps"] / copy_gbps, 4),
            "note": "a plain 2 GiB device copy (torch copy_), read + write "
                    "bytes per second"},
        "stream_ceiling": rec["stream_ceiling"],
        "verified": rec["verified"],
        "timing": ("HIP events recorded on the kernels' stream right "
                   "before and after each call (" +
                   ("default, fenced" if TimingEvent.fenced else
                    "hipEventDisableSystemFence") + ")"),
    }
    if args.cpu_baseline:
        log("timing the CPU oracle")
        res["cpu_baseline"] = cpu_baseline(S)
    del S
    torch.cuda.empty_cache()

    if args.others:
        # the OLMoE layer: the same record at B = 512 and at B = 1, then its
        # block-hash, rANS, fp16 and overlap variants
        olmoe = synth.WORKLOADS["olmoe_layer_c0.1"]
        So = Setup(olmoe, 512, dev)
        ro = measure_layer(So, args, stream)
        w2_side = ro.pop("_cache_is_w2")
        ro["encode_hashed"] = time_encode_hashed(So, args.steps, stream,
                                                 w2_side)
        ro["ans"] = (time_ans(So, args.steps, stream, w2_side)
                     if args.ans else None)
        ro["overlap"] = (time_overlap(So, args.overlap_layers, 3, w2_side)
                         if args.overlap_layers > 0 else None)
        res["olmoe_layer"] = ro
        del So
        torch.cuda.empty_cache()
        So1 = Setup(olmoe, 1, dev)
        r1 = measure_layer(So1, args, stream)
        r1.pop("_cache_is_w2")
        res["olmoe_layer_b1"] = r1
        del So1
        torch.cuda.empty_cache()
        res["fp16"] = (time_f16(olmoe, 512, dev, args.steps, stream)
                       if args.fp16 else None)
        res["small_configs"] = time_small_configs(512, dev, args.steps,
                                                  stream)
        res["mixed_layer"] = time_mixed_layer(512, dev,
                                              min(args.steps, 20), stream)
        res["mixed_layer_warmup"] = time_mixed_layer(
            512, dev, min(args.steps, 20), stream, warmup_regime=True)
        # the OLMoE layer's other forced change rates (1% and 5%)
        for name in ("olmoe_layer_c1", "olmoe_layer_c5"):
            Sr = Setup(synth.WORKLOADS[name], 512, dev)
            rr = measure_layer(Sr, args, stream)
            rr.pop("_cache_is_w2")
            res[name] = rr
            del Sr
            torch.cuda.empty_cache()
    if args.copy_calibration:
        # a plain device copy of a known size, for scaling the HBM byte
        # counters of a rocprofv3 --pmc run of this same command
        src = torch.ones(COPY_CAL_BYTES, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="dsv3_layer")
    ap.add_argument("--block", type=int, default=512)
    ap.add_argument("--no-cpu-baseline", dest="cpu_baseline",
                    action="store_false")
    ap.add_argument("--no-ans", dest="ans", action="store_false",
                    help="skip the rANS-coded exception measurements")
    ap.add_argument("--no-fp16", dest="fp16", action="store_false",
                    help="skip the fp16 measurement")
    ap.add_argument("--overlap-layers", type=int, default=4,
                    help="layer groups in the overlap measurement (0: skip)")
    ap.add_argument("--no-others", dest="others", action="store_false",
                    help="time the headline workload only (no OLMoE layer "
                         "records, small configurations or mixed layer)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="finish with three 1 GiB device copies (counter "
                         "calibration for rocprofv3 --pmc runs)")
    ap.add_argument("--fenced-events", action="store_true",
                    help="time with default HIP events (a system-scope "
                         "release at every event) instead of fence-free ones")
    args = ap.parse_args()
    TimingEvent.fenced = args.fenced_events
    if args.gpus != 1:
        print("bench.py measures one GPU: the codec is rank-local and the "
              "Allgather is stood in for by one HBM buffer, so --gpus must "
              "be 1", file=sys.stderr)
        sys.exit(2)
    run(args)


if __name__ == "__main__":
    main()
