"""Computation-communication overlap of the codec on one GPU (Section 3.3).

The paper schedules, for every layer i, the sender's hash and compress and
the receiver's cache preparation ahead of the Allgather, so that while
Allgather_i is in flight the codec work of layer i+1 proceeds and only the
decode Decmp_i stays in front of Compute_i. On one GPU this module runs the
same dependency graph for L layer groups in two schedules:

  sequential  every kernel on one stream: encode_i, Allgather_i, decode_i,
              compute_i, layer after layer;
  overlapped  four streams at default priority joined by events:
                sender    encode_0, encode_1, ...           (runs ahead)
                link      Allgather_i after encode_i
                receiver  decode_i after Allgather_i
                compute   compute_i after decode_i

Every layer has its own gathered buffers. The other ranks' shards in them
were placed at set-up; rank 0's slot is filled during the step: the sender
stream first overwrites the slot with 0xFF bytes and then encodes rank 0's
shard into it, and the receiver decodes the buffer. A decode that ran ahead
of its encode would meet a bad header or stale bytes and leave wrong values,
so the schedule's event waits carry the data, not only the timing. The
Allgather itself is a stand-in: a one-thread spin kernel (torch.cuda._sleep)
lasting the alpha-beta time alpha + (R-1) x / bw of the encoded payload x.
Compute_i is a bf16 linear layer over the decoded weights. Encode, cache
update and decode are the library's kernels through the C ABI; nothing here
computes codec data.
"""
from __future__ import annotations

import numpy as np
import torch

from . import ciera


def calibrate_sleep(stream, cycles=2_000_000, reps=5):
    """Microseconds per spin cycle of torch.cuda._sleep on this device."""
    with torch.cuda.stream(stream):
        torch.cuda._sleep(1000)
        evs = [(torch.cuda.Event(enable_timing=True),
                torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in evs:
            a.record(stream)
            torch.cuda._sleep(cycles)
            b.record(stream)
    torch.cuda.synchronize()
    us = np.median([a.elapsed_time(b) * 1e3 for a, b in evs])
    return us / cycles


class OverlapPipeline:
    """L layer groups sharing one set of shards (the codec work per layer is
    the same), each with its own receiver caches, sender cache and output."""

    def __init__(self, setup, layers, link_bw_Bps, alpha_s=10e-6,
                 tokens=256, caches_hold_w2=False):
        S = setup
        self.S, self.L = S, layers
        self.n, self.R, self.B = S.n, S.R, S.B
        dev = S.dev
        self.caches = [S.cache.clone() for _ in range(layers)]
        self.send = [S.send_cache.clone() for _ in range(layers)]
        self.outs = [torch.empty_like(S.out) for _ in range(layers)]
        self.ws_enc = [ciera.Workspace(self.n, 1, self.B, dev)
                       for _ in range(layers)]
        self.ws_dec = [ciera.Workspace(self.n, self.R, self.B, dev)
                       for _ in range(layers)]
        # per layer the A (W -> W') and B (W' -> W) gathered buffers; rank
        # 0's slot [0, total_0) is rewritten by the sender every step
        self.gath = [(S.gA.clone(), S.gB.clone()) for _ in range(layers)]
        self.slot0 = (int(S.totA[0]), int(S.totB[0]))
        # compute stand-in: x [tokens, 4096] times the decoded layer viewed as
        # [R n / 4096, 4096] bf16 weights
        self.k = 4096
        self.rows = (self.R * self.n) // self.k
        self.act = torch.randn(tokens, self.k, device=dev,
                               dtype=torch.bfloat16)
        self.y = [torch.empty(tokens, self.rows, device=dev,
                              dtype=torch.bfloat16) for _ in range(layers)]
        self.s_send = torch.cuda.Stream(device=dev)
        self.s_link = torch.cuda.Stream(device=dev)
        self.s_recv = torch.cuda.Stream(device=dev)
        self.s_comp = torch.cuda.Stream(device=dev)
        self.streams = (self.s_send, self.s_link, self.s_recv, self.s_comp)
        self.us_per_cycle = calibrate_sleep(self.s_link)
        # the link time of one layer's Allgather for the A and B payloads
        self.link_us = []
        for tot in (S.totA, S.totB):
            per_rank = float(np.mean(tot))
            t = alpha_s + (self.R - 1) * per_rank / link_bw_Bps
            self.link_us.append(t * 1e6)
        # 0: the caches hold exp(W), the next step is W -> W' (gA);
        # 1: they hold exp(W'), the next step is W' -> W (gB)
        self.parity = 1 if caches_hold_w2 else 0

    def _inputs(self):
        """(rank 0's new values, A or B side, offsets, link time) of the next
        step."""
        S = self.S
        if self.parity == 0:
            return S.W2[:self.n], 0, S.offA, self.link_us[0]
        return S.W[:self.n], 1, S.offB, self.link_us[1]

    def _poison(self, i, side):
        """Overwrite rank 0's slot of layer i's gathered buffer with 0xFF
        (stale bytes until the sender's encode lands), on the current
        stream."""
        g = self.gath[i][side]
        g[:self.slot0[side]].fill_(0xFF)
        return g

    def _encode(self, i, w_in, side):
        """Encode rank 0's shard into its slot, bringing the sender's cache
        forward, on the current stream."""
        g = self.gath[i][side]
        ciera.encode_t(w_in, self.send[i], self.B, self.ws_enc[i], g,
                       update_cache=True)
        return g

    def _send(self, i, w_in, side):
        self._poison(i, side)
        return self._encode(i, w_in, side)

    def _layer(self, i, w_in, side, off, link_us, st_send, st_link, st_recv,
               st_comp, ev=None):
        n, B = self.n, self.B
        with torch.cuda.stream(st_send):
            g = self._send(i, w_in, side)
            if ev is not None:
                ev["enc"][i].record(st_send)
        with torch.cuda.stream(st_link):
            if ev is not None:
                st_link.wait_event(ev["enc"][i])
            torch.cuda._sleep(int(link_us / self.us_per_cycle))
            if ev is not None:
                ev["link"][i].record(st_link)
        with torch.cuda.stream(st_recv):
            if ev is not None:
                st_recv.wait_event(ev["link"][i])
            ciera.decode_gathered_t(g, off, n, B, self.outs[i],
                                    self.caches[i], self.ws_dec[i])
            if ev is not None:
                ev["dec"][i].record(st_recv)
        with torch.cuda.stream(st_comp):
            if ev is not None:
                st_comp.wait_event(ev["dec"][i])
            w = self.outs[i].view(torch.bfloat16).view(self.rows, self.k)
            torch.mm(self.act, w.t(), out=self.y[i])

    def step(self, overlapped):
        """One iteration over all L layers; returns the wall time in us
        (HIP events on the caller's stream, which every stream joins)."""
        w_in, side, off, link_us = self._inputs()
        main = torch.cuda.current_stream()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(main)
        if overlapped:
            for st in self.streams:
                st.wait_event(t0)
            ev = {k: [torch.cuda.Event() for _ in range(self.L)]
                  for k in ("enc", "link", "dec")}
            for i in range(self.L):
                self._layer(i, w_in, side, off, link_us, *self.streams, ev)
            for st in self.streams:
                done = torch.cuda.Event()
                done.record(st)
                main.wait_event(done)
        else:
            for i in range(self.L):
                self._layer(i, w_in, side, off, link_us, main, main, main,
                            main)
        t1.record(main)
        torch.cuda.synchronize()
        self.parity ^= 1
        return t0.elapsed_time(t1) * 1e3

    def last_gathered(self, i):
        """Layer i's gathered buffer and offsets of the last step."""
        side = self.parity ^ 1
        return self.gath[i][side], (self.S.offA, self.S.offB)[side]

    def check(self):
        """Every layer's output and caches equal the last decoded side, rank
        0's slot holds the bytes of the set-up's encoding of the same shard
        against the same cache, and no device error was raised."""
        S = self.S
        side = self.parity ^ 1
        expect = S.W2 if side == 0 else S.W
        ref = (S.gA, S.gB)[side][:self.slot0[side]]
        for i in range(self.L):
            if not torch.equal(self.outs[i], expect):
                return False
            if not torch.equal(self.caches[i][:self.n], self.send[i]):
                return False
            if not torch.equal(self.gath[i][side][:self.slot0[side]], ref):
                return False
            if self.ws_enc[i].error() or self.ws_dec[i].error():
                return False
        return True

    def component_us(self, reps=5):
        """Stand-alone times of one layer's pieces (events, one stream)."""
        main = torch.cuda.current_stream()
        w_in, side, off, link_us = self._inputs()
        out = {}
        names = ["encode", "link", "decode", "compute"]
        acc = {k: [] for k in names}
        for _ in range(reps):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
            self._poison(0, side)
            ev[0].record(main)
            g = self._encode(0, w_in, side)
            ev[1].record(main)
            torch.cuda._sleep(int(link_us / self.us_per_cycle))
            ev[2].record(main)
            ciera.decode_gathered_t(g, off, self.n, self.B, self.outs[0],
                                    self.caches[0], self.ws_dec[0])
            ev[3].record(main)
            w = self.outs[0].view(torch.bfloat16).view(self.rows, self.k)
            torch.mm(self.act, w.t(), out=self.y[0])
            ev[4].record(main)
            torch.cuda.synchronize()
            for k, name in enumerate(names):
                acc[name].append(ev[k].elapsed_time(ev[k + 1]) * 1e3)
            # undo the encode's sender-cache step and the decode's cache
            # step so that layer 0 stays on the same side as the others
            self._replay_back(0)
        for name in names:
            out[name] = round(float(np.median(acc[name])), 2)
        return out

    def _replay_back(self, i):
        """Bring layer i's caches back by encoding and decoding the reverse
        side."""
        S = self.S
        w_back, side, off = ((S.W[:self.n], 1, S.offB) if self.parity == 0
                             else (S.W2[:self.n], 0, S.offA))
        g = self._send(i, w_back, side)
        ciera.decode_gathered_t(g, off, self.n, self.B, self.outs[i],
                                self.caches[i], self.ws_dec[i])
        torch.cuda.synchronize()
