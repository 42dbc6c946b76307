"""Seeded synthetic inputs for the CIERA codec (bf16 weight shards).

This module only draws numbers: it holds none of the codec's arithmetic, and
both the HIP path and the CPU oracle receive the very bytes it produces. The
paper's models and datasets are not available; these recipes stand in for
them with the shapes and change structure of the workloads the paper studies
(OLMoE-1B-7B and DeepSeek-style expert shards, Section 2 and Section 4):

* weights W ~ N(0, std) drawn in fp32 and rounded to bf16 (round to nearest
  even, torch's conversion);
* a natural update W' = bf16(fp32(W) + noise * N(0, 1));
* a forced update that moves the exponent field of a chosen set of elements
  by +1 or -1 and keeps their sign and mantissa bits (an exponent of 0 always
  moves up, one of 254 or 255 always moves down);
* the chosen set is a Bernoulli(c) draw per element, exactly k elements, or
  a clustered draw in which a random fraction of fixed-size blocks carries
  most of the changes.

Every draw takes an explicit integer seed; ``seed_for`` derives one from the
workload, tensor, shard and purpose so that any shard can be regenerated on
its own. Generation runs on the device given (CPU or a GPU) with torch's
counter-based generator; the bits depend on the device type, so a parity test
generates once and hands the same bytes to both sides.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import torch

BASE_SEED = 0x5EED_C1E2A


def seed_for(*parts) -> int:
    """A 63-bit seed from any tuple of labels (stable across runs)."""
    h = hashlib.blake2b(repr((BASE_SEED,) + tuple(parts)).encode(),
                        digest_size=8)
    return int.from_bytes(h.digest(), "little") & ((1 << 63) - 1)


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def as_bits(x_bf16: torch.Tensor) -> torch.Tensor:
    """bf16 tensor -> its 16-bit patterns (int16 storage, same bytes)."""
    return x_bf16.contiguous().view(torch.int16)


def bits_to_bf16(bits: torch.Tensor) -> torch.Tensor:
    return bits.contiguous().view(torch.bfloat16)


def normal_bf16_bits(numel: int, std: float, seed: int,
                     device="cpu") -> torch.Tensor:
    """W ~ N(0, std) in fp32, rounded to bf16; returned as int16 bit patterns."""
    g = _gen(device, seed)
    x = torch.randn(numel, generator=g, device=device, dtype=torch.float32)
    x.mul_(std)
    return as_bits(x.to(torch.bfloat16))


def natural_update_bits(w_bits: torch.Tensor, noise: float,
                        seed: int) -> torch.Tensor:
    """W' = bf16(fp32(W) + noise * N(0, 1))."""
    g = _gen(w_bits.device, seed)
    z = torch.randn(w_bits.numel(), generator=g, device=w_bits.device,
                    dtype=torch.float32)
    x = bits_to_bf16(w_bits).to(torch.float32)
    x.add_(z, alpha=noise)
    return as_bits(x.to(torch.bfloat16))


def _shift_exponents(w_bits: torch.Tensor, mask: torch.Tensor,
                     up: torch.Tensor) -> torch.Tensor:
    """Move the 8-bit exponent field (bits 14..7) of masked elements by +-1."""
    w = w_bits.to(torch.int32) & 0xFFFF
    field_ = (w >> 7) & 0xFF
    go_up = torch.where(field_ == 0, torch.ones_like(up),
                        torch.where(field_ >= 254, torch.zeros_like(up), up))
    step = torch.where(go_up, 1 << 7, -(1 << 7)).to(torch.int32)
    w = torch.where(mask, w + step, w)
    # back to the int16 storage of the same 16-bit pattern
    w = torch.where(w >= 0x8000, w - 0x10000, w)
    return w.to(torch.int16)


def forced_bernoulli_bits(w_bits: torch.Tensor, c: float,
                          seed: int) -> torch.Tensor:
    """Each element's exponent moves by +-1 with probability c."""
    g = _gen(w_bits.device, seed)
    u = torch.rand(w_bits.numel(), generator=g, device=w_bits.device)
    up = torch.rand(w_bits.numel(), generator=g, device=w_bits.device) < 0.5
    return _shift_exponents(w_bits, u < c, up)


def normal_f16_bits(numel: int, std: float, seed: int,
                    device="cuda") -> torch.Tensor:
    """fp16 bit patterns of N(0, std) weights (fp32 draw, rounded to fp16)."""
    g = _gen(device, seed)
    x = torch.randn(numel, generator=g, device=device, dtype=torch.float32)
    x.mul_(std)
    return x.to(torch.float16).view(torch.int16)


def forced_bernoulli_f16_bits(w_bits: torch.Tensor, c: float,
                              seed: int) -> torch.Tensor:
    """fp16: each element's 5-bit exponent (bits 14..10) moves by +-1 with
    probability c (up from 0, down from 30 and 31)."""
    g = _gen(w_bits.device, seed)
    u = torch.rand(w_bits.numel(), generator=g, device=w_bits.device)
    up = torch.rand(w_bits.numel(), generator=g, device=w_bits.device) < 0.5
    w = w_bits.to(torch.int32) & 0xFFFF
    field_ = (w >> 10) & 0x1F
    go_up = torch.where(field_ == 0, torch.ones_like(up),
                        torch.where(field_ >= 30, torch.zeros_like(up), up))
    step = torch.where(go_up, 1 << 10, -(1 << 10)).to(torch.int32)
    w = torch.where(u < c, w + step, w)
    w = torch.where(w >= 0x8000, w - 0x10000, w)
    return w.to(torch.int16)


def forced_exact_k_bits(w_bits: torch.Tensor, k: int, seed: int):
    """Exactly k distinct elements, uniform at random, move by +-1.

    Returns (new bits, sorted int64 indices of the moved elements)."""
    n = w_bits.numel()
    g = _gen(w_bits.device, seed)
    idx = torch.randperm(n, generator=g, device=w_bits.device)[:k]
    idx, _ = torch.sort(idx)
    mask = torch.zeros(n, dtype=torch.bool, device=w_bits.device)
    mask[idx] = True
    up = torch.rand(n, generator=g, device=w_bits.device) < 0.5
    return _shift_exponents(w_bits, mask, up), idx


def forced_clustered_bits(w_bits: torch.Tensor, c_hot: float, c_cold: float,
                          hot_frac: float, cluster: int, seed: int):
    """A random hot_frac of the cluster-sized blocks draw changes at rate
    c_hot, the rest at c_cold (the DeepSeek-style clustered workload: 10% of
    4096-element blocks hold 90% of a 0.5% change rate)."""
    n = w_bits.numel()
    g = _gen(w_bits.device, seed)
    nclus = (n + cluster - 1) // cluster
    hot = torch.rand(nclus, generator=g, device=w_bits.device) < hot_frac
    rate = torch.where(hot, c_hot, c_cold).repeat_interleave(cluster)[:n]
    u = torch.rand(n, generator=g, device=w_bits.device)
    up = torch.rand(n, generator=g, device=w_bits.device) < 0.5
    return _shift_exponents(w_bits, u < rate, up)


# --------------------------------------------------------------------------
# Workloads. Sizes are the expert and layer shapes of OLMoE-1B-7B (64 experts,
# hidden 2048, expert FFN 1024) and of a DeepSeek-V3-style fine-grained MoE
# layer (256 experts, hidden 7168, expert FFN 2048).
# --------------------------------------------------------------------------

@dataclass
class Workload:
    name: str
    shards: int                 # R: ranks the tensor group is sharded over
    shard_elems: int            # n: bf16 elements in one rank's shard
    std: float                  # weight scale
    update: str                 # "natural" | "bernoulli" | "exact_k" | "clustered"
    rate: float = 0.0           # c for bernoulli / exact_k (fraction)
    noise: float = 1e-4         # natural update scale
    cluster: dict = field(default_factory=dict)

    @property
    def total_elems(self) -> int:
        return self.shards * self.shard_elems


OLMOE_EXPERT = 2048 * 1024 * 3           # gate, up (2048x1024) + down (1024x2048)
OLMOE_LAYER = 64 * OLMOE_EXPERT          # 402,653,184
DSV3_EXPERT = 7168 * 2048 * 3
DSV3_LAYER = 256 * DSV3_EXPERT           # 11,274,289,152

WORKLOADS = {
    # one 1024x1024 tensor, one shard, natural drift
    "tiny": Workload("tiny", 1, 1024 * 1024, 0.02, "natural"),
    # one OLMoE expert matrix (gate 2048x1024, up 2048x1024 or down
    # 1024x2048: 2,097,152 elements each) as 16 row shards, natural drift;
    # the three matrices are three tensors (tag "gate", "up", "down")
    "olmoe_expert": Workload("olmoe_expert", 16, 2048 * 1024 // 16, 0.02,
                             "natural"),
    # same, 1% of elements forced (exactly k per shard)
    "olmoe_expert_forced": Workload("olmoe_expert_forced", 16,
                                    2048 * 1024 // 16, 0.02, "exact_k",
                                    rate=0.01),
    # full OLMoE MoE layer, 16 shards, forced uniform change rates
    "olmoe_layer_c0.1": Workload("olmoe_layer_c0.1", 16, OLMOE_LAYER // 16,
                                 0.02, "bernoulli", rate=0.001),
    "olmoe_layer_c1": Workload("olmoe_layer_c1", 16, OLMOE_LAYER // 16, 0.02,
                               "bernoulli", rate=0.01),
    "olmoe_layer_c5": Workload("olmoe_layer_c5", 16, OLMOE_LAYER // 16, 0.02,
                               "bernoulli", rate=0.05),
    # DeepSeek-V3-style layer, 128 shards, 0.5% clustered
    "dsv3_layer": Workload("dsv3_layer", 128, DSV3_LAYER // 128, 0.006,
                           "clustered",
                           cluster=dict(c_hot=0.9 * 0.005 / 0.10,
                                        c_cold=0.1 * 0.005 / 0.90,
                                        hot_frac=0.10, cluster=4096)),
}


def shard_pair(wl: Workload, shard: int, device="cpu", tag=""):
    """(W bits, W' bits) of one rank's shard of a workload."""
    w = normal_bf16_bits(wl.shard_elems, wl.std,
                         seed_for(wl.name, tag, "W", shard), device)
    s2 = seed_for(wl.name, tag, "update", shard)
    if wl.update == "natural":
        w2 = natural_update_bits(w, wl.noise, s2)
    elif wl.update == "bernoulli":
        w2 = forced_bernoulli_bits(w, wl.rate, s2)
    elif wl.update == "exact_k":
        w2, _ = forced_exact_k_bits(w, int(round(wl.rate * wl.shard_elems)),
                                    s2)
    elif wl.update == "clustered":
        cl = wl.cluster
        w2 = forced_clustered_bits(w, cl["c_hot"], cl["c_cold"],
                                   cl["hot_frac"], cl["cluster"], s2)
    else:
        raise ValueError(wl.update)
    return w, w2


# The mixed model step: 16 transformer layers of OLMoE-1B-7B shape.
MIXED_LAYERS = 16
MIXED_SHARDS = 16
# per-element change rates chosen so that the block change rate at B=512
# matches the per-type medians the paper reports for OLMoE (expert FFN 0.22,
# attention 0.96, router 0.94, layer norm 0.64); c = 1 - (1 - q)^(1/512)
MIXED_TENSORS = [
    # name, elements, kind
    ("q_proj", 2048 * 2048, "attention"),
    ("k_proj", 2048 * 2048, "attention"),
    ("v_proj", 2048 * 2048, "attention"),
    ("o_proj", 2048 * 2048, "attention"),
    ("router", 2048 * 64, "router"),
    ("ln_attn", 2048, "layernorm"),
    ("ln_ffn", 2048, "layernorm"),
    ("experts", OLMOE_LAYER, "expert"),
]
STEADY_RATE = {"expert": 0.000485, "attention": 0.00627, "router": 0.00548,
               "layernorm": 0.00202}
WARMUP_RATE = 0.30
