"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

This module only draws random numbers and fixes shapes; it holds none of the
method's arithmetic (no quantisation, packing or attention).  Every draw is
seeded.  Shapes follow the backbones of App. B (Qwen2.5-7B: 28 layers, 4 KV
heads; Qwen2.5-14B: 48 layers, 8 KV heads; head dim 128) and the workloads of
the decode benchmark; key tensors carry a per-channel log-normal outlier scale,
the per-channel key structure App. A cites from KVQuant.

Plans are drawn the way the workloads describe them: a random subset of layers
inherits (never layer 0), anchor bit-widths (and, for the MLA-style stack, kept
latent widths) are drawn uniformly.  The MLA-style stack follows the paper's
converted 7B geometry (latent 512 + 64, App. C.2) with 32 heads and 128-wide
no-RoPE and value heads; its up-projections are N(0, 1/r).
"""
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

GQA, MLA = 0, 1
KIVI32, SYMROW = 0, 1


@dataclass
class Workload:
    name: str
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    batch: int
    tokens: int
    keep_tokens: int = 0
    in_dtype: torch.dtype = torch.bfloat16
    q_dtype: torch.dtype = torch.bfloat16
    key_outliers: bool = True
    scale: float = 0.0
    qscheme: int = KIVI32
    plan: List[tuple] = field(default_factory=list)  # (inherit, bits) per layer
    seed: int = 0

    def softmax_scale(self) -> float:
        return self.scale if self.scale > 0 else 1.0 / float(np.sqrt(self.head_dim))


def plan_uniform(n_layers: int, bits: int):
    return [(0, bits)] * n_layers


def plan_mixed(seed: int, n_layers: int, n_inherit: int, bit_choices=(16, 8, 4, 2)):
    """A random plan: n_inherit layers drawn from 1..L-1 inherit; every anchor's
    bit-width is drawn uniformly from bit_choices."""
    rng = np.random.default_rng(seed)
    inh = set(int(x) for x in rng.choice(np.arange(1, n_layers), n_inherit, replace=False))
    plan = []
    for l in range(n_layers):
        if l in inh:
            plan.append((1, 16))
        else:
            plan.append((0, int(rng.choice(bit_choices))))
    return plan


def plan_grouped(seed: int, group_sizes, anchor_bits):
    """Anchors each followed by inheritors: group_sizes[i] consecutive layers share
    one anchor whose bit-width is anchor_bits[i]; the order of the groups and of
    the bit-widths is shuffled with the seed."""
    rng = np.random.default_rng(seed)
    sizes = list(rng.permutation(group_sizes))
    bits = list(rng.permutation(anchor_bits))
    plan = []
    for g, b in zip(sizes, bits):
        plan.append((0, int(b)))
        plan.extend([(1, 16)] * (int(g) - 1))
    return plan


def workload(cfg: int, variant: Optional[str] = None) -> Workload:
    """The five decode workloads.  cfg 0: tiny single layer; 1: Qwen2.5-7B-shaped
    all-int4 (variants 'bf16', 'int8', 'int2': every layer at that precision); 2: Qwen2.5-14B-shaped mixed plan with
    depth sharing (variant 'one-anchor-<bits>': layer 0's cache serves all 48); 4: 14B-shaped, 128k context, half the positions evicted, an
    int2/int4 plan in pairs and triples."""
    if cfg == 0:
        return Workload("tiny-gqa-int8", 1, 4, 1, 64, 1, 256, in_dtype=torch.float32,
                        q_dtype=torch.float32, key_outliers=False, scale=1.0 / 8.0,
                        plan=plan_uniform(1, 8), seed=1000)
    if cfg == 1:
        bits = {"bf16": 16, "int8": 8, "int2": 2}.get(variant, 4)
        name = "bf16" if bits == 16 else f"int{bits}"
        return Workload(f"qwen2.5-7b-shape-{name}", 28, 28, 4, 128, 8, 8192, plan=plan_uniform(28, bits), seed=1001)
    if cfg == 2:
        if variant and variant.startswith("one-anchor-"):  # depth's extreme: one cache for all 48 layers
            bits = int(variant.split("-")[-1])
            return Workload(f"qwen2.5-14b-shape-one-anchor-b{bits}", 48, 40, 8, 128, 32, 8192,
                            plan=[(0, bits)] + [(1, 16)] * 47, seed=1002)
        return Workload("qwen2.5-14b-shape-mixed", 48, 40, 8, 128, 32, 8192,
                        plan=plan_mixed(1002, 48, 16), seed=1002)
    if cfg == 4:
        plan = plan_grouped(1004, [2] * 12 + [3] * 8, [2] * 16 + [4] * 4)
        return Workload("qwen2.5-14b-shape-128k-evict", 48, 40, 8, 128, 4, 131072,
                        keep_tokens=65536, plan=plan, seed=1004)
    raise ValueError(f"unknown workload {cfg}")


def plans_per_sequence(w: Workload, n_inherit: int = 16):
    """One plan per sequence of the 14B-shaped mixed workload, each drawn like the
    shared plan (its own seed): the selector maps every prompt to its own plan."""
    return [plan_mixed(w.seed * 1000 + b, w.n_layers, n_inherit) for b in range(w.batch)]


def mla_plans_per_sequence(w: "MlaWorkload"):
    """One plan per sequence of an MLA workload, each drawn like the shared plan
    (its own seed): every anchor's kept width from {r, r/2, r/4, r/8}, the shared
    plan's bit-width."""
    bits = w.plan[0][1]
    return [plan_ranks(w.seed * 1000 + b, w.n_layers, w.latent_dim, bits) for b in range(w.batch)]


@dataclass
class MlaWorkload:
    """An MLA-style stack (§2.1 rank axis): one latent of width r per token shared by
    the heads, a 64-wide positional key, per-head no-RoPE query/key width 128 and
    value width 128.  plan entries are (inherit, bits, rank)."""
    name: str
    n_layers: int
    n_q_heads: int
    latent_dim: int
    batch: int
    tokens: int
    plan: List[tuple]
    rope_dim: int = 64
    nope_dim: int = 128
    v_dim: int = 128
    keep_tokens: int = 0
    qscheme: int = KIVI32
    ref_kv_heads: int = 4    # the bf16 GQA model eq. (2) is quoted against
    ref_head_dim: int = 128
    d_model: int = 2048      # hidden-state width the down-projection W_DKV reads
    in_dtype: torch.dtype = torch.bfloat16
    q_dtype: torch.dtype = torch.bfloat16
    seed: int = 1003

    def softmax_scale(self) -> float:
        return 1.0 / float(np.sqrt(self.nope_dim + self.rope_dim))


def plan_ranks(seed: int, n_layers: int, latent_dim: int, bits: int, n_inherit: int = 0):
    """Every anchor's kept width drawn uniformly from {r, r/2, r/4, r/8}; n_inherit
    layers drawn from 1..L-1 inherit."""
    rng = np.random.default_rng(seed)
    inh = set()
    if n_inherit:
        inh = set(int(x) for x in rng.choice(np.arange(1, n_layers), n_inherit, replace=False))
    ranks = [latent_dim, latent_dim // 2, latent_dim // 4, latent_dim // 8]
    return [(1, 16, 0) if l in inh else (0, bits, int(rng.choice(ranks))) for l in range(n_layers)]


def plan_ranks_grouped(seed: int, n_layers: int, latent_dim: int, bits: int, sizes=(2, 3, 4)):
    """Depth groups on the rank axis: consecutive groups of 2-4 layers (sizes drawn
    uniformly, the last group cut to fit), each an anchor whose kept width is drawn
    from {r, r/2, r/4, r/8} followed by inheritors."""
    rng = np.random.default_rng(seed)
    ranks = [latent_dim, latent_dim // 2, latent_dim // 4, latent_dim // 8]
    plan = []
    while len(plan) < n_layers:
        g = min(int(rng.choice(sizes)), n_layers - len(plan))
        plan.append((0, bits, int(rng.choice(ranks))))
        plan.extend([(1, 16, 0)] * (g - 1))
    return plan


def mla_workload(variant: Optional[str] = None) -> MlaWorkload:
    """The MLA-style decode workload: 32 layers, 32 query heads, latent 512 + 64,
    batch 16, context 16384, per-layer kept width drawn from {512, 256, 128, 64};
    variant None: bf16 cache, 'int4': KIVI32 4-bit latent and positional key;
    'depth' / 'int4-depth': the same with the layers in depth groups of 2-4 (one
    anchor each, its kept width drawn as above).  '14b' / '14b-int4': Qwen2.5-14B's
    latent shape (48 layers, 40 query heads, latent 1024 + 64, the bf16 GQA model
    it is quoted against 8 KV heads of 128, model width 5120), batch 32, context
    8192, kept widths drawn from {1024, 512, 256, 128}.  The 32-layer stack's model
    width (for the projected write) is DeepSeek-V2-Lite's, 2048."""
    if variant in ("14b", "14b-int4"):
        bits = 4 if variant == "14b-int4" else 16
        return MlaWorkload("mla-48l-r1024-" + ("bf16" if bits == 16 else "int4"), 48, 40, 1024, 32, 8192,
                           plan_ranks(1007, 48, 1024, bits), ref_kv_heads=8, d_model=5120, seed=1007)
    bits = 4 if variant in ("int4", "int4-depth") else 16
    name = "mla-32l-r512-" + ("bf16" if bits == 16 else "int4")
    if variant in ("depth", "int4-depth"):
        return MlaWorkload(name + "-depth", 32, 32, 512, 16, 16384, plan_ranks_grouped(1005, 32, 512, bits))
    return MlaWorkload(name, 32, 32, 512, 16, 16384, plan_ranks(1003, 32, 512, bits))


def mla_layer(w: MlaWorkload, layer: int, device="cpu", batch: Optional[int] = None,
              tokens: Optional[int] = None):
    """Latent [B, T, r] and positional key [B, T, d_R] of one layer, N(0,1), in w.in_dtype."""
    B = w.batch if batch is None else batch
    T = w.tokens if tokens is None else tokens
    g = generator(w.seed * 1000 + layer, device)
    c = torch.randn((B, T, w.latent_dim), generator=g, device=device, dtype=torch.float32)
    r = torch.randn((B, T, w.rope_dim), generator=g, device=device, dtype=torch.float32)
    return c.to(w.in_dtype), r.to(w.in_dtype)


def mla_weights(w: MlaWorkload, n_layers: int, device="cpu"):
    """W_UK [L, Hq, nope, r] and W_UV [L, Hq, v, r], N(0, 1/r), bf16."""
    g = generator(w.seed * 1000 + 777, device)
    sd = 1.0 / float(np.sqrt(w.latent_dim))
    wk = torch.randn((n_layers, w.n_q_heads, w.nope_dim, w.latent_dim), generator=g, device=device) * sd
    wv = torch.randn((n_layers, w.n_q_heads, w.v_dim, w.latent_dim), generator=g, device=device) * sd
    return wk.to(torch.bfloat16), wv.to(torch.bfloat16)


def mla_queries(w: MlaWorkload, n_layers: int, device="cpu", batch: Optional[int] = None):
    """q [L, B, Hq, nope + d_R] ~ N(0,1): per head q_nope then q_rope."""
    B = w.batch if batch is None else batch
    g = generator(w.seed * 1000 + 999, device)
    q = torch.randn((n_layers, B, w.n_q_heads, w.nope_dim + w.rope_dim), generator=g, device=device)
    return q.to(w.q_dtype)


def generator(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def kv_layer(w: Workload, layer: int, device="cpu", batch: Optional[int] = None,
             tokens: Optional[int] = None):
    """K, V [B, Hkv, T, D] of one layer in w.in_dtype: N(0,1) values; keys times a
    per-(layer, KV head, channel) LogNormal(0,1) scale when w.key_outliers."""
    B = w.batch if batch is None else batch
    T = w.tokens if tokens is None else tokens
    g = generator(w.seed * 1000 + layer, device)
    shape = (B, w.n_kv_heads, T, w.head_dim)
    k = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    v = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if w.key_outliers:
        ch = torch.randn((1, w.n_kv_heads, 1, w.head_dim), generator=g, device=device,
                         dtype=torch.float32).exp()
        k = k * ch
    return k.to(w.in_dtype), v.to(w.in_dtype)


def queries(w: Workload, n_layers: int, device="cpu", seed_offset: int = 0,
            batch: Optional[int] = None):
    """q [n_layers, B, Hq, D] ~ N(0,1) in w.q_dtype."""
    B = w.batch if batch is None else batch
    g = generator(w.seed * 1000 + 999 + seed_offset, device)
    q = torch.randn((n_layers, B, w.n_q_heads, w.head_dim), generator=g, device=device,
                    dtype=torch.float32)
    return q.to(w.q_dtype)


def keep_positions(w: Workload, layer: int, device="cpu", batch: Optional[int] = None,
                   tokens: Optional[int] = None, keep: Optional[int] = None):
    """Sorted kept positions [B, Hkv, keep] (int32): a seeded uniform subset of
    size keep of range(T) per (sequence, KV head)."""
    B = w.batch if batch is None else batch
    T = w.tokens if tokens is None else tokens
    K = w.keep_tokens if keep is None else keep
    g = generator(w.seed * 1000 + 500 + layer, device)
    r = torch.rand((B, w.n_kv_heads, T), generator=g, device=device)
    idx = torch.topk(r, K, dim=-1).indices
    return torch.sort(idx, dim=-1).values.to(torch.int32)


def kv_random(seed: int, B: int, H: int, T: int, D: int, dtype=torch.bfloat16, outliers=True,
              device="cpu", scale: float = 1.0):
    """K, V [B, H, T, D]: N(0, scale^2) values, keys times a per-(head, channel)
    LogNormal(0,1) factor when outliers."""
    g = generator(seed, device)
    k = torch.randn((B, H, T, D), generator=g, device=device) * scale
    v = torch.randn((B, H, T, D), generator=g, device=device) * scale
    if outliers:
        k = k * torch.randn((1, H, 1, D), generator=g, device=device).exp()
    return k.to(dtype), v.to(dtype)


def latent_random(seed: int, B: int, T: int, W: int, dtype=torch.bfloat16, device="cpu", scale: float = 1.0):
    """[B, T, W] ~ N(0, scale^2) (latents or positional keys)."""
    g = generator(seed, device)
    return (torch.randn((B, T, W), generator=g, device=device) * scale).to(dtype)


def weights_random(seed: int, L: int, H: int, rows: int, r: int, device="cpu"):
    """[L, H, rows, r] ~ N(0, 1/r), bf16 (up-projections)."""
    g = generator(seed, device)
    return (torch.randn((L, H, rows, r), generator=g, device=device) / float(np.sqrt(r))).to(torch.bfloat16)


def q_random(seed: int, L: int, B: int, Hq: int, D: int, dtype=torch.bfloat16, device="cpu"):
    """q [L, B, Hq, D] ~ N(0, 1)."""
    g = generator(seed, device)
    return torch.randn((L, B, Hq, D), generator=g, device=device).to(dtype)


def keep_random(seed: int, B: int, H: int, T: int, keep: int, device="cpu"):
    """Sorted kept positions [B, H, keep] (int32), a uniform subset per (b, h)."""
    g = generator(seed, device)
    r = torch.rand((B, H, T), generator=g, device=device)
    idx = torch.topk(r, keep, dim=-1).indices
    return torch.sort(idx, dim=-1).values.to(torch.int32)
