"""Seeded synthetic inputs for the DisDP parameter-server hot path.

This module only draws random numbers and holds the workload recipes.  It
contains none of the method's arithmetic (no aggregation, no optimizer step,
no rounding of results), and both the oracle side and the HIP side take their
inputs from here.

The paper trains OPT and custom OPT-shaped models (Table V) whose weights and
dataset are not available here; the shards below stand in for one
data-parallel shard of those models: N elements, W worker gradient
contributions of that shard, fp32 master weights and Adam moments.

Recipe (every value is seeded):
  * gradients: i.i.d. normal with standard deviation ``sigma`` per (workload,
    step, worker); an optional outlier tail multiplies a Bernoulli(frac)
    subset by ``outlier_scale``; bf16 contributions are the fp32 draw rounded
    to bf16 by torch's conversion;
  * master weights: normal with standard deviation 0.02; m = v = 0 at t = 1.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

BASE_SEED = 0xD15D9


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n: int                    # shard length (elements)
    W: int                    # worker contributions
    gdtype: str               # "f32" or "bf16"
    mode: str                 # "fp32" or "fixed"
    frac_bits: int            # fixed-point scale 2^k (fixed mode)
    sigma: float              # gradient standard deviation
    outlier_frac: float       # share of elements scaled by outlier_scale
    outlier_scale: float
    p_sigma: float            # master-weight standard deviation
    lr: float
    beta1: float
    beta2: float
    eps: float
    wd: float
    steps: int                # optimizer steps t = 1..steps
    wid: int                  # index used in seed derivation


WORKLOADS = {
    w.name: w for w in [
        # a tiny shard: parity at a size the oracle finishes in seconds
        Workload("tiny_n1M_w4_f32", 1_048_576, 4, "f32", "fp32", 0, 1e-3,
                 0.0, 1.0, 0.02, 1e-4, 0.9, 0.95, 1e-8, 0.1, 10, 0),
        # one 1/8 shard of a 7B-parameter model, 8 fp32 contributions with a
        # 1% x100 outlier tail
        Workload("opt7b_shard8_w8_f32", 875_000_000, 8, "f32", "fp32", 0, 1e-4,
                 0.01, 100.0, 0.02, 1e-4, 0.9, 0.95, 1e-8, 0.1, 5, 1),
        # one 1/16 shard of a 13B-parameter model, 16 bf16 contributions
        Workload("opt13b_shard16_w16_bf16", 812_500_000, 16, "bf16", "fp32", 0,
                 1e-4, 0.0, 1.0, 0.02, 3e-4, 0.9, 0.95, 1e-8, 0.1, 5, 2),
        # one 1/64 shard of a 175B-parameter model, integer aggregation at 2^24
        Workload("c175b_shard64_w8_fixed24", 2_734_375_000, 8, "f32", "fixed",
                 24, 1e-4, 0.0, 1.0, 0.02, 1e-4, 0.9, 0.95, 1e-8, 0.1, 5, 3),
    ]
}


def opt_tensor_shards(hidden: int = 4096, ffn: int = 16384, layers: int = 32,
                      vocab: int = 50272, positions: int = 2048, shards: int = 8):
    """Element counts of one data-parallel shard (1/shards, rounded up) of
    each parameter tensor of an OPT-style decoder, in model order: token and
    position embeddings, then per layer the fused QKV weight and bias, the
    output projection and bias, the first LayerNorm (weight and bias), the
    two MLP weights and biases, and the second LayerNorm.  The defaults are
    OPT-6.7B's shapes (about 6.66e9 parameters, 8.3e8 per shard of 8)."""
    def cut(x):
        return -(-x // shards)
    sizes = [cut(vocab * hidden), cut(positions * hidden)]
    for _ in range(layers):
        sizes += [cut(3 * hidden * hidden), cut(3 * hidden), cut(hidden * hidden), cut(hidden),
                  cut(2 * hidden), cut(hidden * ffn), cut(ffn), cut(ffn * hidden), cut(hidden),
                  cut(2 * hidden)]
    return sizes


def seed_for(wid: int, step: int, stream: int) -> int:
    """A 63-bit seed per (workload, step, stream); stream < 1000 are workers,
    1000 is the master weights, 1001+ are auxiliary draws."""
    x = (BASE_SEED * 1_000_003 + wid) * 1_000_003 + step
    x = x * 1_000_003 + stream
    # splitmix64 finaliser to decorrelate neighbouring seeds
    x &= (1 << 64) - 1
    x ^= x >> 30
    x = (x * 0xBF58476D1CE4E5B9) & ((1 << 64) - 1)
    x ^= x >> 27
    x = (x * 0x94D049BB133111EB) & ((1 << 64) - 1)
    x ^= x >> 31
    return x & ((1 << 63) - 1)


# --------------------------------------------------------------------- host --
def host_normal(seed: int, n: int, sigma: float) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(n, dtype=np.float32) * np.float32(sigma))


def host_grads(wid: int, step: int, W: int, n: int, sigma: float,
               gdtype: str = "f32", outlier_frac: float = 0.0,
               outlier_scale: float = 1.0) -> List[np.ndarray]:
    """W contributions as numpy arrays: float32, or uint16 bf16 bits."""
    out = []
    for w in range(W):
        s = seed_for(wid, step, w)
        g = host_normal(s, n, sigma)
        if outlier_frac > 0:
            u = np.random.default_rng(s ^ 0x5EED).random(n, dtype=np.float32)
            g = np.where(u < outlier_frac, g * np.float32(outlier_scale), g)
            g = g.astype(np.float32)
        if gdtype == "bf16":
            import torch
            g = torch.from_numpy(g).to(torch.bfloat16).view(torch.int16) \
                .numpy().view(np.uint16).copy()
        out.append(np.ascontiguousarray(g))
    return out


def host_state(wid: int, n: int, p_sigma: float = 0.02,
               mv_sigma: Optional[float] = None):
    """(p, m, v) float32.  m = v = 0 unless mv_sigma is given, in which case
    m ~ N(0, mv_sigma) and v = |N(0, mv_sigma)|^2 (a state after some steps)."""
    p = host_normal(seed_for(wid, 0, 1000), n, p_sigma)
    if mv_sigma is None:
        return p, np.zeros(n, np.float32), np.zeros(n, np.float32)
    m = host_normal(seed_for(wid, 0, 1001), n, mv_sigma)
    r = host_normal(seed_for(wid, 0, 1002), n, mv_sigma)
    v = (r * r).astype(np.float32)
    return p, m, v


# ------------------------------------------------------------------- device --
def device_grad(wid: int, step: int, w: int, n: int, sigma: float,
                gdtype: str = "f32", outlier_frac: float = 0.0,
                outlier_scale: float = 1.0, device="cuda"):
    """Worker w's contribution as a device tensor (float32, or int16 bf16
    bits), drawn by torch's device generator."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed_for(wid, step, w))
    g = torch.randn(n, generator=gen, device=device, dtype=torch.float32)
    g.mul_(sigma)
    if outlier_frac > 0:
        u = torch.rand(n, generator=gen, device=device, dtype=torch.float32)
        g = torch.where(u < outlier_frac, g * outlier_scale, g)
        del u
    if gdtype == "bf16":
        g = g.to(torch.bfloat16).view(torch.int16)
    return g


def device_grads(wid: int, step: int, W: int, n: int, sigma: float,
                 gdtype: str = "f32", outlier_frac: float = 0.0,
                 outlier_scale: float = 1.0, device="cuda", out=None):
    """The W contributions (see device_grad).  ``out`` (a list of W tensors of
    the right dtype and length) is refilled in place when given."""
    bufs = []
    for w in range(W):
        g = device_grad(wid, step, w, n, sigma, gdtype, outlier_frac, outlier_scale, device)
        if out is not None:
            out[w].copy_(g)
            del g
        else:
            bufs.append(g)
    return out if out is not None else bufs


def device_state(wid: int, n: int, p_sigma: float = 0.02, device="cuda", out=None):
    """(p, m, v) on the device: p ~ N(0, p_sigma), m = v = 0.  `out` (three
    float32 tensors of length n) is filled in place when given."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed_for(wid, 0, 1000))
    p = torch.randn(n, generator=gen, device=device, dtype=torch.float32)
    p.mul_(p_sigma)
    if out is not None:
        out[0].copy_(p)
        del p
        out[1].zero_()
        out[2].zero_()
        return tuple(out)
    m = torch.zeros(n, device=device, dtype=torch.float32)
    v = torch.zeros(n, device=device, dtype=torch.float32)
    return p, m, v
